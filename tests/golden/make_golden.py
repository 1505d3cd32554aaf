"""Writes the stored expected counts of the five benchmark workloads.

    python tests/golden/make_golden.py [tiny chat ... longctx_leaf] [--threads N]

Every count comes from the CPU oracle (``oracle.replay_memo``: each distinct
inclusive tier cache replayed once, literally; exclusive configurations
replayed literally one by one) over the trace the seeded generator builds on
the CPU.  Nothing here touches the GPU library.  Each file records the
generator version, the seed, a sha256 of the trace arrays and of the
configuration batch, and the indices of the configurations it covers: all
of them, except for the two largest batches: of the long-context workload's
2,048 exclusive configurations the 8 corners of its 8 x 16 x 16 grid plus 56
seeded draws (exclusive configurations cannot share caches, so each one is a
full literal replay), and of the full workload's 11,000 configurations over
387 M accesses the 8 corners of its LRU grid, 8 more LRU draws and 8 draws
each of its FIFO and LFU points (every distinct tier cache is a literal
replay of the whole trace).  Two variants evaluate the chat trace under other
batches: its grid under radix-tree (leaf-first) eviction (``chat_leaf``), an
HBM x DRAM x disk-TTL grid over an unbounded TTL disk tier (``chat_ttl``),
and a 32-point grid of exclusive FIFO and LFU hierarchies (``chat_excl``), all
configurations of each; and two over the large traces:
the full workload's trace over a 16-point HBM x DRAM x disk-TTL grid
(``full_ttl``) and the long-context trace under leaf-first eviction on a
64-point inclusive subset of its grid (``longctx_leaf``).
"""
from __future__ import annotations

import argparse
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import tracegen as tg  # noqa: E402
from tracegen.digest import configs_digest, trace_digest  # noqa: E402
from oracle import oracle as O  # noqa: E402

NAMES = ("tiny", "chat", "tenant", "longctx", "full", "chat_leaf", "chat_ttl", "chat_excl",
         "full_ttl", "longctx_leaf")


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"counts_{name}.npz")


def subset(name: str, n_cfg: int) -> np.ndarray:
    if name == "full":
        # 10,000 LRU grid points (25 x 20 x 20, index (h * 20 + d) * 20 + s),
        # then 500 FIFO and 500 LFU points: the 8 LRU grid corners, 8 more
        # LRU draws and 8 draws of each replay policy
        corners = [(h * 20 + d) * 20 + s for h in (0, 24) for d in (0, 19) for s in (0, 19)]
        rng = np.random.default_rng([5, 23])
        lru = rng.choice(np.setdiff1d(np.arange(10000), corners), size=8, replace=False)
        fifo = 10000 + rng.choice(500, size=8, replace=False)
        lfu = 10500 + rng.choice(500, size=8, replace=False)
        return np.sort(np.concatenate([corners, lru, fifo, lfu])).astype(np.uint32)
    if name != "longctx":
        return np.arange(n_cfg, dtype=np.uint32)
    # grid index = (h * 16 + d) * 16 + s over the 8 x 16 x 16 grid
    corners = [(h * 16 + d) * 16 + s for h in (0, 7) for d in (0, 15) for s in (0, 15)]
    rest = np.setdiff1d(np.arange(n_cfg), corners)
    rng = np.random.default_rng([5, 17])
    pick = rng.choice(rest, size=56, replace=False)
    return np.sort(np.concatenate([corners, pick])).astype(np.uint32)


def make(name: str, threads: int) -> str:
    t0 = time.time()
    rec = tg.recipe(tg.trace_of(name))
    tr = rec.to_trace()
    seed = int(tr.meta.get("seed", -1))
    cfgs = tg.configs_for(name, tr)
    idx = subset(name, cfgs.n)
    sub = cfgs.subset(idx)
    dig = trace_digest(tr.hash, tr.req, tr.group, tr.weight, tr.req_time)
    t1 = time.time()
    print(f"[golden] {name}: {tr.n} accesses, {sub.n} of {cfgs.n} configs, trace {t1 - t0:.1f} s",
          flush=True)
    # with a disk TTL tier, also the oracle's storage-time integral of the
    # unbounded ones (the objectives bill it)
    store = None
    if np.any(sub.disk_ttl):
        counts, store = O.replay(tr, sub, threads, memo=True, with_store=True)
    else:
        counts = O.replay_memo(tr, sub, threads=threads)
    t2 = time.time()
    src = open(os.path.join(ROOT, "oracle", "kvoracle.cpp"), "rb").read()
    out = golden_path(name)
    np.savez_compressed(
        out, counts=counts, idx=idx, n_cfg_total=np.uint32(cfgs.n),
        trace_sha=np.array(dig), configs_sha=np.array(configs_digest(cfgs)),
        generator_version=np.uint32(tg.GENERATOR_VERSION), seed=np.int64(seed),
        n=np.uint64(tr.n), n_groups=np.uint32(tr.n_groups),
        oracle_sha=np.array(hashlib.sha256(src).hexdigest()),
        oracle_seconds=np.float64(t2 - t1), threads=np.uint32(threads),
        **({"store": store} if store is not None else {}))
    print(f"[golden] {name}: oracle {t2 - t1:.1f} s on {threads} threads -> {out}", flush=True)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("names", nargs="*", default=list(NAMES))
    ap.add_argument("--threads", type=int, default=O.default_threads())
    a = ap.parse_args()
    O.build(force=False)
    for n in a.names:
        make(n, a.threads)


if __name__ == "__main__":
    main()
