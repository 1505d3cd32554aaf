"""Python entry to the CPU oracle (``kvoracle.cpp``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg call this module; the GPU library never does, and this
module never imports the GPU library.

* :func:`replay`     literal per-configuration tiered replay -> counts
                     uint64[n_cfg, n_groups, 3, 8] with fields
                     (hit, miss, ins, evict, hit_w, miss_w, ins_w, evict_w).
* :func:`replay_memo` the same counts, with each distinct inclusive tier
                     cache (partition, policy, capacity) replayed once and
                     shared by the configurations that use it (for the
                     full-size expected values).
* :func:`objectives` (cost, throughput, latency) per configuration.
* :func:`pareto`     non-dominated flags by brute force.
* :func:`ttl_curves` per group and time-to-live, the disk tier's hits and
                     storage integral from the inter-arrival times
                     (Section 4.3), in plain Python and numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "kvoracle.cpp")

FIELDS = ("hit", "miss", "ins", "evict", "hit_w", "miss_w", "ins_w", "evict_w")
HIT, MISS, INS, EVICT, HIT_W, MISS_W, INS_W, EVICT_W = range(8)

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (no GPU compiler involved)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fPIC", "-shared",
               "-pthread", SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        p = ctypes.c_void_p
        lib.oracle_replay.restype = ctypes.c_int
        lib.oracle_replay.argtypes = [ctypes.c_uint64, p, p, p, p, ctypes.c_uint32,
                                      ctypes.c_uint32, p, p, p, p, p, p, p, p,
                                      ctypes.c_uint32, p, p]
        lib.oracle_replay_memo.restype = ctypes.c_int
        lib.oracle_replay_memo.argtypes = lib.oracle_replay.argtypes
        lib.oracle_objectives.restype = ctypes.c_int
        lib.oracle_objectives.argtypes = [ctypes.c_uint32, p, p, ctypes.c_uint32, p,
                                          ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_double, ctypes.c_uint64, p, p, p, p]
        lib.oracle_pareto.restype = ctypes.c_int64
        lib.oracle_pareto.argtypes = [ctypes.c_uint32, p, p, p, p]
        _lib = lib
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def replay(trace, cfgs, threads: int | None = None, memo: bool = False,
           with_store: bool = False):
    """Literal replay of every configuration of ``cfgs`` over ``trace``.

    With ``memo`` the inclusive configurations share their tier caches: an
    inclusive tier is an independent cache that sees every access of its
    partition, so each distinct (partition, policy, capacity) cache is
    replayed once, literally, with a presence bit per access, and every
    configuration is classified from its tiers' bits (served by k = present
    in k and in no faster present tier).  The results are the same.

    With ``with_store`` also returns, per configuration, the occupancy
    integral (granule-seconds) of an unbounded disk TTL tier (0 otherwise)."""
    lib = _load()
    n_cfg = cfgs.n
    g = trace.n_groups
    out = np.zeros((n_cfg, g, 3, 8), dtype=np.uint64)
    h = np.ascontiguousarray(trace.hash, dtype=np.uint64)
    gr = np.ascontiguousarray(trace.group, dtype=np.uint8)
    w = np.ascontiguousarray(trace.weight, dtype=np.uint8)
    cap = np.ascontiguousarray(cfgs.cap, dtype=np.uint64)
    cg = np.ascontiguousarray(cfgs.cap_group, dtype=np.uint64)
    mode = np.ascontiguousarray(cfgs.mode, dtype=np.uint8)
    part = np.ascontiguousarray(cfgs.partitioned, dtype=np.uint8)
    pol = np.ascontiguousarray(cfgs.policy, dtype=np.uint8)
    rq = np.ascontiguousarray(trace.req, dtype=np.uint32)
    dt = np.ascontiguousarray(cfgs.disk_ttl, dtype=np.uint8)
    tl = np.ascontiguousarray(cfgs.ttl, dtype=np.float64)
    rt = np.ascontiguousarray(trace.req_time, dtype=np.float64)
    store = np.zeros(n_cfg, dtype=np.float64)
    fn = lib.oracle_replay_memo if memo else lib.oracle_replay
    rc = fn(trace.n, _ptr(h), _ptr(gr), _ptr(w), _ptr(rq), g, n_cfg, _ptr(cap), _ptr(cg),
            _ptr(mode), _ptr(part), _ptr(pol), _ptr(dt), _ptr(tl), _ptr(rt),
            threads or default_threads(), _ptr(out), _ptr(store))
    if rc != 0:
        raise ValueError(f"oracle_replay rejected the batch (code {rc})")
    return (out, store) if with_store else out


def replay_memo(trace, cfgs, threads: int | None = None) -> np.ndarray:
    return replay(trace, cfgs, threads, memo=True)


def cost_vector(cost: dict) -> np.ndarray:
    media = list(cost.get("media", ()))
    v = [cost["price_gpu_per_hour"], *cost["price_per_gib_hour"], cost["bw_dram"],
         cost["ssd_bw_base"], cost["ssd_bw_per_gib"], cost["ssd_bw_max"],
         cost["t_prefill_per_token"], float(len(media))]
    for m in media:
        v.extend(float(x) for x in m)
    return np.array(v, dtype=np.float64)


def objectives(trace, cfgs, counts, cost: dict, store=None) -> np.ndarray:
    """(cost, throughput, latency) per configuration.  ``store`` is the
    occupancy integral of unbounded disk TTL tiers (from ``replay(...,
    with_store=True)``); when omitted and needed it is replayed here."""
    lib = _load()
    need = (np.asarray(cfgs.disk_ttl) != 0) & (np.asarray(cfgs.cap)[:, 2] == 0)
    if store is None:
        store = np.zeros(cfgs.n, dtype=np.float64)
        if need.any():
            sub = cfgs.subset(np.nonzero(need)[0])
            store[need] = replay(trace, sub, memo=True, with_store=True)[1]
    store = np.ascontiguousarray(store, dtype=np.float64)
    n_cfg = cfgs.n
    obj = np.zeros((n_cfg, 3), dtype=np.float64)
    cap = np.ascontiguousarray(cfgs.cap, dtype=np.uint64)
    cnt = np.ascontiguousarray(counts, dtype=np.uint64)
    cm = cost_vector(cost)
    n_w = int(trace.weight.astype(np.uint64).sum())
    span = float(trace.req_time[-1] - trace.req_time[0])
    dt = np.ascontiguousarray(cfgs.disk_ttl, dtype=np.uint8)
    md = np.ascontiguousarray(cfgs.medium, dtype=np.uint8)
    lib.oracle_objectives(n_cfg, _ptr(cap), _ptr(cnt), trace.n_groups, _ptr(cm),
                          float(trace.granule_bytes), float(trace.tokens_per_granule),
                          span, float(trace.n_req), n_w, _ptr(dt), _ptr(md), _ptr(store),
                          _ptr(obj))
    return obj


def pareto(obj, segment=None, bounds=None) -> np.ndarray:
    lib = _load()
    o = np.ascontiguousarray(obj, dtype=np.float64)
    n = o.shape[0]
    seg = None if segment is None else np.ascontiguousarray(segment, dtype=np.uint32)
    b = None if bounds is None else np.ascontiguousarray(bounds, dtype=np.float64)
    flag = np.zeros(n, dtype=np.uint8)
    rc = lib.oracle_pareto(n, _ptr(o), _ptr(seg), _ptr(b), _ptr(flag))
    if rc < 0:
        raise ValueError("NaN objective")
    return flag


def ttl_curves(trace, ttl):
    """TTL retention curves of the disk tier (Section 4.3).

    A block stays on disk for ``t`` seconds after each access.  Delta_g is the
    multiset of inter-arrival times of group g's blocks: for every access
    whose block was accessed before, the request time of the access minus the
    request time of the block's previous access.  Per group g and each t:

    * hits[g, k]  = H_g(t) = #{delta in Delta_g : delta <= t}
    * hitw[g, k]  = the summed block weight of those accesses
    * store[g, k] = sum over g's blocks b of w_b * (sum of min(t, delta) over
      b's gaps + t), the storage-time integral in granule-seconds; with unit
      weights this is C_g(t) = |B_g| * t + sum over Delta_g of min(t, delta).

    A walk over the accesses in trace order (pure Python: small traces).
    Returns (hits uint64 [G, K], hitw uint64 [G, K], store float64 [G, K]).
    """
    G = int(trace.n_groups)
    ttl = [float(x) for x in ttl]
    last = {}                               # block hash -> time of its latest access
    gaps = [[] for _ in range(G)]           # per group: (delta, weight)
    block_w = [0] * G                       # per group: weight of its distinct blocks
    times = np.asarray(trace.req_time, dtype=np.float64)
    for i in range(int(trace.n)):
        h = int(trace.hash[i])
        now = float(times[int(trace.req[i])])
        g = int(trace.group[i])
        w = int(trace.weight[i])
        if h in last:
            gaps[g].append((now - last[h], w))
        else:
            block_w[g] += w
        last[h] = now
    hits = np.zeros((G, len(ttl)), dtype=np.uint64)
    hitw = np.zeros((G, len(ttl)), dtype=np.uint64)
    store = np.zeros((G, len(ttl)), dtype=np.float64)
    for g in range(G):
        d = np.array([x for x, _ in gaps[g]], dtype=np.float64)
        w = np.array([y for _, y in gaps[g]], dtype=np.float64)
        for k, t in enumerate(ttl):
            hit = d <= t
            hits[g, k] = int(hit.sum())
            hitw[g, k] = int(w[hit].sum())
            store[g, k] = block_w[g] * t + float((w * np.minimum(t, d)).sum())
    return hits, hitw, store
