"""GPU parity of radix-tree (leaf-first) eviction (Section 3.2).

The library evaluates it as LRU stack distances over the trace with every
request followed by a re-touch of its blocks, deepest first (a 2N-position
order whose re-touches are not binned); the oracle keeps the prefix tree
literally.  Counts are compared element by element and objectives to 1e-6.
Cases: random weighted prefix trees (requests spanning many 8,192-position
blocks of the doubled order), inclusive three-tier batches mixed with every
other policy and mode, the tiny workload, and the refusals (traces that are
not prefix chains, capacities below the heaviest request, partitioned
tiers).
"""
import sys

import numpy as np
import pytest

import tracegen as tg
from tests import bruteforce as bf

pytestmark = pytest.mark.gpu
LEAF = tg.POLICY_LEAF


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def chain_trace(seed, n_req, weights=(1,), **kw):
    labels, req = bf.chain_trace_labels(seed, n_req, **kw)
    rng = np.random.default_rng(seed)
    wl = {b: int(rng.choice(weights)) for b in set(labels)}
    t = tg.from_blocks(labels, weights=wl)
    t.req = np.asarray(req, dtype=np.uint32)
    t.req_time = np.cumsum(rng.exponential(1.0, int(t.req[-1]) + 1))
    return t


def heaviest(t):
    return int(np.bincount(t.req, weights=t.weight.astype(np.float64)).max())


def compare(O, t, cfgs, label):
    from paper_2603_08739_amd import host
    say(f"  case {label}: n={t.n} configs={cfgs.n}")
    h = host.load(t)
    counts, obj = host.evaluate(h, cfgs, tg.DEFAULT_COST, t.n_groups)
    h.free()
    ref = O.replay(t, cfgs, memo=True)
    if not np.array_equal(counts, ref):
        bad = np.argwhere(counts != ref)
        c, g, k, f = bad[0]
        raise AssertionError(f"{label}: {len(bad)} mismatches; first cfg {c} tier {k} field {f}: "
                             f"gpu {counts[c, g, k, f]} oracle {ref[c, g, k, f]} cap {cfgs.cap[c]} "
                             f"policy {cfgs.policy[c, 0]}")
    np.testing.assert_allclose(obj, O.objectives(t, cfgs, ref, tg.DEFAULT_COST), rtol=1e-6,
                               atol=0)


def leaf_batch(seed, t, n):
    rng = np.random.default_rng([seed, 9])
    lo = heaviest(t)
    hi = max(lo + 1, int(t.weight.astype(np.int64).sum()))
    items = []
    for _ in range(n):
        caps = [0 if rng.random() < 0.3 else int(rng.integers(lo, hi)) for _ in range(3)]
        if not any(caps):
            caps[0] = lo
        items.append({"cap": tuple(caps), "policy": LEAF})
    return tg.from_list(items)


@pytest.mark.parametrize("seed", range(8))
def test_random_prefix_trees(oracle_mod, seed):
    t = chain_trace(seed, 400 + 200 * seed, weights=(1,) if seed % 2 else (1, 4),
                    n_docs=30 + 10 * seed, doc_len=(1, 40))
    compare(oracle_mod, t, leaf_batch(seed, t, 30), f"tree{seed}")


def test_many_blocks_and_mixed_batch(oracle_mod):
    t = chain_trace(77, 3000, weights=(1, 4), n_sys=5, n_docs=200, sys_len=(4, 30),
                    doc_len=(1, 120))
    say(f"  {t.n} accesses: {2 * t.n // 8192 + 1} blocks of the doubled order")
    lo = heaviest(t)
    leaf = leaf_batch(5, t, 40)
    other = tg.random_configs(5, 30, 1, 4, 3 * lo)
    other.cap = np.maximum(other.cap, 0)
    lru = leaf.subset(np.arange(10))
    lru.policy[:, :] = tg.POLICY_LRU
    compare(oracle_mod, t, tg.ConfigBatch.concat([leaf, other, lru, leaf.subset([0, 3])]),
            "mixed")


def test_tiny_workload(oracle_mod):
    t = tg.tiny(n_req=800)
    gib = (1 << 30) // t.granule_bytes
    items = [{"cap": (h * gib, d * gib, 0), "policy": LEAF} for h in (1, 2) for d in (0, 4, 16)]
    items += [{"cap": (h * gib, d * gib, 0)} for h in (1, 2) for d in (0, 4)]
    compare(oracle_mod, t, tg.from_list(items), "tiny")


def test_refusals():
    from paper_2603_08739_amd import host, kvcfg as K
    t = tg.random_trace(3, 2000, 300, per_request=8)   # blocks re-accessed after other parents
    h = host.load(t)
    with pytest.raises(K.KvError) as e:
        host.evaluate(h, tg.from_list([{"cap": (50, 0, 0), "policy": LEAF}]), tg.DEFAULT_COST, 1)
    assert e.value.status == K.KV_ERR_UNSUPPORTED and "prefix chains" in str(e.value)
    h.free()
    t = chain_trace(4, 300)
    lo = heaviest(t)
    h = host.load(t)
    for item in ({"cap": (lo - 1, 0, 0), "policy": LEAF},
                 {"cap": (lo, 0, 0), "policy": LEAF, "mode": tg.MODE_EXCLUSIVE_DEMOTE},
                 {"cap": (lo, 0, 0), "policy": LEAF, "ttl": 5.0}):
        with pytest.raises(K.KvError) as e:
            host.evaluate(h, tg.from_list([item]), tg.DEFAULT_COST, 1)
        assert e.value.status == K.KV_ERR_UNSUPPORTED, item
    counts, _ = host.evaluate(h, tg.from_list([{"cap": (lo, 0, 0), "policy": LEAF}]),
                              tg.DEFAULT_COST, 1)
    h.free()
    assert counts[0, 0, 0, 0] > 0


def test_refuses_a_trace_beyond_half_the_position_limit():
    """The augmented order has 2N positions; above 2^28 accesses the call is
    refused before anything is built (the trace itself loads: N <= 2^29)."""
    import torch
    from paper_2603_08739_amd import host, kvcfg as K
    n = (1 << 28) + 64
    say(f"  loading {n} cold accesses")
    hsh = torch.arange(1, n + 1, dtype=torch.int64, device="cuda") * 0x9E3779B97F4A7C15
    req = (torch.arange(n, dtype=torch.int64, device="cuda") // 64).to(torch.int32)
    n_req = int(req[-1].item()) + 1
    rt = torch.arange(n_req, dtype=torch.float64, device="cuda")
    h = K.kv_trace_load(hsh, req, rt, n_groups=1, tokens_per_granule=16, granule_bytes=131072)
    del hsh, req, rt
    counts = torch.zeros((1, 1, 3, 8), dtype=torch.int64, device="cuda")
    arr, n_cfg = host.config_array(tg.from_list([{"cap": (1024, 0, 0), "policy": LEAF}]))
    with pytest.raises(K.KvError) as e:
        K.kv_eval_configs(h, arr, n_cfg, host.cost_model(tg.DEFAULT_COST), counts, None)
    assert e.value.status == K.KV_ERR_UNSUPPORTED and "2N positions" in str(e.value)
    h.free()
    torch.cuda.empty_cache()


def test_refuses_a_total_weight_of_2_31():
    """The augmented order carries every access's weight twice, and its sums
    are 32-bit: a trace of 2^31 granules or more is refused."""
    import torch
    from paper_2603_08739_amd import host, kvcfg as K
    n = (1 << 31) // 255 + 64
    hsh = torch.arange(1, n + 1, dtype=torch.int64, device="cuda") * 0x9E3779B97F4A7C15
    req = (torch.arange(n, dtype=torch.int64, device="cuda") // 64).to(torch.int32)
    rt = torch.arange(int(req[-1].item()) + 1, dtype=torch.float64, device="cuda")
    w = torch.full((n,), 255, dtype=torch.uint8, device="cuda")
    h = K.kv_trace_load(hsh, req, rt, weight=w, n_groups=1, tokens_per_granule=16,
                        granule_bytes=131072)
    counts = torch.zeros((1, 1, 3, 8), dtype=torch.int64, device="cuda")
    arr, n_cfg = host.config_array(tg.from_list([{"cap": (1 << 20, 0, 0), "policy": LEAF}]))
    with pytest.raises(K.KvError) as e:
        K.kv_eval_configs(h, arr, n_cfg, host.cost_model(tg.DEFAULT_COST), counts, None)
    assert e.value.status == K.KV_ERR_UNSUPPORTED and "2^31" in str(e.value)
    h.free()
