"""GPU parity of configurations with a disk TTL tier (Section 4.1 planner:
DRAM capacity x disk TTL x disk medium; Section 4.3 retention).

The library serves every (capacity, TTL) from joint histograms of (stack
distance, gap) per group; the oracle replays each tier literally.  Counts are
compared element by element, objectives to 1e-6 relative (the storage
integral of an unbounded tier is a double sum in different orders), Pareto
flags exactly.  Cases: unbounded and bounded tiers, per-group TTLs on shared
tiers, TTLs equal to gaps and zero, media, batches mixing TTL and capacity
disks with FIFO/LFU and exclusive configurations, the forced global-atomic
binning path, and the tiny workload on a DRAM x TTL grid.
"""
import os
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu

MEDIA = ((0.0002, 0.35e9, 0.5e6, 4.0e9), (0.0005, 1.0e9, 1.0e6, 8.0e9),
         (0.0012, 2.5e9, 2.0e6, 16.0e9))


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def compare(O, trace, cfgs, cost=tg.DEFAULT_COST, label=""):
    from paper_2603_08739_amd import host
    say(f"  case {label}: n={trace.n} groups={trace.n_groups} configs={cfgs.n}")
    h = host.load(trace)
    counts, obj = host.evaluate(h, cfgs, cost, trace.n_groups)
    h.free()
    ref, store = O.replay(trace, cfgs, memo=True, with_store=True)
    if not np.array_equal(counts, ref):
        bad = np.argwhere(counts != ref)
        c, g, k, f = bad[0]
        raise AssertionError(f"{label}: {len(bad)} mismatches; first cfg {c} group {g} tier {k} "
                             f"field {f}: gpu {counts[c, g, k, f]} oracle {ref[c, g, k, f]} "
                             f"cap {cfgs.cap[c]} ttl {cfgs.ttl[c, :trace.n_groups]}")
    ref_obj = O.objectives(trace, cfgs, ref, cost, store=store)
    np.testing.assert_allclose(obj, ref_obj, rtol=1e-6, atol=0, err_msg=label)
    # Pareto flags of the GPU objectives, against the brute force over the
    # same objectives (the two objective sets may differ in the last bits)
    flags, _ = host.pareto(obj, segment=cfgs.segment)
    assert np.array_equal(flags, O.pareto(obj, cfgs.segment))
    return counts


def ttl_batch(seed, trace, n, cap_hi, n_ttl=6, with_media=False):
    rng = np.random.default_rng([seed, 3])
    gaps = np.diff(trace.req_time)
    span = float(trace.req_time[-1] - trace.req_time[0])
    # TTL values: zero, exact request gaps, fractions of the span, beyond it
    pool = [0.0, float(gaps[gaps > 0][0]) if (gaps > 0).any() else 0.0,
            0.01 * span, 0.1 * span, 0.5 * span, 2.0 * span + 1.0]
    pool += [float(x) for x in rng.uniform(0, span, n_ttl)]
    items = []
    G = trace.n_groups
    w_max = int(trace.weight.max())
    for i in range(n):
        caps = [0 if rng.random() < 0.3 else int(rng.integers(w_max, cap_hi)) for _ in range(2)]
        bounded = rng.random() < 0.4
        c2 = int(rng.integers(w_max, 2 * cap_hi)) if bounded else 0
        if bounded:
            ttl = float(rng.choice(pool))
        else:
            ttl = [float(rng.choice(pool)) for _ in range(G)]
        it = {"cap": (caps[0], caps[1], c2), "ttl": ttl, "segment": i % 3}
        if with_media:
            it["medium"] = int(rng.integers(0, len(MEDIA)))
        items.append(it)
    return tg.from_list(items)


@pytest.mark.parametrize("seed", range(10))
def test_random_ttl_batches(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    groups = int(rng.choice([1, 2, 3]))
    weights = (1,) if seed % 2 else (1, 4)
    t = tg.random_trace(seed + 300, int(rng.integers(200, 6000)), int(rng.integers(20, 700)),
                        n_groups=groups, weight_choices=weights, zipf_s=0.8, reuse_bias=0.2)
    cfgs = ttl_batch(seed, t, 40, 400, with_media=seed % 3 == 0)
    cost = dict(tg.DEFAULT_COST)
    if seed % 3 == 0:
        cost["media"] = MEDIA
    compare(oracle_mod, t, cfgs, cost, label=f"ttl{seed}")


def test_mixed_batch(oracle_mod):
    t = tg.random_trace(401, 5000, 600, n_groups=2, weight_choices=(1,), zipf_s=0.9)
    ttl = ttl_batch(4, t, 30, 300)
    other = tg.random_configs(401, 30, 2, 1, 300)
    ex = tg.random_configs(402, 10, 2, 1, 300, exclusive=True)
    compare(oracle_mod, t, tg.ConfigBatch.concat([ttl, other, ex, ttl.subset([0, 1])]),
            label="mixed")


def test_global_binning_path(oracle_mod):
    t = tg.random_trace(411, 8000, 900, n_groups=2, weight_choices=(1, 4), zipf_s=0.8)
    cfgs = ttl_batch(11, t, 60, 900, n_ttl=40)
    old = os.environ.get("KVCFG_TEST_THR_LDS")
    os.environ["KVCFG_TEST_THR_LDS"] = "0"
    try:
        compare(oracle_mod, t, cfgs, label="ttl-global")
    finally:
        if old is None:
            os.environ.pop("KVCFG_TEST_THR_LDS")
        else:
            os.environ["KVCFG_TEST_THR_LDS"] = old


def test_many_ttl_values(oracle_mod):
    """More joint bins than the LDS holds (global path without a hook)."""
    t = tg.random_trace(421, 4000, 500, zipf_s=0.7)
    span = float(t.req_time[-1])
    items = [{"cap": (8 + i % 50, 0, 0), "ttl": span * i / 300.0} for i in range(300)]
    compare(oracle_mod, t, tg.from_list(items), label="300-ttls")


def test_tiny_workload_dram_ttl_grid(oracle_mod):
    t = tg.tiny()
    gib = (1 << 30) // t.granule_bytes
    items = [{"cap": (4 * gib, d * gib, 0), "ttl": ttl}
             for d in (0, 16, 64, 256) for ttl in (0.0, 1.0, 5.0, 20.0, 60.0, 1e6)]
    items += [{"cap": (4 * gib, d * gib, 512 * gib), "ttl": 5.0} for d in (0, 64)]
    compare(oracle_mod, t, tg.from_list(items), label="tiny-dram-ttl")


def test_rejected(oracle_mod):
    from paper_2603_08739_amd import host, kvcfg as K
    t = tg.random_trace(431, 300, 40, n_groups=2)
    h = host.load(t)
    bad = [({"cap": (4, 0, 0), "ttl": 5.0, "policy": tg.POLICY_LFU}, K.KV_ERR_UNSUPPORTED),
           ({"cap": (4, 0, 0), "ttl": 5.0, "mode": tg.MODE_INCLUSIVE_PREFIX}, K.KV_ERR_UNSUPPORTED),
           ({"cap": (4, 0, 9), "ttl": [1.0, 2.0]}, K.KV_ERR_UNSUPPORTED),
           ({"cap": (4, 0, 0), "ttl": -1.0}, K.KV_ERR_INVALID),
           ({"cap": (4, 0, 0), "ttl": float("nan")}, K.KV_ERR_INVALID),
           ({"cap": (4, 0, 0), "medium": 1}, K.KV_ERR_INVALID)]
    for item, code in bad:
        with pytest.raises(K.KvError) as e:
            host.evaluate(h, tg.from_list([item]), tg.DEFAULT_COST, 2)
        assert e.value.status == code, item
    h.free()
