"""GPU parity of exclusive (write-back demotion) hierarchies that are no
split stack: FIFO and LFU tiers, and LRU tiers over blocks of mixed weights,
replayed access by access on the device.  Counts are compared with the
oracle element by element, objectives to 1e-6.

* the hand-worked two-tier cases the oracle is pinned to;
* random traces (one to three groups, unit and mixed weights) with shared
  and partitioned configurations, group policies mixed within one
  configuration (an LRU group over unit weights keeps its split stack), and
  small capacities that cascade demotions through every tier;
* batches mixing these with inclusive and split-stack configurations;
* workload-shaped slices (the mixed tenant and long-context traces, and
  the full workload's weighted blocks under exclusive LRU, FIFO and LFU);
* state buffers forced small, so that the configurations run in waves;
* an LFU trace that keeps more count buckets live than the walk holds in LDS.
"""
import os
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu

ALL = (tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU)
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def compare(O, t, cfgs, label, budget=None):
    from paper_2603_08739_amd import host
    say(f"  case {label}: n={t.n} groups={t.n_groups} configs={cfgs.n} budget={budget}")
    old = os.environ.get("KVCFG_TEST_REPLAY_BUDGET")
    if budget is not None:
        os.environ["KVCFG_TEST_REPLAY_BUDGET"] = str(budget)
    try:
        h = host.load(t)
        counts, obj = host.evaluate(h, cfgs, tg.DEFAULT_COST, t.n_groups)
        h.info()  # reports a failed state check of the call
        h.free()
    finally:
        if budget is not None:
            if old is None:
                os.environ.pop("KVCFG_TEST_REPLAY_BUDGET", None)
            else:
                os.environ["KVCFG_TEST_REPLAY_BUDGET"] = old
    ref = O.replay(t, cfgs)
    if not np.array_equal(counts, ref):
        bad = np.argwhere(counts != ref)
        c, g, k, f = bad[0]
        raise AssertionError(
            f"{label}: {len(bad)} mismatches; first cfg {c} group {g} tier {k} field {f}: "
            f"gpu {counts[c, g, k, f]} oracle {ref[c, g, k, f]} cap {cfgs.cap[c]} "
            f"mode {cfgs.mode[c]} policy {cfgs.policy[c, :t.n_groups]} part {cfgs.partitioned[c]}"
            f"\n gpu {counts[c, g]}\n ref {ref[c, g]}")
    np.testing.assert_allclose(obj, O.objectives(t, cfgs, ref, tg.DEFAULT_COST), rtol=1e-6,
                               atol=0, err_msg=label)
    return counts


def test_hand_cases(oracle_mod):
    pol = {"LRU": tg.POLICY_LRU, "FIFO": tg.POLICY_FIFO, "LFU": tg.POLICY_LFU}
    for line in open(os.path.join(GOLD, "exclusive_cases.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        p, caps, string, wts = line.split()[:4]
        weights = None
        if wts != "-":
            weights = {ord(k): int(v) for k, v in (x.split("=") for x in wts.split(","))}
        t = tg.from_blocks([ord(c) for c in string], weights=weights)
        c = tg.from_list([{"cap": tuple(int(x) for x in caps.split(",")), "policy": pol[p],
                           "mode": tg.MODE_EXCLUSIVE_DEMOTE}])
        compare(oracle_mod, t, c, f"hand-{p}-{string}")


@pytest.mark.parametrize("seed", range(9))
def test_random_traces(oracle_mod, seed):
    G = 1 + seed % 3
    wts = (1,) if seed % 3 == 0 else (1, 2, 4)
    t = tg.random_trace(700 + seed, 3000 + 500 * seed, 150 + 40 * seed, n_groups=G,
                        weight_choices=wts, zipf_s=0.6 + 0.05 * seed)
    cfgs = tg.random_configs(seed, 24, G, max(wts), [600, 16, 60][seed % 3], exclusive=True,
                             zero_frac=0.2, exclusive_policies=ALL)
    compare(oracle_mod, t, cfgs, f"random{seed}")


def test_mixed_batch(oracle_mod):
    """Replayed exclusive hierarchies beside inclusive ones (every policy),
    split-stack exclusive ones, and partitioned configurations whose groups
    take both paths."""
    t = tg.random_trace(801, 6000, 500, n_groups=3, weight_choices=(1,), zipf_s=0.8)
    parts = [tg.random_configs(1, 16, 3, 1, 300, exclusive=True, exclusive_policies=ALL),
             tg.random_configs(2, 16, 3, 1, 300),
             tg.random_configs(3, 8, 3, 1, 300, exclusive=True)]
    cfgs = tg.ConfigBatch.concat(parts)
    assert any(cfgs.partitioned[:16]) and any(cfgs.policy[:16, 0] != tg.POLICY_LRU)
    compare(oracle_mod, t, cfgs, "mixed-batch")


def test_workload_slices(oracle_mod):
    t = tg.tenant(total_req=2000)
    cfgs = tg.configs_for("tenant", t).subset(np.arange(0, 1000, 41))
    cfgs.cap //= 64
    cfgs.cap_group //= 64
    cfgs.mode[:] = tg.MODE_EXCLUSIVE_DEMOTE
    compare(oracle_mod, t, cfgs, "tenant-exclusive")
    t = tg.longctx(n_req=120, n_docs=40)
    base = tg.configs_for("longctx", t).subset(np.arange(0, 2048, 131))
    base.cap //= 256
    parts = []
    for p in (tg.POLICY_FIFO, tg.POLICY_LFU):
        c = base.subset(np.arange(base.n))
        c.policy[:, :] = p
        parts.append(c)
    compare(oracle_mod, t, tg.ConfigBatch.concat(parts), "longctx-exclusive")


def test_waves(oracle_mod):
    t = tg.random_trace(811, 5000, 700, n_groups=2, weight_choices=(1, 4), zipf_s=0.7)
    cfgs = tg.random_configs(11, 12, 2, 4, 400, exclusive=True, exclusive_policies=ALL)
    one = compare(oracle_mod, t, cfgs, "one-wave")
    for b in (40_000, 1):
        assert np.array_equal(one, compare(oracle_mod, t, cfgs, f"waves{b}", budget=b))


def test_full_slice_weighted(oracle_mod):
    """A slice of the full workload (16- and 64-token blocks, weights 1 and
    4) as exclusive LRU, FIFO and LFU hierarchies at scaled-down
    capacities: weighted LRU, no split stack, is replayed too."""
    t = tg.full(n_req=4000)
    cfgs = tg.configs_for("full", t)
    pick = np.concatenate([np.arange(0, 10000, 1667), np.arange(10000, 11000, 200)])
    sub = cfgs.subset(pick)
    sub.cap //= 16
    sub.cap[(sub.cap > 0) & (sub.cap < 4)] = 4
    sub.mode[:] = tg.MODE_EXCLUSIVE_DEMOTE
    assert set(sub.policy[:, 0]) == {tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU}
    compare(oracle_mod, t, sub, "full-slice-exclusive")


def test_lfu_many_counts(oracle_mod):
    """Block j of 2,200 accessed j + 1 times in shuffled order: a top tier
    that holds every block ends with 2,200 count buckets, more than the
    walk keeps in LDS, so bucket records in device memory are used too;
    smaller tiers cascade demotions across many buckets."""
    rng = np.random.default_rng(5)
    u = 2200
    labels = np.repeat(np.arange(u), np.arange(1, u + 1))
    rng.shuffle(labels)
    t = tg.from_blocks(labels, per_request=8)
    c = tg.from_list([{"cap": cap, "policy": tg.POLICY_LFU, "mode": tg.MODE_EXCLUSIVE_DEMOTE}
                      for cap in ((u, 0, 0), (1500, 400, 0), (2100, 50, 10), (600, 600, 600))])
    compare(oracle_mod, t, c, "lfu-many-counts")
