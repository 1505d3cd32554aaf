"""Pins of the oracle's disk TTL tier (Section 4.1 planner: a disk TTL;
Section 4.3: a block stays on disk for the TTL after each access).

The oracle replays the tier literally (per-group recency lists, expiry
before each lookup, least-recent displacement when bounded).  It is held
here to things it does not compute that way:
* a disk tier simulated second by second on integer request times
  (hits, hit weights and the storage integral, per group);
* the gap definition: an access hits iff its block's previous access lies at
  most the TTL back, and the tier holds at the last request exactly the
  blocks accessed at most the TTL before it;
* for a bounded tier, a brute force over Mattson stack distances: present iff
  the stack distance fits the capacity and the gap fits the TTL;
* reductions: a TTL longer than the trace is plain LRU at the same capacity;
  a capacity above every distinct block is the unbounded tier;
* a hand-worked three-access case, and the objective's mean occupancy.
"""
import numpy as np
import pytest

import tracegen as tg
from tests import bruteforce as bf
from tests.test_oracle_ttl import small_integer_trace, stepped_tier

HIT, MISS, INS, EVICT, HIT_W, MISS_W, INS_W, EVICT_W = range(8)


def lone_ttl(ttl, cap=0, n_groups=1):
    return tg.from_list([{"cap": (0, 0, cap), "ttl": ttl}])


def gaps(trace):
    """Per access: the gap to the block's previous access (None if cold)."""
    times = trace.req_time[trace.req]
    last, out = {}, []
    for i in range(trace.n):
        h = int(trace.hash[i])
        out.append(times[i] - last[h] if h in last else None)
        last[h] = times[i]
    return out, last


def test_hand_case(oracle_mod):
    """A, B, A at times 0, 1, 5: the second A has a gap of 5."""
    t = tg.from_blocks([0, 1, 0])
    t.req_time = np.array([0.0, 1.0, 5.0])
    for ttl, hit, store in ((4.0, 0, 12.0), (5.0, 1, 15.0)):
        c = lone_ttl(ttl)
        r, st = oracle_mod.replay(t, c, with_store=True)
        assert r[0, 0, 2, HIT] == hit and r[0, 0, 2, MISS] == 3 - hit
        assert r[0, 0, 2, INS] == 3 - hit
        # at time 5 the tier holds A (just accessed) and B only if 5 - 1 <= ttl
        held = 1 + (1 if 4.0 <= ttl else 0)
        assert r[0, 0, 2, EVICT] == 3 - hit - held
        # A: ttl + min(ttl, 5); B: ttl
        assert st[0] == store


@pytest.mark.parametrize("seed", range(10))
def test_unbounded_matches_stepped_tier(oracle_mod, seed):
    t = small_integer_trace(seed)
    ttl_values = [0, 1, 2, 3, 5, 8, 13, 40]
    want_h, want_w, want_s = stepped_tier(t, ttl_values)
    for k, ttl in enumerate(ttl_values):
        for memo in (False, True):
            r, st = oracle_mod.replay(t, lone_ttl(float(ttl)), memo=memo, with_store=True)
            assert r[0, :, 2, HIT].tolist() == want_h[:, k].tolist()
            assert r[0, :, 2, HIT_W].tolist() == want_w[:, k].tolist()
            assert st[0] == pytest.approx(want_s[:, k].sum(), rel=1e-12)
    # per-group TTLs: each group's hits follow its own TTL
    per = [1.0, 5.0, 13.0]
    r, st = oracle_mod.replay(t, tg.from_list([{"cap": (0, 0, 0), "ttl": per}]), with_store=True)
    for g in range(3):
        k = ttl_values.index(int(per[g]))
        assert r[0, g, 2, HIT] == want_h[g, k]
    assert st[0] == pytest.approx(sum(want_s[g, ttl_values.index(int(per[g]))]
                                      for g in range(3)), rel=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_gap_definition_and_final_content(oracle_mod, seed):
    t = tg.random_trace(seed, 600, 80, n_groups=2, weight_choices=(1, 3), zipf_s=0.7)
    d, last = gaps(t)
    tend = float(t.req_time[-1])
    for ttl in (0.0, 0.7, 2.5, 9.0, 1e9):
        r = oracle_mod.replay(t, lone_ttl(ttl))
        for g in range(2):
            sel = t.group == g
            hit = sum(1 for i in np.nonzero(sel)[0] if d[i] is not None and d[i] <= ttl)
            assert r[0, g, 2, HIT] == hit
            assert r[0, g, 2, INS] == sel.sum() - hit
            blocks = {int(h) for h in t.hash[sel]}
            held = sum(1 for h in blocks if tend - last[h] <= ttl)
            assert r[0, g, 2, EVICT] == r[0, g, 2, INS] - held


@pytest.mark.parametrize("seed", range(8))
def test_bounded_is_stack_and_gap(oracle_mod, seed):
    t = tg.random_trace(seed + 50, 500, 60, weight_choices=(1, 4), zipf_s=0.6)
    labels = [int(x) for x in t.meta["labels"]]
    wl = {lab: int(w) for lab, w in zip(labels, t.weight)}
    D = bf.stack_distances(labels, wl)
    d, _ = gaps(t)
    for cap in (4, 17, 60, 300):
        for ttl in (0.5, 3.0, 20.0):
            r = oracle_mod.replay(t, lone_ttl(ttl, cap))
            want = sum(1 for i in range(t.n) if d[i] is not None and d[i] <= ttl and D[i] <= cap)
            assert r[0, 0, 2, HIT] == want
            assert r[0, 0, 2, INS] == t.n - want


def test_reductions(oracle_mod):
    t = tg.random_trace(77, 2000, 150, n_groups=2, weight_choices=(1, 2), zipf_s=0.8,
                        reuse_bias=0.2)
    span = float(t.req_time[-1] - t.req_time[0])
    for caps in ((0, 0, 40), (10, 0, 40), (0, 25, 90), (8, 30, 30)):
        long_ttl = tg.from_list([{"cap": caps, "ttl": span + 1.0}])
        plain = tg.from_list([{"cap": caps}])
        assert np.array_equal(oracle_mod.replay(t, long_ttl), oracle_mod.replay(t, plain))
    big = int(t.weight.astype(np.int64).sum())
    for ttl in (0.0, 1.5, 7.0):
        for up in ((0, 0), (6, 0), (6, 20)):
            a = oracle_mod.replay(t, tg.from_list([{"cap": (*up, big), "ttl": ttl}]))
            b = oracle_mod.replay(t, tg.from_list([{"cap": (*up, 0), "ttl": ttl}]))
            assert np.array_equal(a, b)


def test_inclusive_served_by_disk(oracle_mod):
    """With LRU tiers above it, the disk serves exactly the accesses that miss
    both and find the block within the TTL."""
    t = tg.random_trace(91, 1500, 120, zipf_s=0.8)
    labels = [int(x) for x in t.meta["labels"]]
    D = bf.stack_distances(labels, {lab: 1 for lab in labels})
    d, _ = gaps(t)
    for c0, c1, ttl in ((5, 0, 2.0), (5, 20, 6.0), (0, 12, 30.0)):
        r = oracle_mod.replay(t, tg.from_list([{"cap": (c0, c1, 0), "ttl": ttl}]))[0, 0]
        m1 = max(c0, c1)
        served = sum(1 for i in range(t.n) if D[i] > m1 and d[i] is not None and d[i] <= ttl)
        assert r[2, HIT] == served
        assert r[2, MISS] == sum(1 for i in range(t.n) if D[i] > m1) - served


def test_rejected(oracle_mod):
    t = tg.random_trace(3, 200, 30, n_groups=2)
    bad = [({"cap": (4, 0, 0), "ttl": 5.0, "policy": tg.POLICY_FIFO}, -4),
           ({"cap": (4, 0, 0), "ttl": 5.0, "mode": tg.MODE_EXCLUSIVE_DEMOTE}, -4),
           ({"cap": (4, 0, 10), "ttl": [1.0, 2.0]}, -4),
           ({"cap": (4, 0, 0), "ttl": -1.0}, -1)]
    for item, code in bad:
        with pytest.raises(ValueError, match=f"code {code}"):
            oracle_mod.replay(t, tg.from_list([item]))


def test_mean_occupancy_objective(oracle_mod):
    """An unbounded TTL tier is billed at its mean occupancy over the span:
    the same objectives as a capacity tier of that (fractional) size."""
    t = tg.from_blocks([0, 1, 0, 2, 0])
    t.req_time = np.array([0.0, 1.0, 2.0, 3.0, 4.0])
    cost = dict(tg.DEFAULT_COST)
    c = tg.from_list([{"cap": (1, 0, 0), "ttl": 2.0}])
    r, st = oracle_mod.replay(t, c, with_store=True)
    # A: 2 + 2 + 2 (gaps 2, 2); B: 2; C: 2  -> 10 granule-seconds over 4 s
    assert st[0] == 10.0
    obj = oracle_mod.objectives(t, c, r, cost, store=st)
    gib = 10.0 * t.granule_bytes / 2**30 / 4.0
    p = cost["price_per_gib_hour"]
    bw = min(cost["ssd_bw_base"] + cost["ssd_bw_per_gib"] * gib, cost["ssd_bw_max"])
    hw = r[0, 0, :, HIT_W].astype(np.int64)
    t_ssd = (hw[2] + r[0, 0, 2, INS_W]) * t.granule_bytes / bw
    t_rec = (5 - hw.sum()) * t.tokens_per_granule * cost["t_prefill_per_token"]
    busy = t_rec + t_ssd
    wall = max(4.0, busy)
    want_cost = (cost["price_gpu_per_hour"] + t.granule_bytes / 2**30 * p[0] + gib * p[2]) * wall / 3600
    assert obj[0, 0] == pytest.approx(want_cost, rel=1e-12)
    assert obj[0, 2] == pytest.approx(busy / 5, rel=1e-12)
    # and omitting the store replays it
    assert np.array_equal(oracle_mod.objectives(t, c, r, cost), obj)
