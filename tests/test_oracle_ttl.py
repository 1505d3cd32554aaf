"""Pins of the oracle's TTL retention curves (Section 4.3: cumulative hits
H_g(t) and storage cost C_g(t) of a group under a time-to-live t) against
things it does not compute itself: curves worked by hand from the
definitions, a disk tier simulated second by second, and closed forms."""
import json
import os

import numpy as np
import pytest

import tracegen as tg

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "ttl_hand.json")


def hand_trace(gold, case):
    lab = {"A": 0, "B": 1}
    t = tg.from_blocks([lab[b] for b in gold["blocks"]],
                       weights={lab[k]: v for k, v in case["weight"].items()},
                       groups={lab[k]: v for k, v in case["group"].items()},
                       n_groups=case["n_groups"])
    t.req = np.asarray(gold["req"], dtype=np.uint32)
    t.req_time = np.asarray(gold["req_time"], dtype=np.float64)
    return t


@pytest.mark.parametrize("name", ["unit", "weighted", "two groups"])
def test_hand_worked_curves(oracle_mod, name):
    gold = json.load(open(GOLD))
    case = [c for c in gold["cases"] if c["name"] == name][0]
    hits, hitw, store = oracle_mod.ttl_curves(hand_trace(gold, case), gold["ttl"])
    assert hits.tolist() == case["hits"]
    assert hitw.tolist() == case["hitw"]
    assert store.tolist() == [[float(x) for x in row] for row in case["store"]]


def stepped_tier(trace, ttl):
    """A disk tier run second by second over integer request times: the
    accesses of a second are served in order, a hit when the block's latest
    access lies at most t seconds back; then every block whose latest access
    is under t seconds old occupies its weight for the coming second."""
    G = trace.n_groups
    times = trace.req_time.astype(np.int64)
    horizon = int(times.max()) + int(max(ttl)) + 2
    by_sec = {}
    for i in range(trace.n):
        by_sec.setdefault(int(times[trace.req[i]]), []).append(i)
    hits = np.zeros((G, len(ttl)), dtype=np.uint64)
    hitw = np.zeros((G, len(ttl)), dtype=np.uint64)
    store = np.zeros((G, len(ttl)), dtype=np.float64)
    for k, t in enumerate(int(x) for x in ttl):
        last, wgt, grp = {}, {}, {}
        for sec in range(horizon):
            for i in by_sec.get(sec, ()):
                b = int(trace.hash[i])
                g, w = int(trace.group[i]), int(trace.weight[i])
                if b in last and sec - last[b] <= t:
                    hits[g, k] += 1
                    hitw[g, k] += w
                last[b], wgt[b], grp[b] = sec, w, g
            for b, a in last.items():
                if sec < a + t:
                    store[grp[b], k] += wgt[b]
    return hits, hitw, store


def small_integer_trace(seed):
    rng = np.random.default_rng(seed)
    n_req = int(rng.integers(5, 30))
    blocks = []
    for _ in range(n_req):
        blocks.append(rng.integers(0, 10, int(rng.integers(1, 4))).tolist())
    flat = [b for r in blocks for b in r]
    t = tg.from_blocks(flat, weights=rng.integers(1, 4, 10), groups=rng.integers(0, 3, 10),
                       n_groups=3)
    t.req = np.repeat(np.arange(n_req, dtype=np.uint32), [len(r) for r in blocks])
    t.req_time = np.cumsum(rng.integers(0, 6, n_req)).astype(np.float64)
    return t


@pytest.mark.parametrize("seed", range(12))
def test_matches_a_tier_simulated_second_by_second(oracle_mod, seed):
    t = small_integer_trace(seed)
    ttl = [0, 1, 2, 3, 5, 8, 13, 40]
    got = oracle_mod.ttl_curves(t, ttl)
    want = stepped_tier(t, ttl)
    for a, b in zip(got, want):
        np.testing.assert_array_equal(a, b)


def test_closed_forms(oracle_mod):
    """t = 0 stores nothing; a TTL above every gap keeps every re-access, and
    the gaps of a block add up to its last minus its first access time."""
    t = tg.random_trace(5, 4000, 600, n_groups=3, weight_choices=(1, 2, 4), zipf_s=0.8)
    big = float(t.req_time[-1] - t.req_time[0]) + 1.0
    hits, hitw, store = oracle_mod.ttl_curves(t, [0.0, big])
    assert np.all(store[:, 0] == 0.0)
    times = t.req_time[t.req]
    for g in range(t.n_groups):
        sel = t.group == g
        h = t.hash[sel]
        uniq, first = np.unique(h, return_index=True)
        _, last_rev = np.unique(h[::-1], return_index=True)
        last = len(h) - 1 - last_rev
        w_b = t.weight[sel][first].astype(np.float64)
        tg_ = times[sel]
        assert hits[g, 1] == sel.sum() - len(uniq)
        assert hitw[g, 1] == int(t.weight[sel].astype(np.int64).sum() - w_b.sum())
        want = w_b.sum() * big + float((w_b * (tg_[last] - tg_[first])).sum())
        assert store[g, 1] == pytest.approx(want, rel=1e-12)
