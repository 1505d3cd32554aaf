"""Pins the CPU oracle to facts other than itself (no GPU needed).

Textbook worked examples, hand cases, Mattson's stack-distance definition,
closed forms, reductions (inclusive LRU to single-cache LRU, exclusive
demotion to one LRU of the summed capacity) and invariants.  A plausible
mistake in the oracle (a wrong victim, a dropped count, a swapped tier or a
missed eviction) fails at least one of these.
"""
import itertools
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import tracegen as tg
from tests import bruteforce as bf

GOLD = os.path.join(os.path.dirname(__file__), "golden")
POL = {"LRU": tg.POLICY_LRU, "FIFO": tg.POLICY_FIFO, "LFU": tg.POLICY_LFU}


def single(O, labels, cap, policy, weights=None):
    t = tg.from_blocks(labels, weights=weights)
    c = tg.from_list([{"cap": (cap, 0, 0), "policy": policy}])
    return O.replay(t, c)[0, 0, 0]


def test_belady_string(oracle_mod):
    lines = [l.split() for l in open(os.path.join(GOLD, "belady.txt"))
             if l.strip() and not l.startswith("#")]
    s = [int(x) for x in lines[0][1:]]
    for pol, cap, misses in lines[1:]:
        r = single(oracle_mod, s, int(cap), POL[pol])
        assert r[oracle_mod.MISS] == int(misses), (pol, cap)
        assert r[oracle_mod.HIT] + r[oracle_mod.MISS] == len(s)


def test_hand_cases(oracle_mod):
    for line in open(os.path.join(GOLD, "hand_cases.txt")):
        if not line.strip() or line.startswith("#"):
            continue
        pol, cap, string, misses, ev = line.split()
        labels = [ord(c) for c in string]
        r = single(oracle_mod, labels, int(cap), POL[pol])
        assert r[oracle_mod.MISS] == int(misses), line
        assert r[oracle_mod.EVICT] == int(ev), line


labels_st = st.lists(st.integers(0, 9), min_size=1, max_size=60)
weights_st = st.lists(st.sampled_from([1, 4]), min_size=10, max_size=10)


@settings(max_examples=150, deadline=None)
@given(labels=labels_st, weights=weights_st, cap=st.integers(4, 30))
def test_lru_matches_stack_distance(oracle_mod, labels, weights, cap):
    wd = {b: weights[b] for b in range(10)}
    r = single(oracle_mod, labels, cap, tg.POLICY_LRU, weights=np.array(weights))
    assert r[oracle_mod.HIT] == bf.lru_hits(labels, wd, cap)
    # evictions = insertions - final residents (maximal recency prefix)
    fin = bf.lru_final_resident(labels, wd, cap)
    assert r[oracle_mod.INS] == r[oracle_mod.MISS]
    assert r[oracle_mod.EVICT] == r[oracle_mod.INS] - len(fin)
    assert r[oracle_mod.EVICT_W] == r[oracle_mod.INS_W] - sum(wd[b] for b in fin)


@settings(max_examples=150, deadline=None)
@given(labels=labels_st, weights=weights_st, cap=st.integers(4, 30))
def test_fifo_matches_suffix_rule(oracle_mod, labels, weights, cap):
    wd = {b: weights[b] for b in range(10)}
    r = single(oracle_mod, labels, cap, tg.POLICY_FIFO, weights=np.array(weights))
    assert r[oracle_mod.HIT] == bf.fifo_hits_suffix(labels, wd, cap)


@settings(max_examples=150, deadline=None)
@given(labels=labels_st, weights=weights_st, cap=st.integers(4, 30))
def test_lfu_matches_scan(oracle_mod, labels, weights, cap):
    wd = {b: weights[b] for b in range(10)}
    r = single(oracle_mod, labels, cap, tg.POLICY_LFU, weights=np.array(weights))
    hits, ev = bf.lfu_scan(labels, wd, cap)
    assert r[oracle_mod.HIT] == hits
    assert r[oracle_mod.EVICT] == ev


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_closed_forms(oracle_mod, policy):
    O = oracle_mod
    t = tg.random_trace(5, 3000, 200, weight_choices=(1, 4), zipf_s=0.8)
    u = len(np.unique(t.hash))
    wsum = int(t.weight[np.unique(t.hash, return_index=True)[1]].astype(int).sum())
    # capacity covering every distinct block: only cold misses, no evictions
    c = tg.from_list([{"cap": (wsum, 0, 0), "policy": policy},
                      {"cap": (0, 0, 0), "policy": policy}])
    r = O.replay(t, c)
    assert r[0, 0, 0, O.HIT] == t.n - u and r[0, 0, 0, O.EVICT] == 0
    assert r[1].sum() == 0  # every tier absent: nothing recorded
    # one-block cache (unit weights): hit iff the previous access was the same block
    tu = tg.random_trace(6, 2000, 6, reuse_bias=0.5)
    rr = O.replay(tu, tg.from_list([{"cap": (1, 0, 0), "policy": policy}]))
    assert rr[0, 0, 0, O.HIT] == int((tu.hash[1:] == tu.hash[:-1]).sum())


def test_lru_monotone_in_capacity(oracle_mod):
    O = oracle_mod
    t = tg.random_trace(11, 5000, 400, weight_choices=(1, 4), zipf_s=0.9)
    caps = list(range(4, 1800, 37))
    c = tg.from_list([{"cap": (x, 0, 0)} for x in caps])
    h = O.replay(t, c)[:, 0, 0, O.HIT]
    assert np.all(np.diff(h.astype(np.int64)) >= 0)


def test_inclusive_lru_reduces_to_single_caches(oracle_mod):
    O = oracle_mod
    t = tg.random_trace(12, 4000, 300, weight_choices=(1, 4), zipf_s=0.7)
    caps = [0, 8, 40, 120, 400]
    combos = [c for c in itertools.product(caps, caps, caps) if any(c)]
    batch = tg.from_list([{"cap": c} for c in combos])
    r = O.replay(t, batch)[:, 0]
    single_hits = {x: O.replay(t, tg.from_list([{"cap": (x, 0, 0)}]))[0, 0, 0, O.HIT]
                   if x else 0 for x in caps}
    for i, c in enumerate(combos):
        m = 0
        for k in range(3):
            if c[k] == 0:
                assert r[i, k].sum() == 0
                continue
            want = max(0, int(single_hits[c[k]]) - int(single_hits[m]))
            assert r[i, k, O.HIT] == want, (c, k)
            m = max(m, c[k])
        # every access is served once or recomputed
        last = max(k for k in range(3) if c[k])
        assert r[i, :, O.HIT].sum() + r[i, last, O.MISS] == t.n
        live = [k for k in range(3) if c[k]]
        ms = [int(r[i, k, O.MISS]) for k in live]
        assert all(a >= b for a, b in zip(ms, ms[1:]))


@settings(max_examples=100, deadline=None)
@given(labels=st.lists(st.integers(0, 14), min_size=1, max_size=80),
       caps=st.tuples(st.integers(0, 6), st.integers(0, 6), st.integers(0, 6)))
def test_exclusive_split_stack(oracle_mod, labels, caps):
    """Exclusive demotion = one LRU stack cut at the cumulative capacities."""
    O = oracle_mod
    if not any(caps):
        return
    t = tg.from_blocks(labels)
    r = O.replay(t, tg.from_list([{"cap": caps, "mode": tg.MODE_EXCLUSIVE_DEMOTE}]))[0, 0]
    d = bf.unit_stack_distances(labels)
    u = len(set(labels))
    s_prev = 0
    live = [k for k in range(3) if caps[k]]
    for k in range(3):
        if caps[k] == 0:
            assert r[k].sum() == 0
            continue
        s_k = s_prev + caps[k]
        assert r[k, O.HIT] == sum(1 for x in d if s_prev < x <= s_k)
        assert r[k, O.MISS] == sum(1 for x in d if x > s_k)
        want_ev = sum(1 for x in d if x != bf.INF and x > s_k) + max(0, u - s_k)
        assert r[k, O.EVICT] == want_ev
        s_prev = s_k
    top = live[0]
    assert r[top, O.INS] == len(labels) - r[top, O.HIT]
    for a, b in zip(live, live[1:]):
        assert r[b, O.INS] == r[a, O.EVICT]
    # sum of hits = single LRU at the summed capacity; top hits = LRU at top capacity
    assert r[:, O.HIT].sum() == sum(1 for x in d if x <= sum(caps))
    assert r[top, O.HIT] == sum(1 for x in d if x <= caps[top])


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_partitioned_is_per_group_sum(oracle_mod, policy):
    """A partitioned configuration replays each group's sub-trace on its own."""
    O = oracle_mod
    t = tg.random_trace(21, 3000, 250, n_groups=3, weight_choices=(1, 4), zipf_s=0.6)
    cg = np.array([[40, 17, 90], [0, 60, 200], [300, 0, 8]], dtype=np.uint64)
    pol = [policy, (policy + 1) % 3, (policy + 2) % 3]
    c = tg.from_list([{"cap": tuple(cg.sum(1)), "cap_group": cg, "partitioned": 1,
                       "policy": pol}])
    r = O.replay(t, c)[0]
    for g in range(3):
        m = t.group == g
        sub = tg.Trace("sub", t.hash[m], t.req[m], np.zeros(m.sum(), np.uint8), t.weight[m],
                       t.req_time, 1)
        rs = O.replay(sub, tg.from_list([{"cap": tuple(cg[:, g]), "policy": pol[g]}]))[0, 0]
        np.testing.assert_array_equal(r[g], rs)


def test_shared_group_attribution(oracle_mod):
    """Shared cache on a multi-group trace: per-group counts add up to the total."""
    O = oracle_mod
    t = tg.random_trace(22, 3000, 250, n_groups=4, weight_choices=(1, 4), zipf_s=0.6)
    c = tg.from_list([{"cap": (30, 100, 400), "policy": p} for p in range(3)])
    r = O.replay(t, c)
    t1 = tg.Trace("one", t.hash, t.req, np.zeros(t.n, np.uint8), t.weight, t.req_time, 1)
    r1 = O.replay(t1, c)
    np.testing.assert_array_equal(r.sum(axis=1), r1[:, 0])
    for g in range(4):
        n_g = int((t.group == g).sum())
        live_last = r[:, g, 2, O.MISS]
        assert np.all(r[:, g, :, O.HIT].sum(1) + live_last == n_g)


def test_invalid_capacity_rejected(oracle_mod):
    t = tg.from_blocks([1, 2, 3], weights={1: 4, 2: 4, 3: 4})
    with pytest.raises(ValueError):
        oracle_mod.replay(t, tg.from_list([{"cap": (3, 0, 0)}]))
    with pytest.raises(ValueError):   # prefix reuse is defined for LRU only
        oracle_mod.replay(tg.from_blocks([1, 2]),
                          tg.from_list([{"cap": (3, 0, 0), "mode": 2, "policy": 1}]))
