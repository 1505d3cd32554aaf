"""Pins for the oracle's objective proxy and Pareto filter (no GPU needed)."""
import json
import os

import numpy as np
from hypothesis import given, settings, strategies as st

import tracegen as tg

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _fake_trace(n_w, n_req, span, gb, tpg):
    t = tg.from_blocks(np.arange(n_w) % 97)
    t.req_time = np.linspace(0.0, span, n_req)
    t.granule_bytes = gb
    t.tokens_per_granule = tpg
    return t


def test_objective_worked_examples(oracle_mod):
    O = oracle_mod
    spec = json.load(open(os.path.join(GOLD, "objective_cases.json")))
    for case in spec["cases"]:
        t = _fake_trace(spec["n_w"], spec["n_req"], case["span"], spec["granule_bytes"],
                        spec["tokens_per_granule"])
        c = tg.from_list([{"cap": case["cap"]}])
        counts = np.zeros((1, 1, 3, 8), np.uint64)
        counts[0, 0, :, O.HIT_W] = case["hit_w"]
        counts[0, 0, 2, O.INS_W] = case["ssd_ins_w"]
        obj = O.objectives(t, c, counts, spec["cost"])[0]
        np.testing.assert_allclose(obj, case["expect"], rtol=1e-13, err_msg=case["name"])


def test_objective_directions(oracle_mod):
    """More hits in faster tiers never raise latency; capacity prices add linearly."""
    O = oracle_mod
    t = tg.make("tiny", n_req=200)
    c = tg.from_list([{"cap": (8192, 0, 0)}, {"cap": (16384, 0, 0)},
                      {"cap": (16384, 8192 * 64, 0)}])
    r = O.replay(t, c)
    obj = O.objectives(t, c, r, tg.DEFAULT_COST)
    assert obj[1, 2] <= obj[0, 2] and obj[2, 2] <= obj[1, 2]
    assert np.all(obj[:, 1] > 0)


def dominates(a, b):
    return (a[0] <= b[0] and a[1] >= b[1] and a[2] <= b[2]
            and (a[0] < b[0] or a[1] > b[1] or a[2] < b[2]))


objs_st = st.lists(st.tuples(st.integers(0, 6), st.integers(0, 6), st.integers(0, 6)),
                   min_size=1, max_size=40)


@settings(max_examples=200, deadline=None)
@given(pts=objs_st, perm_seed=st.integers(0, 1000))
def test_pareto_properties(oracle_mod, pts, perm_seed):
    O = oracle_mod
    obj = np.array(pts, dtype=np.float64)
    f = O.pareto(obj).astype(bool)
    front = obj[f]
    # antichain: no member dominates another member
    for a in front:
        for b in front:
            assert not dominates(a, b)
    # every non-member is dominated by some member
    for b in obj[~f]:
        assert any(dominates(a, b) for a in front)
    # equal vectors are kept together
    for i in range(len(obj)):
        for j in range(len(obj)):
            if np.array_equal(obj[i], obj[j]):
                assert f[i] == f[j]
    # permutation invariance
    p = np.random.default_rng(perm_seed).permutation(len(obj))
    np.testing.assert_array_equal(O.pareto(obj[p]).astype(bool), f[p])


@settings(max_examples=100, deadline=None)
@given(pts=st.lists(st.integers(0, 20), min_size=1, max_size=30))
def test_pareto_one_objective_is_argmin(oracle_mod, pts):
    O = oracle_mod
    obj = np.zeros((len(pts), 3))
    obj[:, 0] = pts
    f = O.pareto(obj).astype(bool)
    np.testing.assert_array_equal(f, obj[:, 0] == obj[:, 0].min())


def skyline_2d(cost, thr):
    """Textbook 2-D staircase: sort by cost asc (thr desc), sweep the best thr."""
    order = sorted(range(len(cost)), key=lambda i: (cost[i], -thr[i]))
    keep = [False] * len(cost)
    best = -np.inf
    i = 0
    while i < len(order):
        j = i
        while j < len(order) and cost[order[j]] == cost[order[i]]:
            j += 1
        group = order[i:j]
        top = thr[group[0]]            # best thr at this cost
        if top > best:
            for g in group:
                keep[g] = thr[g] == top
            best = top
        i = j
    return np.array(keep)


@settings(max_examples=150, deadline=None)
@given(pts=st.lists(st.tuples(st.integers(0, 8), st.integers(0, 8)), min_size=1, max_size=40))
def test_pareto_two_objectives_staircase(oracle_mod, pts):
    O = oracle_mod
    obj = np.zeros((len(pts), 3))
    obj[:, 0] = [p[0] for p in pts]
    obj[:, 1] = [p[1] for p in pts]
    f = O.pareto(obj).astype(bool)
    np.testing.assert_array_equal(f, skyline_2d(list(obj[:, 0]), list(obj[:, 1])))


@settings(max_examples=100, deadline=None)
@given(pts=objs_st, seg=st.lists(st.integers(0, 2), min_size=40, max_size=40),
       b=st.tuples(st.integers(0, 6), st.integers(0, 6), st.integers(0, 6)))
def test_pareto_segments_and_bounds(oracle_mod, pts, seg, b):
    """Segments are independent problems; bounds filter before or after alike."""
    O = oracle_mod
    obj = np.array(pts, dtype=np.float64)
    sg = np.array(seg[:len(pts)], dtype=np.uint32)
    f = O.pareto(obj, sg).astype(bool)
    for s in np.unique(sg):
        m = sg == s
        np.testing.assert_array_equal(f[m], O.pareto(obj[m]).astype(bool))
    bounds = np.array([b[0], b[1], np.nan])
    fb = O.pareto(obj, None, bounds).astype(bool)
    feas = (obj[:, 0] <= b[0]) & (obj[:, 1] >= b[1])
    want = np.zeros(len(obj), bool)
    if feas.any():
        want[feas] = O.pareto(obj[feas]).astype(bool)
    np.testing.assert_array_equal(fb, want)
    # filtering after dominance gives the same set (bounds are monotone)
    np.testing.assert_array_equal(fb, O.pareto(obj).astype(bool) & feas)
