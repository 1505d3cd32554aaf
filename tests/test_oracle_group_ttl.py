"""Pins of the oracle-side ROI-aware group TTL (Alg. 2, Section 4.3): the
top-K subtree grouping, the ROI-optimal TTLs and the budget scaling worked
by hand, and the optimiser against a linear case whose optimum follows from
marginal hits per unit of storage."""
import numpy as np
import pytest

from oracle import group_ttl as A


def test_subtree_grouping_by_hand():
    first = np.array([5, 7, 5, 9, 7, 5, 11], dtype=np.uint64)
    g, roots = A.subtree_groups(first, 2)
    assert roots == [5, 7] and g.tolist() == [0, 1, 0, 2, 1, 0, 2]
    g, roots = A.subtree_groups(first, 3)          # a tie of 9 and 11: the smaller hash
    assert roots == [5, 7, 9] and g.tolist() == [0, 1, 0, 2, 1, 0, 3]


def test_roi_and_budget_scaling_by_hand():
    ttl = [0.0, 10.0, 20.0, 40.0]
    hits = [[0, 10, 12, 13], [0, 1, 8, 9]]
    store = [[0, 100, 200, 400], [0, 50, 100, 200]]
    # ROI: group 0 peaks at t = 10 (0.1), group 1 at t = 20 (0.08);
    # unscaled cost 100 + 100 = 200, budget 100: alpha = 1/2
    r = A.allocate(hits, store, ttl, 100.0)
    assert r["t_roi"].tolist() == [10.0, 20.0]
    assert r["alpha"] == 0.5 and r["t_init"].tolist() == [5.0, 10.0]
    assert r["starts"] == 3
    assert r["cost"] <= 100.0 * (1 + 1e-9)


def test_linear_case_optimum():
    # group 1 yields 0.2 hits per unit of storage, group 0 0.1: the budget of
    # 500 first fills group 1 up to t = 100 (cost 250, 50 hits), the rest
    # buys group 0 up to t = 25 (25 hits)
    ttl = [0.0, 100.0]
    hits = [[0.0, 100.0], [0.0, 50.0]]
    store = [[0.0, 1000.0], [0.0, 250.0]]
    r = A.allocate(hits, store, ttl, 500.0)
    assert r["hits"] == pytest.approx(75.0, rel=1e-4)
    assert r["t"][0] == pytest.approx(25.0, abs=0.05) and r["t"][1] == pytest.approx(100.0, abs=0.05)
    # one TTL for both: 12.5 t <= 500 -> t = 40, 60 hits
    t, h = A.best_uniform(hits, store, ttl, 500.0)
    assert t == pytest.approx(40.0, abs=1e-9) and h == pytest.approx(60.0, abs=1e-9)
