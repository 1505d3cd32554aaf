"""Host logic of the group TTL (Alg. 2, Section 4.3) without a device: the
library-side grouping and allocation against the oracle's on the same
inputs."""
import numpy as np
import pytest

from oracle import group_ttl as A


def synthetic_curves(seed, G, m):
    rng = np.random.default_rng(seed)
    ttl = np.concatenate([[0.0], np.sort(rng.uniform(1, 1000, m))])
    gaps = rng.integers(100, 5000, G)
    hits = np.zeros((G, m + 1))
    store = np.zeros((G, m + 1))
    for g in range(G):
        d = rng.exponential(rng.uniform(20, 400), gaps[g])
        blocks = rng.integers(10, 200)
        for k, t in enumerate(ttl):
            hits[g, k] = (d <= t).sum()
            store[g, k] = blocks * t + np.minimum(t, d).sum()
    return ttl, hits, store


@pytest.mark.parametrize("seed", range(4))
def test_allocation_matches_oracle(seed):
    from paper_2603_08739_amd import group_ttl as P
    ttl, hits, store = synthetic_curves(seed, 2 + seed, 24)
    budget = 0.3 * store[:, -1].sum()
    a = P.allocate(hits, store, ttl, budget, seed=seed)
    b = A.allocate(hits, store, ttl, budget, seed=seed)
    np.testing.assert_array_equal(a["t_roi"], b["t_roi"])
    assert a["alpha"] == pytest.approx(b["alpha"], rel=1e-12)
    np.testing.assert_allclose(a["t_init"], b["t_init"], rtol=1e-12)
    assert a["starts"] == b["starts"]
    assert a["hits"] == pytest.approx(b["hits"], rel=1e-6)
    assert a["cost"] <= budget * (1 + 1e-9)
    tu, hu = P.uniform_ttl(hits, store, ttl, budget)
    to, ho = A.best_uniform(hits, store, ttl, budget)
    assert tu == pytest.approx(to, rel=1e-12) and hu == pytest.approx(ho, rel=1e-12)
    assert a["hits"] >= hu * (1 - 1e-6)          # the group TTLs never lose to one TTL


def test_grouping_matches_oracle():
    from paper_2603_08739_amd import group_ttl as P
    rng = np.random.default_rng(9)
    first = rng.choice(np.array([3, 1, 4, 15, 9, 26, 5, 35], dtype=np.uint64), 500,
                       p=[0.3, 0.2, 0.15, 0.1, 0.1, 0.05, 0.05, 0.05])
    for k in (1, 3, 7, 8):
        ga, ra = P.subtree_groups(first, k)
        gb, rb = A.subtree_groups(first, k)
        assert ra == rb
        np.testing.assert_array_equal(ga, gb)
