"""Input generators: determinism and structural properties (no GPU needed)."""
import numpy as np

import tracegen as tg


def _check_structure(t):
    assert t.hash.dtype == np.uint64 and t.req.dtype == np.uint32
    assert np.all(np.diff(t.req.astype(np.int64)) >= 0)
    assert np.all(np.diff(t.req_time) >= 0)
    assert int(t.req.max()) < t.n_req
    # each block hash has one weight and one group
    _, first, inv = np.unique(t.hash, return_index=True, return_inverse=True)
    assert np.array_equal(t.weight, t.weight[first][inv])
    assert np.array_equal(t.group, t.group[first][inv])


def test_tiny_deterministic_and_shaped():
    a = tg.tiny()
    b = tg.tiny()
    assert np.array_equal(a.hash, b.hash) and np.array_equal(a.req_time, b.req_time)
    assert a.n_req == 2000 and 150_000 < a.n < 400_000
    _check_structure(a)
    # shared prefixes: the first block of a popular prompt is reused many times
    _, counts = np.unique(a.hash, return_counts=True)
    assert counts.max() > 100


def test_small_variants_structure():
    for t in (tg.chat(n_sessions=300), tg.tenant(total_req=2000),
              tg.longctx(n_req=300, n_docs=50), tg.full(n_req=3000)):
        _check_structure(t)
        assert t.n > 0
    t = tg.tenant(total_req=2000)
    assert t.n_groups == 8 and set(np.unique(t.group)) <= set(range(8))
    f = tg.full(n_req=3000)
    assert set(np.unique(f.weight)) == {1, 4}


def test_config_grids():
    t = tg.tiny(n_req=10)
    assert tg.configs_for("tiny", t).n == 64
    assert tg.configs_for("chat", t).n == 512
    tt = tg.tenant(total_req=200)
    c3 = tg.configs_for("tenant", tt)
    assert c3.n == 1000 and np.all(c3.partitioned == 1)
    assert np.all(c3.cap_group.sum(axis=2) == c3.cap)
    c4 = tg.configs_for("longctx", tg.longctx(n_req=5, n_docs=5))
    assert c4.n == 2048 and np.all(c4.mode == tg.MODE_EXCLUSIVE_DEMOTE)
    c5 = tg.configs_for("full", t)
    assert c5.n == 11000
    assert np.array_equal(np.bincount(c5.policy[:, 0]), [10000, 500, 500])
