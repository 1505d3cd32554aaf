"""Group TTL (Alg. 2, Section 4.3) end to end on the device against the
oracle: subtree groups, TTL curves from kv_ttl_curves, allocation; the same
pipeline on the oracle's curves must give the same ROI TTLs and scaling and
the same hits (1e-6 relative) within the budget."""
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("k", [3, 7])
def test_group_ttl_matches_oracle(oracle_mod, k):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from oracle import group_ttl as A
    from paper_2603_08739_amd import group_ttl as P
    from paper_2603_08739_amd import host
    t = tg.tiny(n_req=1500)
    starts = np.r_[0, np.nonzero(np.diff(t.req))[0] + 1]
    counts = np.diff(np.r_[starts, t.n])
    g_req, _ = P.subtree_groups(t.hash[starts], k)
    t.group = np.repeat(g_req, counts).astype(np.uint8)
    t.n_groups = k + 1
    ttl = [0.0] + [float(x) for x in np.geomspace(0.05, 100.0, 40)]
    say(f"  group ttl: n={t.n} groups={t.n_groups}")
    h = host.load(t)
    hits, hitw, store = host.ttl_curves(h, ttl, t.n_groups)
    h.free()
    rh, _, rs = oracle_mod.ttl_curves(t, ttl)
    np.testing.assert_array_equal(hits, rh)
    budget = 0.2 * float(rs[:, -1].sum())
    a = P.allocate(hits, store, ttl, budget)
    b = A.allocate(rh, rs, ttl, budget)
    np.testing.assert_array_equal(a["t_roi"], b["t_roi"])
    np.testing.assert_allclose(a["t_init"], b["t_init"], rtol=1e-9)
    assert a["hits"] == pytest.approx(b["hits"], rel=1e-6)
    assert a["cost"] <= budget * (1 + 1e-9)
    _, hu = A.best_uniform(rh, rs, ttl, budget)
    say(f"  group ttl: {a['hits']:.0f} hits against {hu:.0f} with one TTL")
    assert a["hits"] >= hu * (1 - 1e-6)
