"""Alg. 1 (adaptive Pareto exploration, Section 4.2) on the device against
the oracle: the library-side explorer, evaluating each round with
kv_eval_configs, must visit the configurations the oracle's Alg. 1 visits
with the oracle's replay as evaluator, reach the same objectives (1e-6
relative, as every parity test) and the same front and hypervolume."""
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("policy", [0, 1])
def test_search_matches_oracle(oracle_mod, policy):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from oracle import search as S
    from paper_2603_08739_amd import host
    from paper_2603_08739_amd import search as P
    t = tg.tiny(n_req=600)
    hbm = 2048
    d_rng, t_rng, res = (0, 24000, 6000), (0, 48000, 12000), (750, 1500)
    tau = (0.02, 0.05, 0.02)
    say(f"  search: n={t.n} policy={policy}")
    h = host.load(t)
    ex = P.Explorer(h, t.n_groups, host.cost_model(tg.DEFAULT_COST), hbm=hbm, policy=policy)
    rounds = ex.run(d_rng, t_rng, *tau, res=res)
    flags = ex.front()
    h.free()

    def simulate(points):
        cfgs = tg.from_list([{"cap": (hbm, d, s), "policy": policy} for d, s in points])
        return oracle_mod.objectives(t, cfgs, oracle_mod.replay(t, cfgs), tg.DEFAULT_COST)

    pts, obj, r_or = S.explore(simulate, *d_rng, *t_rng, *tau, res_d=res[0], res_t=res[1])
    say(f"  search: {len(pts)} configurations in {r_or} rounds")
    assert ex.points == pts and rounds == r_or
    np.testing.assert_allclose(ex.obj, obj, rtol=1e-6, atol=0)
    np.testing.assert_array_equal(flags, oracle_mod.pareto(obj).astype(bool))
    mo = P.minimised(obj)
    ref = mo.max(axis=0) + 1.0
    hv = P.hypervolume(P.minimised(ex.obj)[flags], ref)
    assert hv == pytest.approx(S.hypervolume(mo[flags], ref), rel=1e-9)
    assert len(pts) > 25


def test_search_over_ttl_matches_oracle(oracle_mod):
    """Alg. 1 over (DRAM, disk TTL): the planner's two dimensions."""
    from oracle import search as S
    from paper_2603_08739_amd import host
    from paper_2603_08739_amd import search as P
    t = tg.tiny(n_req=600)
    hbm = 2048
    d_rng, t_rng, res = (0, 24000, 6000), (0, 40, 10), (750, 1)
    tau = (0.02, 0.05, 0.02)
    unit = 0.5  # seconds per TTL step
    h = host.load(t)
    ex = P.Explorer(h, t.n_groups, host.cost_model(tg.DEFAULT_COST), hbm=hbm, second="ttl",
                    ttl_unit=unit)
    rounds = ex.run(d_rng, t_rng, *tau, res=res)
    flags = ex.front()
    h.free()

    def simulate(points):
        cfgs = tg.from_list([{"cap": (hbm, d, 0), "ttl": s * unit} for d, s in points])
        return oracle_mod.objectives(t, cfgs, oracle_mod.replay(t, cfgs), tg.DEFAULT_COST)

    pts, obj, r_or = S.explore(simulate, *d_rng, *t_rng, *tau, res_d=res[0], res_t=res[1])
    say(f"  ttl search: {len(pts)} configurations in {r_or} rounds")
    assert ex.points == pts and rounds == r_or
    np.testing.assert_allclose(ex.obj, obj, rtol=1e-6, atol=0)
    np.testing.assert_array_equal(flags, oracle_mod.pareto(ex.obj).astype(bool))
    assert len(pts) > 25
