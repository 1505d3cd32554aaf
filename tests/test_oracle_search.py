"""Pins of the oracle-side Alg. 1 (adaptive Pareto exploration, Section 4.2)
and of the hypervolume indicator: volumes worked by hand, and explorations
over evaluators with a known shape whose visited points follow from the
algorithm's rules by hand."""
import itertools

import numpy as np
import pytest

from oracle import search as S


def test_hypervolume_hand_cases():
    ref = (4.0, 4.0, 4.0)
    assert S.hypervolume([(1.0, 2.0, 3.0)], ref) == 3.0 * 2.0 * 1.0
    # two boxes [1,4]x[2,4]x[3,4] (6) and [2,4]x[1,4]x[3,4] (6) overlap in
    # [2,4]x[2,4]x[3,4] (4): 6 + 6 - 4
    assert S.hypervolume([(1.0, 2.0, 3.0), (2.0, 1.0, 3.0)], ref) == 8.0
    # a dominated point and a point outside the reference add nothing
    assert S.hypervolume([(1.0, 2.0, 3.0), (2.0, 3.0, 3.5), (0.0, 5.0, 0.0)], ref) == 6.0
    assert S.hypervolume([], ref) == 0.0


def test_hypervolume_invariances():
    rng = np.random.default_rng(3)
    pts = rng.uniform(0, 1, (12, 3))
    ref = (1.0, 1.0, 1.0)
    v = S.hypervolume(pts, ref)
    assert v == pytest.approx(S.hypervolume(pts[::-1], ref), rel=1e-12)
    for perm in itertools.permutations(range(3)):
        assert v == pytest.approx(S.hypervolume(pts[:, perm], ref), rel=1e-12)
    # scaling one objective scales the volume
    sc = pts.copy()
    sc[:, 0] *= 2.0
    assert S.hypervolume(sc, (2.0, 1.0, 1.0)) == pytest.approx(2 * v, rel=1e-12)


def step_evaluator(points):
    """Latency drops from 2 to 1 at d = 37; cost grows with d + t."""
    return [(float(d + t + 1), 1.0 / (2.0 if d < 37 else 1.0), 2.0 if d < 37 else 1.0)
            for d, t in points]


def test_refinement_localises_a_step():
    pts, obj, rounds = S.explore(step_evaluator, 0, 100, 20, 0, 0, 1, tau_e=0.5,
                                 tau_perf=0.1, tau_cost=0.01)
    # grid, then the midpoints 30, 35, 37, 36 of the pairs that straddle the step
    assert pts == [(0, 0), (20, 0), (40, 0), (60, 0), (80, 0), (100, 0),
                   (30, 0), (35, 0), (37, 0), (36, 0)]
    assert rounds == 5
    assert obj[-1].tolist() == [37.0, 0.5, 2.0]


def smooth_evaluator(points):
    """Latency 10 / (10 + d) + t / 1000; cost d + t."""
    return [(float(d + t), (10.0 + d) / 10.0, 10.0 / (10.0 + d) + t / 1000.0)
            for d, t in points]


def test_dram_expansion_stops_in_the_long_tail():
    # the last step's relative latency gain 10 / (10 + d) first drops to
    # tau_e = 0.105 or below at d = 90: columns up to 90 are simulated, for
    # both t values of the initial grid
    pts, _, rounds = S.explore(smooth_evaluator, 0, 20, 10, 0, 5, 5, tau_e=0.105,
                               tau_perf=10.0, tau_cost=10.0)
    assert sorted(pts) == [(d, t) for d in range(0, 100, 10) for t in (0, 5)]
    assert rounds == 8


def test_refinement_stays_on_each_axis_resolution():
    # along d the resolution is 8: the step at 37 is bracketed by 32 and 40
    pts, _, _ = S.explore(step_evaluator, 0, 64, 32, 0, 0, 1, tau_e=0.5, tau_perf=0.1,
                          tau_cost=0.01, res_d=8, res_t=3)
    assert pts == [(0, 0), (32, 0), (64, 0), (48, 0), (40, 0)]
