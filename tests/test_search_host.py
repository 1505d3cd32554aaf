"""Host logic of the adaptive search (Alg. 1, Section 4.2) and of its
hypervolume indicator, without a device: the library-side explorer, given
the same evaluator, visits the same configurations in the same order as the
oracle's Alg. 1, and the sweep hypervolume equals the oracle's cell sum."""
import numpy as np
import pytest

from oracle import search as S


def explorer_with(evaluator):
    from paper_2603_08739_amd import search as P

    class Synthetic(P.Explorer):
        def __init__(self):
            super().__init__(None, 1, None, hbm=0)

        def evaluate(self, pts):
            self.calls += 1
            return np.asarray(evaluator(pts), dtype=np.float64).reshape(-1, 3)

    return Synthetic()


def wavy(points):
    """Cost grows with capacity; latency falls with a kink at d = 700 and a
    plateau in t beyond 3000."""
    out = []
    for d, t in points:
        lat = (3.0 if d < 700 else 1.0) / (1.0 + d / 400.0) + 2.0 / (1.0 + min(t, 3000) / 500.0)
        out.append((1.0 + d / 100.0 + t / 400.0, 1.0 / lat, lat))
    return out


@pytest.mark.parametrize("case", [
    dict(evaluator=wavy, d=(0, 1600, 400), t=(0, 4000, 1000), tau=(0.02, 0.05, 0.02), res=(25, 50)),
    dict(evaluator=wavy, d=(0, 800, 200), t=(0, 6000, 2000), tau=(0.2, 0.01, 0.001), res=(10, 10)),
])
def test_explorer_follows_the_oracle(case):
    ex = explorer_with(case["evaluator"])
    rounds = ex.run(case["d"], case["t"], *case["tau"], res=case["res"])
    pts, obj, r_or = S.explore(case["evaluator"], *case["d"], *case["t"], *case["tau"],
                               res_d=case["res"][0], res_t=case["res"][1])
    assert ex.points == pts
    assert rounds == r_or
    np.testing.assert_array_equal(ex.obj, obj)
    assert len(pts) > (case["d"][1] // case["d"][2] + 1) * (case["t"][1] // case["t"][2] + 1)


@pytest.mark.parametrize("seed", range(6))
def test_sweep_hypervolume_matches_cell_sum(seed):
    from paper_2603_08739_amd import search as P
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 25))
    pts = rng.uniform(0, 1, (n, 3))
    if seed % 2:
        pts = np.round(pts * 4) / 4    # ties in every coordinate
    ref = (1.1, 1.0, 1.05)
    assert P.hypervolume(pts, ref) == pytest.approx(S.hypervolume(pts, ref), rel=1e-12, abs=1e-15)
