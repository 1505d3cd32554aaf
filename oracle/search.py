"""Adaptive Pareto exploration (Alg. 1, Section 4.2) and the hypervolume
indicator, plain Python.

TEST INFRASTRUCTURE ONLY: the test suite calls this module with the oracle's
evaluator; the GPU library never imports it, and it imports nothing from the
GPU package.

* :func:`explore`      Alg. 1 over two capacity dimensions, with any evaluator
                       ``simulate(points) -> [(cost, throughput, latency)]``.
* :func:`hypervolume`  volume dominated by a set of points (all objectives
                       minimised) up to a reference point, by summing the
                       cells of the grid the points' coordinates span.

Reading of Alg. 1 used here (the paper leaves these open):
* the two dimensions are the DRAM capacity d and the second dimension t of
  the paper's grid (here a disk capacity), both integers;
* a difference between two configurations is relative:
  |a - b| / max(|a|, |b|) (0 when both are 0);
* "adjacent pair" = two simulated configurations on one line of constant t
  (or constant d) with no simulated configuration between them;
* a midpoint is taken only if it is a new point at least one resolution
  step (`res_d` along d, `res_t` along t) away from both ends:
  d1 + res_d * floor((d2 - d1) / (2 * res_d)), likewise for t;
* the DRAM expansion looks at the line t = t_min (the paper's TTL = 0) and
  adds the column d_top + step_d over the initial t grid;
* rounds stop when no new point is proposed, or after `max_rounds`.
"""
from __future__ import annotations

import numpy as np


def _rel(a: float, b: float) -> float:
    m = max(abs(a), abs(b))
    return 0.0 if m == 0.0 else abs(a - b) / m


def explore(simulate, d_min, d_max, d_step, t_min, t_max, t_step, tau_e, tau_perf, tau_cost,
            res_d=1, res_t=1, max_rounds=64):
    """Alg. 1.  Returns (points [(d, t)] in simulation order, objectives
    float64 [n, 3] as (cost, throughput, latency), rounds run)."""
    t_grid = list(range(t_min, t_max + 1, t_step))
    todo = [(d, t) for d in range(d_min, d_max + 1, d_step) for t in t_grid]
    seen = {}
    order = []
    rounds = 0
    while todo and rounds < max_rounds:
        rounds += 1
        new = sorted(p for p in set(todo) if p not in seen)
        if new:
            res_obj = simulate(new)
            for p, o in zip(new, res_obj):
                seen[p] = tuple(float(x) for x in o)
                order.append(p)
        todo = []
        # DRAM expansion along t = t_min, while the last step still pays
        line = sorted(d for (d, t) in seen if t == t_min)
        top = line[-1]
        if (top - d_step, t_min) in seen:
            lat_prev = seen[(top - d_step, t_min)][2]
            lat_top = seen[(top, t_min)][2]
            if _rel(lat_prev, lat_top) > tau_e:
                todo += [(top + d_step, t) for t in t_grid]
        # refinement between neighbours whose objectives differ a lot
        for axis in (0, 1):
            lines = {}
            for p in seen:
                lines.setdefault(p[1 - axis], []).append(p[axis])
            for fixed, vals in lines.items():
                vals.sort()
                for a, b in zip(vals, vals[1:]):
                    pa = (a, fixed) if axis == 0 else (fixed, a)
                    pb = (b, fixed) if axis == 0 else (fixed, b)
                    oa, ob = seen[pa], seen[pb]
                    perf = _rel(oa[2], ob[2]) > tau_perf or _rel(oa[1], ob[1]) > tau_perf
                    res = res_d if axis == 0 else res_t
                    if perf and _rel(oa[0], ob[0]) > tau_cost and b - a >= 2 * res:
                        m = a + res * ((b - a) // (2 * res))
                        todo.append((m, fixed) if axis == 0 else (fixed, m))
        todo = [p for p in todo if p not in seen]
    obj = np.array([seen[p] for p in order], dtype=np.float64).reshape(-1, 3)
    return order, obj, rounds


def hypervolume(points, ref) -> float:
    """Volume of the union of boxes [p, ref] over the points that lie below
    ref in every objective (all objectives minimised)."""
    ref = np.asarray(ref, dtype=np.float64)
    pts = np.asarray(points, dtype=np.float64).reshape(-1, ref.size)
    pts = pts[(pts < ref).all(axis=1)]
    if len(pts) == 0:
        return 0.0
    cuts = [np.unique(np.concatenate([pts[:, k], [ref[k]]])) for k in range(ref.size)]
    vol = 0.0
    for i in range(len(cuts[0]) - 1):
        for j in range(len(cuts[1]) - 1):
            for k in range(len(cuts[2]) - 1):
                lo = np.array([cuts[0][i], cuts[1][j], cuts[2][k]])
                if (pts <= lo).all(axis=1).any():
                    vol += ((cuts[0][i + 1] - cuts[0][i]) * (cuts[1][j + 1] - cuts[1][j]) *
                            (cuts[2][k + 1] - cuts[2][k]))
    return float(vol)
