"""Adaptive Pareto exploration (Alg. 1, Section 4.2) over the library.

The planner's coarse-to-fine search: evaluate a coarse grid of (DRAM
capacity d, second dimension t) configurations, widen the DRAM range while
the last DRAM step still cuts latency by more than tau_e, and put a new
configuration between neighbours whose latency or throughput differ by more
than tau_perf while their cost differs by more than tau_cost; repeat until
nothing new is proposed, then keep the non-dominated configurations.  Every
round's new configurations are evaluated in one ``kv_eval_configs`` call and
the front comes from ``kv_pareto``: this module only proposes configurations
and keeps the books.

Conventions (where the paper leaves them open): d is an integer granule
capacity of the DRAM tier and t either an integer granule capacity of the
disk tier (the paper's ablation grid, Section 5.3.1) or the disk TTL in
integer multiples of `ttl_unit` seconds (the paper's planner and Alg. 1:
an unbounded disk TTL tier, TTL 0 holding nothing); the HBM capacity, mode
and policy are fixed per search;
differences are relative, |a - b| / max(|a|, |b|); neighbours are
consecutive evaluated configurations on a line of constant t or constant d;
a midpoint must be a new point on the axis' resolution grid,
a + res * floor((b - a) / (2 * res)); the expansion follows the line
t = t_min and adds the next DRAM column over the initial t grid.
"""
from __future__ import annotations

import numpy as np
import torch

from . import kvcfg


def _relative(a, b):
    m = np.maximum(np.abs(a), np.abs(b))
    return np.where(m > 0, np.abs(a - b) / np.where(m > 0, m, 1.0), 0.0)


class Explorer:
    """One Alg. 1 search over a loaded trace."""

    def __init__(self, trace: kvcfg.Trace, n_groups: int, cost_model: kvcfg.kv_cost_model,
                 hbm: int, mode: int = 0, policy: int = 0, stream=None, second: str = "disk",
                 ttl_unit: float = 1.0):
        if second not in ("disk", "ttl"):
            raise ValueError("second dimension: 'disk' or 'ttl'")
        self.trace, self.G, self.model = trace, n_groups, cost_model
        self.hbm, self.mode, self.policy, self.stream = hbm, mode, policy, stream
        self.second, self.ttl_unit = second, float(ttl_unit)
        self.points: list[tuple[int, int]] = []   # evaluation order
        self.obj = np.zeros((0, 3))
        self.index: dict[tuple[int, int], int] = {}
        self.calls = 0

    def evaluate(self, pts):
        """(cost, throughput, latency) of configurations (hbm, d, t), one call."""
        n = len(pts)
        p = np.asarray(pts, dtype=np.int64).reshape(n, 2)
        cap = np.zeros((n, 3), dtype=np.uint64)
        cap[:, 0] = self.hbm
        cap[:, 1] = p[:, 0]
        disk_ttl = np.zeros(n, dtype=np.uint8)
        ttl = np.zeros((n, kvcfg.KV_MAX_GROUPS), dtype=np.float64)
        if self.second == "disk":
            cap[:, 2] = p[:, 1]
        else:
            disk_ttl[:] = 1
            ttl[:, :] = (p[:, 1] * self.ttl_unit)[:, None]
        cap_group = np.zeros((n, 3, kvcfg.KV_MAX_GROUPS), dtype=np.uint64)
        mode = np.full(n, self.mode, dtype=np.uint8)
        part = np.zeros(n, dtype=np.uint8)
        pol = np.full((n, kvcfg.KV_MAX_GROUPS), self.policy, dtype=np.uint8)
        arr, n_cfg = kvcfg.config_array(cap, cap_group, mode, part, pol, disk_ttl, None, ttl)
        counts = torch.zeros((n, self.G, 3, 8), dtype=torch.int64, device="cuda")
        obj = torch.zeros((n, 3), dtype=torch.float64, device="cuda")
        kvcfg.kv_eval_configs(self.trace, arr, n_cfg, self.model, counts, obj,
                              stream=self.stream)
        self.calls += 1
        return obj.cpu().numpy()

    def _add(self, pts):
        pts = sorted(set(p for p in pts if p not in self.index))
        if not pts:
            return 0
        o = self.evaluate(pts)
        for p in pts:
            self.index[p] = len(self.points)
            self.points.append(p)
        self.obj = np.concatenate([self.obj, o])
        return len(pts)

    def _of(self, p):
        return self.obj[self.index[p]]

    def run(self, d_range, t_range, tau_e, tau_perf, tau_cost, res=(1, 1), max_rounds=64):
        """d_range / t_range = (min, max, step); returns the number of rounds."""
        d0, d1, dd = d_range
        t0, t1, dt = t_range
        t_grid = list(range(t0, t1 + 1, dt))
        proposal = [(d, t) for d in range(d0, d1 + 1, dd) for t in t_grid]
        rounds = 0
        while proposal and rounds < max_rounds:
            rounds += 1
            self._add(proposal)
            proposal = []
            # widen the DRAM range while its last step still pays
            top = max(d for d, t in self.points if t == t0)
            if (top - dd, t0) in self.index:
                gain = _relative(self._of((top - dd, t0))[2], self._of((top, t0))[2])
                if gain > tau_e:
                    proposal.extend((top + dd, t) for t in t_grid)
            # refine between neighbours on every line of either axis
            pts = np.asarray(self.points, dtype=np.int64)
            for axis in (0, 1):
                step = res[axis]
                other = pts[:, 1 - axis]
                for fixed in np.unique(other):
                    on = np.nonzero(other == fixed)[0]
                    on = on[np.argsort(pts[on, axis], kind="stable")]
                    if len(on) < 2:
                        continue
                    a, b = on[:-1], on[1:]
                    oa, ob = self.obj[a], self.obj[b]
                    perf = (_relative(oa[:, 2], ob[:, 2]) > tau_perf) | \
                           (_relative(oa[:, 1], ob[:, 1]) > tau_perf)
                    gap = pts[b, axis] - pts[a, axis]
                    want = perf & (_relative(oa[:, 0], ob[:, 0]) > tau_cost) & (gap >= 2 * step)
                    for i in np.nonzero(want)[0]:
                        m = int(pts[a[i], axis] + step * (gap[i] // (2 * step)))
                        proposal.append((m, int(fixed)) if axis == 0 else (int(fixed), m))
            proposal = [p for p in proposal if p not in self.index]
        return rounds

    def front(self):
        """Non-dominated flags over every evaluated configuration."""
        obj = torch.from_numpy(np.ascontiguousarray(self.obj)).to("cuda")
        flags = torch.zeros(obj.shape[0], dtype=torch.uint8, device="cuda")
        kvcfg.kv_pareto(obj, flags, want_count=False, stream=self.stream)
        torch.cuda.synchronize()
        return flags.cpu().numpy().astype(bool)


def hypervolume(points, ref) -> float:
    """Volume dominated by `points` (all three objectives minimised) below
    `ref`: a sweep over the third objective, each slab's area from a
    staircase over the first two."""
    ref = np.asarray(ref, dtype=np.float64)
    p = np.asarray(points, dtype=np.float64).reshape(-1, 3)
    p = p[(p < ref).all(axis=1)]
    if len(p) == 0:
        return 0.0
    p = p[np.argsort(p[:, 2], kind="stable")]
    zs = np.append(p[:, 2], ref[2])
    vol = 0.0
    for i in range(len(p)):
        dz = zs[i + 1] - zs[i]
        if dz <= 0:
            continue
        act = p[: i + 1, :2]
        act = act[np.lexsort((act[:, 1], act[:, 0]))]
        area, best_y = 0.0, ref[1]
        for k in range(len(act)):
            best_y = min(best_y, act[k, 1])
            x_next = act[k + 1, 0] if k + 1 < len(act) else ref[0]
            area += (x_next - act[k, 0]) * (ref[1] - best_y)
        vol += area * dz
    return float(vol)


def minimised(obj):
    """(cost, throughput, latency) rows as all-minimised (cost, -throughput,
    latency)."""
    o = np.asarray(obj, dtype=np.float64).reshape(-1, 3).copy()
    o[:, 1] = -o[:, 1]
    return o
