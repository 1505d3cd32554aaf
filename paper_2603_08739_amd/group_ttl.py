"""ROI-aware group TTL (Alg. 2, Section 4.3) over the library's TTL curves.

Requests are grouped by prefix subtree (the K subtrees with the most
requests, plus one residual group); the disk-tier curves H_g(t) and C_g(t)
of every group come from one ``kv_ttl_curves`` call on the device; the
host then picks each group's ROI-optimal TTL, scales the TTLs to the
storage budget and refines them with multi-start SLSQP (scipy), maximising
the total hits under the budget.

Conventions (where the paper leaves them open): a request's subtree is the
hash of its first block; subtrees rank by request count, ties to the smaller
hash; the curves are taken as piecewise linear between the TTL grid's
points; the ROI-optimal TTL is the first grid TTL with nonzero storage that
maximises H/C; the perturbed starts are t_init * (1 + u), u uniform in
[-1/2, 1/2) per group from numpy's default generator seeded with `seed`,
clipped to the grid's range; SLSQP works on t / t_max with the hits
normalised by all gaps and the storage by the budget; a start counts if its
result meets the budget (to 1e-9 relative), and the most hits win.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.optimize import minimize


def subtree_groups(first_hash, k):
    """Group of every request (uint8) and the top-k subtree roots, from the
    requests' first block hashes."""
    first = np.asarray(first_hash, dtype=np.uint64)
    roots, inv, cnt = np.unique(first, return_inverse=True, return_counts=True)
    rank = np.lexsort((roots, -cnt.astype(np.int64)))   # most requests first, then hash
    top = rank[:k]
    gid = np.full(len(roots), k, dtype=np.uint8)
    gid[top] = np.arange(len(top), dtype=np.uint8)
    return gid[inv], [int(roots[i]) for i in top]


def allocate(hits, store, ttl, budget, seed=0):
    """Per-group TTLs from curves hits/store [G, m+1] on the grid `ttl`."""
    H = np.asarray(hits, dtype=np.float64)
    C = np.asarray(store, dtype=np.float64)
    T = np.asarray(ttl, dtype=np.float64)
    G, t_max = H.shape[0], float(T[-1])
    roi = np.where(C > 0, H / np.where(C > 0, C, 1.0), -1.0)
    j = np.argmax(roi, axis=1)                       # first maximum
    t_roi = np.where(roi[np.arange(G), j] >= 0, T[j], 0.0)

    def at(curves, t):
        return np.array([np.interp(t[g], T, curves[g]) for g in range(G)])

    unscaled = float(at(C, t_roi).sum())
    alpha = budget / unscaled if unscaled > 0 else 0.0
    t_init = np.clip(alpha * t_roi, 0.0, t_max)
    rng = np.random.default_rng(seed)
    n_pert = math.isqrt(max(G - 1, 0)) + 1
    starts = [t_init] + [np.clip(t_init * (1.0 + rng.uniform(-0.5, 0.5, G)), 0.0, t_max)
                         for _ in range(n_pert)]
    scale = max(float(H[:, -1].sum()), 1.0)
    best = (-1.0, np.zeros(G))
    for t0 in starts:
        sol = minimize(lambda x: -at(H, x * t_max).sum() / scale, t0 / t_max, method="SLSQP",
                       bounds=[(0.0, 1.0)] * G,
                       constraints=[{"type": "ineq",
                                     "fun": lambda x: 1.0 - at(C, x * t_max).sum() / budget}])
        t = np.clip(sol.x, 0.0, 1.0) * t_max
        if at(C, t).sum() <= budget * (1.0 + 1e-9):
            h = float(at(H, t).sum())
            if h > best[0]:
                best = (h, t)
    return {"t_roi": t_roi, "alpha": alpha, "t_init": t_init, "starts": len(starts),
            "t": best[1], "hits": best[0], "cost": float(at(C, best[1]).sum())}


def uniform_ttl(hits, store, ttl, budget):
    """One TTL for all groups: the largest t whose summed storage fits the
    budget, and its hits."""
    H = np.asarray(hits, dtype=np.float64).sum(axis=0)
    C = np.asarray(store, dtype=np.float64).sum(axis=0)
    T = np.asarray(ttl, dtype=np.float64)
    if np.interp(T[-1], T, C) <= budget:
        t = float(T[-1])
    else:
        lo, hi = 0.0, float(T[-1])
        for _ in range(200):
            mid = 0.5 * (lo + hi)
            lo, hi = (mid, hi) if np.interp(mid, T, C) <= budget else (lo, mid)
        t = lo
    return t, float(np.interp(t, T, H))
