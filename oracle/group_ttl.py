"""ROI-aware group TTL (Alg. 2, Section 4.3), plain Python with scipy.

TEST INFRASTRUCTURE ONLY: the test suite runs this on the oracle's TTL
curves; the GPU library never imports it, and it imports nothing from the
GPU package.

* :func:`subtree_groups`  requests -> top-K prefix subtrees + a residual group
* :func:`allocate`        per-group ROI-optimal TTLs, budget scaling, multi-start
                          SLSQP over the groups' TTLs

Readings used here (the paper leaves these open):
* a request's prefix subtree is the hash of its first block (block hashes
  are prefix chains, so every block lies in exactly one subtree); the K
  subtrees with the most requests (ties: smaller hash) are groups 0..K-1
  in that order, every other request goes to group K;
* H_g and C_g are known on a TTL grid 0 = t_0 < ... < t_m and taken as
  piecewise linear in between (the optimiser needs a continuous curve);
* the ROI-optimal TTL of a group is the first grid TTL with C_g > 0 that
  maximises H_g / C_g;
* the perturbed starts are t_init * (1 + u), u uniform in [-1/2, 1/2) per
  group from numpy's default generator seeded with `seed`, clipped to
  [0, t_m];
* SLSQP runs on x = t / t_m in [0, 1] with objective -sum_g H_g / (total
  gaps) and constraint 1 - sum_g C_g / B >= 0 (scipy defaults otherwise);
  a start's result counts if it meets the budget (to 1e-9 relative); the
  most hits win, the earlier start on ties.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.optimize import minimize


def subtree_groups(first_hash, k):
    """first_hash: the first block hash of every request.  Returns (group
    per request uint8, the top-k subtree roots)."""
    count = {}
    for h in first_hash:
        count[int(h)] = count.get(int(h), 0) + 1
    ranked = sorted(count, key=lambda h: (-count[h], h))[:k]
    gid = {h: g for g, h in enumerate(ranked)}
    groups = np.array([gid.get(int(h), k) for h in first_hash], dtype=np.uint8)
    return groups, ranked


def _interp(ttl, curve, t):
    return float(np.interp(t, ttl, curve))


def allocate(hits, store, ttl, budget, seed=0):
    """hits, store: [G, m+1] curves at the TTL grid `ttl`; budget in the
    store's unit.  Returns a dict with the chosen TTLs and their hits/cost."""
    hits = np.asarray(hits, dtype=np.float64)
    store = np.asarray(store, dtype=np.float64)
    ttl = np.asarray(ttl, dtype=np.float64)
    G = hits.shape[0]
    t_max = float(ttl[-1])
    # per-group ROI-optimal TTL on the grid
    t_roi = np.zeros(G)
    for g in range(G):
        best, arg = -1.0, None
        for j in range(len(ttl)):
            if store[g, j] > 0:
                r = hits[g, j] / store[g, j]
                if r > best:
                    best, arg = r, j
        t_roi[g] = ttl[arg] if arg is not None else 0.0
    unscaled = sum(_interp(ttl, store[g], t_roi[g]) for g in range(G))
    alpha = budget / unscaled if unscaled > 0 else 0.0
    t_init = np.clip(alpha * t_roi, 0.0, t_max)
    K = G - 1
    rng = np.random.default_rng(seed)
    starts = [t_init]
    for _ in range(math.isqrt(max(K, 0)) + 1):
        starts.append(np.clip(t_init * (1.0 + rng.uniform(-0.5, 0.5, G)), 0.0, t_max))
    total = max(float(hits[:, -1].sum()), 1.0)

    def total_hits(t):
        return sum(_interp(ttl, hits[g], t[g]) for g in range(G))

    def total_cost(t):
        return sum(_interp(ttl, store[g], t[g]) for g in range(G))

    best_t, best_h = np.zeros(G), -1.0
    for t0 in starts:
        res = minimize(lambda x: -total_hits(x * t_max) / total, t0 / t_max, method="SLSQP",
                       bounds=[(0.0, 1.0)] * G,
                       constraints=[{"type": "ineq",
                                     "fun": lambda x: 1.0 - total_cost(x * t_max) / budget}])
        t = np.clip(res.x, 0.0, 1.0) * t_max
        if total_cost(t) <= budget * (1.0 + 1e-9):
            h = total_hits(t)
            if h > best_h:
                best_t, best_h = t, h
    return {"t_roi": t_roi, "alpha": alpha, "t_init": t_init, "starts": len(starts),
            "t": best_t, "hits": best_h, "cost": total_cost(best_t)}


def best_uniform(hits, store, ttl, budget):
    """The one TTL for every group with the most hits within the budget:
    the largest t whose summed storage fits (storage grows with t)."""
    hits = np.asarray(hits, dtype=np.float64)
    store = np.asarray(store, dtype=np.float64)
    ttl = np.asarray(ttl, dtype=np.float64)
    tot_c = store.sum(axis=0)
    lo, hi = 0.0, float(ttl[-1])
    if float(np.interp(hi, ttl, tot_c)) <= budget:
        t = hi
    else:
        for _ in range(200):
            mid = 0.5 * (lo + hi)
            if float(np.interp(mid, ttl, tot_c)) <= budget:
                lo = mid
            else:
                hi = mid
        t = lo
    return t, float(np.interp(t, ttl, hits.sum(axis=0)))
