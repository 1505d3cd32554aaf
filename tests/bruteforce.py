"""Independent brute-force formulations used to pin the oracle on tiny inputs.

Each function states a cache fact in a form different from the oracle's
replay, so a mistake in the oracle's data structures or bookkeeping shows up
as a disagreement:

* weighted LRU stack distance straight from Mattson's definition (distinct
  blocks touched since the previous access, plus the block itself);
* FIFO residency as "the longest suffix of the insertion history whose total
  weight fits", recomputed from scratch at every access;
* LFU with the victim found by a linear scan over the resident set.
"""
from __future__ import annotations

import math

INF = math.inf


def stack_distances(labels, weights):
    """D_i = w_i + total weight of distinct other blocks accessed since prev(i)."""
    out = []
    last = {}
    for i, b in enumerate(labels):
        if b not in last:
            out.append(INF)
        else:
            p = last[b]
            seen = set(labels[p + 1:i])
            out.append(weights[b] + sum(weights[x] for x in seen))
        last[b] = i
    return out


def unit_stack_distances(labels):
    return stack_distances(labels, {b: 1 for b in set(labels)})


def lru_hits(labels, weights, cap):
    """LRU hits of one cache: access i hits iff D_i <= cap (cap >= max weight)."""
    if cap == 0:
        return 0
    return sum(1 for d in stack_distances(labels, weights) if d <= cap)


def lru_final_resident(labels, weights, cap):
    """Blocks resident at the end: the maximal recency prefix of weight <= cap."""
    order = []
    for b in reversed(labels):
        if b not in order:
            order.append(b)
    res, used = [], 0
    for b in order:
        if used + weights[b] > cap:
            break
        used += weights[b]
        res.append(b)
    return res


def fifo_hits_suffix(labels, weights, cap):
    """FIFO via the insertion-history suffix characterisation."""
    history = []  # blocks in insertion order (one entry per miss)
    hits = 0
    for b in labels:
        # resident set = longest suffix of history with total weight <= cap
        res, used = set(), 0
        for x in reversed(history):
            if used + weights[x] > cap:
                break
            used += weights[x]
            res.add(x)
        if b in res:
            hits += 1
        else:
            history.append(b)
    return hits


def lfu_scan(labels, weights, cap):
    """LFU by linear victim scan; returns (hits, evictions)."""
    res = {}  # block -> [freq, last]
    used = 0
    hits = ev = 0
    for t, b in enumerate(labels):
        if b in res:
            hits += 1
            res[b][0] += 1
            res[b][1] = t
            continue
        while used + weights[b] > cap:
            v = min(res, key=lambda x: (res[x][0], res[x][1]))
            used -= weights[v]
            del res[v]
            ev += 1
        res[b] = [1, t]
        used += weights[b]
    return hits, ev


def chain_trace_labels(seed, n_req, n_sys=3, n_docs=12, sys_len=(2, 6), doc_len=(1, 9)):
    """Requests that are prefix chains of a small tree: each document hangs
    below one of a few system prompts; a request reads a prefix of
    (system prompt + document).  Labels: (system s, index j) -> 1000 * s + j,
    (document d, index j) -> 100000 + 1000 * d + j.  Returns (labels, request
    index per access)."""
    import random
    rnd = random.Random(seed)
    sys_l = [rnd.randint(*sys_len) for _ in range(n_sys)]
    docs = [(rnd.randrange(n_sys), rnd.randint(*doc_len)) for _ in range(n_docs)]
    labels, req = [], []
    for r in range(n_req):
        d = min(int(rnd.paretovariate(1.2)) - 1, n_docs - 1)
        s, dl = docs[d]
        full = [1000 * s + j for j in range(sys_l[s])] + [100000 + 1000 * d + j for j in range(dl)]
        k = rnd.randint(1, len(full))
        labels += full[:k]
        req += [r] * k
    return labels, req


def leaf_first_distances(labels, req, weights):
    """Radix-tree eviction as a priority order: a block ranks by (request of
    its latest access, then shallower first), so at access i of block b,
    with q the request of b's previous access, the blocks ranked above b
    are those accessed after request q (up to i); D'_i = w_b + their weight
    (INF for a first access)."""
    out, last_req = [], {}
    end = {}
    for i, r in enumerate(req):
        end[r] = i
    for i, b in enumerate(labels):
        if b not in last_req:
            out.append(INF)
        else:
            e = end[last_req[b]]
            seen = set(labels[e + 1:i])
            out.append(weights[b] + sum(weights[x] for x in seen))
        last_req[b] = req[i]
    return out


def leaf_first_final(labels, req, weights, cap):
    """Blocks held at the end: the maximal prefix, of weight <= cap, of the
    blocks ordered by (latest request descending, position in it ascending)."""
    last = {}
    for i, b in enumerate(labels):
        last[b] = (req[i], i)
    order = sorted(last, key=lambda b: (-last[b][0], last[b][1]))
    res, used = [], 0
    for b in order:
        if used + weights[b] > cap:
            break
        used += weights[b]
        res.append(b)
    return res
