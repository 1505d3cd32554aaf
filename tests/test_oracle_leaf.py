"""Pins of the oracle's radix-tree (leaf-first) eviction (Section 3.2: KV
blocks shared through a prefix tree; a radix cache evicts leaves).

The oracle keeps the tree literally (cached children per block, a set of
leaves ordered by latest access).  It is held to:
* a hand case where it keeps a block that LRU drops;
* a brute force of the priority order it amounts to on prefix-chain traces
  whose requests fit the cache: a block ranks by the request of its latest
  access, shallower blocks first within a request, so an access hits iff its
  block plus every block accessed since the end of the previous access's
  request fits the capacity; the blocks held at the end are the maximal
  prefix of that order;
* reductions: one-block requests are plain LRU; a cache holding every
  distinct block misses only first accesses;
* its refusals: traces that are not prefix chains, capacities below the
  heaviest request, and the unsupported hierarchies.
"""
import numpy as np
import pytest

import tracegen as tg
from tests import bruteforce as bf

HIT, MISS, INS, EVICT = 0, 1, 2, 3
LEAF = 3


def trace_of(labels, req, weights=None):
    t = tg.from_blocks(labels, weights=weights)
    t.req = np.asarray(req, dtype=np.uint32)
    t.req_time = np.arange(int(t.req[-1]) + 1, dtype=np.float64)
    return t


def test_hand_case(oracle_mod):
    # requests [A B] [C] [A] at capacity 2: LRU evicts A for C, leaf-first B
    labels, req = [0, 1, 2, 0], [0, 0, 1, 2]
    t = trace_of(labels, req)
    lru = oracle_mod.replay(t, tg.from_list([{"cap": (2, 0, 0)}]))[0, 0, 0]
    leaf = oracle_mod.replay(t, tg.from_list([{"cap": (2, 0, 0), "policy": LEAF}]))[0, 0, 0]
    assert lru[HIT] == 0 and leaf[HIT] == 1
    assert leaf[INS] == 3 and leaf[EVICT] == 1


@pytest.mark.parametrize("seed", range(12))
def test_priority_order_brute_force(oracle_mod, seed):
    labels, req = bf.chain_trace_labels(seed, 60)
    rng = np.random.default_rng(seed)
    wl = {b: int(rng.choice([1, 1, 2, 4])) for b in set(labels)}
    t = trace_of(labels, req, wl)
    D = bf.leaf_first_distances(labels, req, wl)
    req_w = {}
    for b, r in zip(labels, req):
        req_w[r] = req_w.get(r, 0) + wl[b]
    lo = max(req_w.values())
    distinct = sum(wl.values())
    for cap in sorted({lo, lo + 1, lo + 3, (lo + distinct) // 2, distinct}):
        for memo in (False, True):
            r = oracle_mod.replay(t, tg.from_list([{"cap": (cap, 0, 0), "policy": LEAF}]),
                                  memo=memo)[0, 0, 0]
            hits = sum(1 for d in D if d <= cap)
            assert r[HIT] == hits, (cap, memo)
            fin = bf.leaf_first_final(labels, req, wl, cap)
            assert r[EVICT] == r[INS] - len(fin)


def test_inclusive_tiers(oracle_mod):
    labels, req = bf.chain_trace_labels(99, 80)
    wl = {b: 1 for b in set(labels)}
    t = trace_of(labels, req, wl)
    D = bf.leaf_first_distances(labels, req, wl)
    lo = max(np.bincount(req))
    for caps in ((lo, lo + 4, 0), (lo + 2, 0, lo + 9), (lo + 5, lo + 1, lo + 20)):
        r = oracle_mod.replay(t, tg.from_list([{"cap": caps, "policy": LEAF}]))[0, 0]
        m = 0
        for k, c in enumerate(caps):
            if not c:
                continue
            want = sum(1 for d in D if m < d <= c) if c > m else 0
            assert r[k, HIT] == want
            m = max(m, c)


def test_reductions(oracle_mod):
    t = tg.random_trace(5, 800, 90, per_request=1, zipf_s=0.8)
    for cap in (1, 7, 30):
        a = oracle_mod.replay(t, tg.from_list([{"cap": (cap, 0, 0)}]))
        b = oracle_mod.replay(t, tg.from_list([{"cap": (cap, 0, 0), "policy": LEAF}]))
        assert np.array_equal(a, b)
    labels, req = bf.chain_trace_labels(7, 50)
    t = trace_of(labels, req)
    big = len(set(labels))
    r = oracle_mod.replay(t, tg.from_list([{"cap": (big, 0, 0), "policy": LEAF}]))[0, 0, 0]
    assert r[HIT] == len(labels) - big and r[EVICT] == 0


def test_refusals(oracle_mod):
    labels, req = bf.chain_trace_labels(3, 40)
    t = trace_of(labels, req)
    heavy = max(np.bincount(req))
    with pytest.raises(ValueError, match="code -4"):
        oracle_mod.replay(t, tg.from_list([{"cap": (heavy - 1, 0, 0), "policy": LEAF}]))
    for item in ({"cap": (heavy, 0, 0), "policy": LEAF, "mode": tg.MODE_EXCLUSIVE_DEMOTE},
                 {"cap": (heavy, 0, 0), "policy": LEAF, "mode": tg.MODE_INCLUSIVE_PREFIX}):
        with pytest.raises(ValueError, match="code -4"):
            oracle_mod.replay(t, tg.from_list([item]))
    # a block re-accessed after a different parent: not a prefix chain
    bad = trace_of([0, 1, 2, 1], [0, 0, 1, 1])
    with pytest.raises(ValueError, match="code -4"):
        oracle_mod.replay(bad, tg.from_list([{"cap": (4, 0, 0), "policy": LEAF}]))
    with pytest.raises(ValueError, match="code -1"):
        oracle_mod.replay(t, tg.from_list([{"cap": (heavy, 0, 0), "policy": 4}]))
