"""Memo mode of the oracle equals its literal replay.

Memo mode rests on one fact of the inclusive hierarchy: every tier is an
independent cache that sees every access of its partition, so a tier's
presence bits, inserts and evictions depend only on (partition, policy,
capacity).  These tests pin that decomposition against the literal
per-configuration replay, element by element, on random traces that mix
policies, groups, block weights, partitioned and shared configurations,
repeated capacities (shared caches) and the non-inclusive modes (which memo
mode replays literally), so a wrong mask, a swapped tier order or a dropped
weight plane shows up as a difference.
"""
from __future__ import annotations

import numpy as np
import pytest

import tracegen as tg


@pytest.mark.parametrize("seed,n_groups,weights", [
    (1, 1, (1,)), (2, 1, (1, 4)), (3, 3, (1,)), (4, 4, (1, 2, 4)), (5, 2, (3, 7)),
    (6, 1, (1, 255)),
])
def test_memo_equals_literal(oracle_mod, seed, n_groups, weights):
    O = oracle_mod
    w_max = max(weights)
    t = tg.random_trace(seed, 3000, 240, n_groups=n_groups, weight_choices=weights,
                        zipf_s=0.9, reuse_bias=0.3)
    c = tg.random_configs(seed, 60, n_groups, w_max, 60 * w_max)
    # repeat tier capacities across configs so that caches are shared
    c.cap[30:40] = c.cap[0:10]
    c.cap_group[30:40] = c.cap_group[0:10]
    lit = O.replay(t, c)
    memo = O.replay_memo(t, c)
    assert np.array_equal(lit, memo)


def test_memo_mixed_modes(oracle_mod):
    O = oracle_mod
    t = tg.random_trace(9, 2000, 150, zipf_s=0.8, reuse_bias=0.2)
    items = []
    for caps in [(8, 0, 30), (8, 16, 0), (0, 12, 40), (20, 20, 20), (5, 0, 0)]:
        for pol in (tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU):
            items.append({"cap": caps, "policy": pol})
        items.append({"cap": caps, "mode": tg.MODE_EXCLUSIVE_DEMOTE})
        items.append({"cap": caps, "mode": tg.MODE_INCLUSIVE_PREFIX})
    c = tg.from_list(items)
    assert np.array_equal(O.replay(t, c), O.replay_memo(t, c))


def test_memo_word_boundaries(oracle_mod):
    """Lists whose length is 63, 64, 65 and 129 accesses (bit words and tails)."""
    O = oracle_mod
    for n in (1, 63, 64, 65, 129):
        t = tg.random_trace(n, n, 20, n_groups=2, weight_choices=(1, 3))
        c = tg.random_configs(n, 12, 2, 3, 30)
        assert np.array_equal(O.replay(t, c), O.replay_memo(t, c))


def test_memo_rejects_like_literal(oracle_mod):
    O = oracle_mod
    t = tg.from_blocks([1, 2, 1], weights={1: 4, 2: 1})
    with pytest.raises(ValueError):
        O.replay_memo(t, tg.from_list([{"cap": (3, 0, 0)}]))
