"""Pins of the oracle's exclusive (write-back demotion) hierarchy under every
replacement policy and under mixed block weights (no GPU needed).

* hand-worked two-tier cases (``golden/exclusive_cases.txt``, derivations
  inside): the promotion of a lower-tier hit, the demotion cascade, FIFO's
  unreordered hits, LFU's entry of a demoted block as its tier's newest
  member, eviction until a weighted block fits;
* one live tier: the hierarchy is that tier's single cache, whose policies
  the single-cache pins fix;
* a top tier that holds every block: only cold misses, nothing below it;
* flow identities on random traces: every access not served by the top tier
  enters it, every block a tier demotes enters the next live tier, hits plus
  the last tier's misses count every access, and what a tier still holds at
  the end is non-negative and within its capacity.
A wrong victim, a promotion that keeps the block below, a demotion to the
wrong tier or a dropped count fails one of these.
"""
import os

import numpy as np
import pytest

import tracegen as tg

GOLD = os.path.join(os.path.dirname(__file__), "golden")
POL = {"LRU": tg.POLICY_LRU, "FIFO": tg.POLICY_FIFO, "LFU": tg.POLICY_LFU}


def cases():
    for line in open(os.path.join(GOLD, "exclusive_cases.txt")):
        if line.strip() and not line.startswith("#"):
            yield line.split()


@pytest.mark.parametrize("case", list(cases()), ids=lambda c: f"{c[0]}-{c[2]}")
def test_hand_cases(oracle_mod, case):
    pol, caps, string, wts = case[:4]
    per_tier = case[4:]
    labels = [ord(c) for c in string]
    weights = None
    if wts != "-":
        weights = {ord(k): int(v) for k, v in (x.split("=") for x in wts.split(","))}
    t = tg.from_blocks(labels, weights=weights)
    c = tg.from_list([{"cap": tuple(int(x) for x in caps.split(",")), "policy": POL[pol],
                       "mode": tg.MODE_EXCLUSIVE_DEMOTE}])
    r = oracle_mod.replay(t, c)[0, 0]
    for k in range(3):
        cnt = [int(x) for x in per_tier[2 * k].split("/")]
        wsum = [int(x) for x in per_tier[2 * k + 1].split("/")]
        assert list(r[k, :4]) == cnt, (case, k)
        assert list(r[k, 4:]) == wsum, (case, k)


def random_trace(seed, n=3000, blocks=220, groups=1, weights=(1, 3, 4)):
    return tg.random_trace(seed, n, blocks, n_groups=groups, weight_choices=weights, zipf_s=0.7)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("policy", [tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU])
def test_one_live_tier_is_a_single_cache(oracle_mod, seed, policy):
    t = random_trace(seed, groups=2)
    items = []
    for c in (4, 37, 150, 600):
        for k in range(3):
            caps = [0, 0, 0]
            caps[k] = c
            items.append({"cap": tuple(caps), "policy": policy})
    inc = tg.from_list(items)
    exc = tg.from_list([dict(x, mode=tg.MODE_EXCLUSIVE_DEMOTE) for x in items])
    np.testing.assert_array_equal(oracle_mod.replay(t, exc), oracle_mod.replay(t, inc))


@pytest.mark.parametrize("policy", [tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU])
def test_top_tier_holding_everything(oracle_mod, policy):
    O = oracle_mod
    t = random_trace(11)
    u = len(np.unique(t.hash))
    dw = int(sum(int(t.weight[np.nonzero(t.hash == h)[0][0]]) for h in np.unique(t.hash)))
    c = tg.from_list([{"cap": (dw, 50, 80), "policy": policy, "mode": tg.MODE_EXCLUSIVE_DEMOTE}])
    r = O.replay(t, c)[0, 0]
    assert r[0, O.HIT] == t.n - u and r[0, O.INS] == u and r[0, O.EVICT] == 0
    assert r[0, O.INS_W] == dw
    for k in (1, 2):
        assert r[k, O.MISS] == u and r[k, O.HIT] == 0 and r[k, O.INS] == 0 and r[k, O.EVICT] == 0


def flow_check(O, t, cfgs, r):
    G = t.n_groups
    for i in range(cfgs.n):
        part = bool(cfgs.partitioned[i])
        for g in range(G):
            m = t.group == g
            n_g, nw_g = int(m.sum()), int(t.weight[m].astype(np.int64).sum())
            caps = [int(cfgs.cap_group[i, k, g]) if part else int(cfgs.cap[i, k])
                    for k in range(3)]
            live = [k for k in range(3) if caps[k]]
            x = r[i, g].astype(np.int64)
            for k in range(3):
                if not caps[k]:
                    assert not x[k].any()
            if not live:
                continue
            top, last = live[0], live[-1]
            for f, tot in ((0, n_g), (4, nw_g)):      # hits, then weights
                hit, miss, ins, ev = f + O.HIT, f + O.MISS, f + O.INS, f + O.EVICT
                assert x[live, hit].sum() + x[last, miss] == tot
                assert x[top, ins] == tot - x[top, hit]
                for a, b in zip(live, live[1:]):
                    assert x[b, ins] == x[a, ev]
                    assert x[b, miss] == x[a, miss] - x[b, hit]
                for k in live:
                    held = x[k, ins] - x[k, ev] - (x[k, hit] if k != top else 0)
                    assert held >= 0
                    if f == 4 and part:
                        assert held <= caps[k]


@pytest.mark.parametrize("seed", range(6))
def test_flow_identities(oracle_mod, seed):
    t = random_trace(100 + seed, groups=3)
    cfgs = tg.random_configs(seed, 40, 3, 4, 500, exclusive=True,
                             exclusive_policies=(tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU))
    r = oracle_mod.replay(t, cfgs)
    flow_check(oracle_mod, t, cfgs, r)
    # a shared hierarchy holds at most its capacity over all groups
    for i in range(cfgs.n):
        if cfgs.partitioned[i]:
            continue
        x = r[i].astype(np.int64).sum(axis=0)
        live = [k for k in range(3) if cfgs.cap[i, k]]
        for k in live:
            held = x[k, 6] - x[k, 7] - (x[k, 4] if k != live[0] else 0)
            assert 0 <= held <= int(cfgs.cap[i, k])


def test_policies_differ(oracle_mod):
    """The three policies give different counts on one hierarchy (the
    policy is not ignored below the top tier)."""
    t = random_trace(5)
    c = tg.from_list([{"cap": (40, 60, 90), "policy": p, "mode": tg.MODE_EXCLUSIVE_DEMOTE}
                      for p in (tg.POLICY_LRU, tg.POLICY_FIFO, tg.POLICY_LFU)])
    r = oracle_mod.replay(t, c)
    assert not np.array_equal(r[0], r[1]) and not np.array_equal(r[0], r[2])
    assert not np.array_equal(r[1], r[2])
