"""Pins of the oracle's prefix-reuse hierarchy (inclusive LRU tiers where a
request reuses only a run of its blocks from its first block on, as a
radix-tree KV cache does): hand-worked counts, the reduction to the plain
inclusive mode for one-block requests, and a brute-force replay written
here on small random traces."""
from collections import OrderedDict

import numpy as np
import pytest

import tracegen as tg

HIT, MISS, INS, EVICT = 0, 1, 2, 3


def trace_of(requests):
    lab = {}
    flat = [lab.setdefault(b, len(lab)) for r in requests for b in r]
    t = tg.from_blocks(flat)
    t.req = np.repeat(np.arange(len(requests), dtype=np.uint32), [len(r) for r in requests])
    t.req_time = np.arange(len(requests), dtype=np.float64)
    return t


def run(oracle_mod, t, caps, mode):
    cfgs = tg.from_list([{"cap": c, "mode": mode} for c in caps])
    return oracle_mod.replay(t, cfgs).astype(np.int64)


def test_single_tier_by_hand(oracle_mod):
    # [A B C] [A B D] [B C] [X A B]: with room for everything, plain reuse
    # hits A, B (request 2), B, C (request 3), A, B (request 4) = 6; prefix
    # reuse loses request 4's A and B behind the cold X = 4
    t = trace_of([["A", "B", "C"], ["A", "B", "D"], ["B", "C"], ["X", "A", "B"]])
    plain = run(oracle_mod, t, [(100, 0, 0)], 0)[0, 0, 0]
    pref = run(oracle_mod, t, [(100, 0, 0)], 2)[0, 0, 0]
    assert plain[HIT] == 6 and pref[HIT] == 4
    assert pref[MISS] == 11 - 4
    assert pref[INS] == plain[INS] == 5 and pref[EVICT] == plain[EVICT] == 0


def test_two_tiers_by_hand(oracle_mod):
    # HBM holds 3, DRAM 100.  [A B C D] leaves HBM with B C D; in [A C] the
    # HBM misses A (inserting it evicts B) and holds C, but with prefix
    # reuse C cannot come from HBM after A did not: DRAM serves both
    t = trace_of([["A", "B", "C", "D"], ["A", "C"]])
    plain = run(oracle_mod, t, [(3, 100, 0)], 0)[0, 0]
    pref = run(oracle_mod, t, [(3, 100, 0)], 2)[0, 0]
    assert plain[0, :4].tolist() == [1, 5, 5, 2] and plain[1, :4].tolist() == [1, 4, 4, 0]
    assert pref[0, :4].tolist() == [0, 6, 5, 2] and pref[1, :4].tolist() == [2, 4, 4, 0]


def test_one_block_requests_reduce_to_plain(oracle_mod):
    t = tg.random_trace(41, 3000, 400, weight_choices=(1, 2), zipf_s=0.9, per_request=1)
    caps = [(8, 0, 0), (40, 90, 0), (16, 64, 300)]
    np.testing.assert_array_equal(run(oracle_mod, t, caps, 2), run(oracle_mod, t, caps, 0))


def brute_force(t, cap):
    """Independent replay: one OrderedDict per tier, unit weights."""
    tiers = [OrderedDict() if c else None for c in cap]
    out = np.zeros((3, 4), dtype=np.int64)
    run_ok = [True] * 3
    prev_req = None
    for i in range(t.n):
        b, r = int(t.hash[i]), int(t.req[i])
        if r != prev_req:
            run_ok = [True] * 3
            prev_req = r
        pres = [tiers[k] is not None and b in tiers[k] for k in range(3)]
        avail = [pres[k] and run_ok[k] for k in range(3)]
        run_ok = avail
        served = next((k for k in range(3) if avail[k]), None)
        for k in range(3):
            if tiers[k] is None:
                continue
            if served == k:
                out[k, HIT] += 1
            elif served is None or served > k:
                out[k, MISS] += 1
            if pres[k]:
                tiers[k].move_to_end(b)
            else:
                out[k, INS] += 1
                if len(tiers[k]) >= cap[k]:
                    tiers[k].popitem(last=False)
                    out[k, EVICT] += 1
                tiers[k][b] = True
    return out


@pytest.mark.parametrize("seed", range(8))
def test_matches_brute_force(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    t = tg.random_trace(50 + seed, 1500, 120, zipf_s=0.8, reuse_bias=0.3,
                        per_request=int(rng.integers(2, 9)))
    caps = [(int(rng.integers(1, 40)), int(rng.integers(0, 90)), int(rng.integers(0, 140)))
            for _ in range(4)]
    got = run(oracle_mod, t, caps, 2)
    for c, cap in enumerate(caps):
        np.testing.assert_array_equal(got[c, 0, :, :4], brute_force(t, cap), err_msg=str(cap))
