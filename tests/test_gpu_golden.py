"""Full-size parity on the five benchmark workloads.

For each workload the trace is generated on the device exactly as the
benchmark does, its arrays are digested and matched to the stored expected
values (written by ``tests/golden/make_golden.py`` from the CPU oracle
alone), and the GPU library evaluates the stored configurations (every
configuration of the tiny, chat and tenant workloads; 64 of the
long-context workload's 2,048 exclusive ones; 32 of the full workload's
11,000: its LRU grid corners and seeded draws of each policy).  Two
variants evaluate the chat trace under radix-tree (leaf-first) eviction on
its whole grid and under an HBM x DRAM x disk-TTL grid (unbounded TTL disk
tier; the objectives then include its storage integral, a double sum whose
order differs between the two sides, stored beside the counts); two more
evaluate the full workload's trace over a 16-point HBM x DRAM x disk-TTL
grid and the long-context trace under leaf-first eviction on 64 inclusive
points of its grid.  Counts must be equal element by
element; objectives match the oracle's objectives of the stored counts to
1e-6 relative; Pareto flags equal the oracle's brute force over those
objectives, in one segment and per policy.
"""
import os
import sys

import numpy as np
import pytest

import tracegen as tg
from tracegen.digest import configs_digest, trace_digest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
NAMES = ("tiny", "chat", "tenant", "longctx", "full", "chat_leaf", "chat_ttl", "chat_excl",
         "full_ttl", "longctx_leaf")
FIELDS = ("hit", "miss", "ins", "evict", "hit_w", "miss_w", "ins_w", "evict_w")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def first_mismatch(a, b):
    bad = np.argwhere(a != b)
    c, g, k, f = bad[0]
    return (f"{len(bad)} mismatching values; first: config {c} group {g} tier {k} "
            f"{FIELDS[f]}: gpu {a[c, g, k, f]} oracle {b[c, g, k, f]}")


@pytest.mark.parametrize("name", NAMES)
def test_golden_workload(name, oracle_mod):
    import torch
    from paper_2603_08739_amd import host, kvcfg as K
    O = oracle_mod
    gold = np.load(os.path.join(HERE, "golden", f"counts_{name}.npz"))
    assert int(gold["generator_version"]) == tg.GENERATOR_VERSION, "stale expected values"
    say(f"  {name}: generating the trace on the device")
    rec = tg.recipe(tg.trace_of(name))
    dev = rec.expand("cuda")
    torch.cuda.synchronize()
    hst = tg.Trace(name=name, hash=dev["hash"].cpu().numpy().view(np.uint64),
                   req=dev["req"].cpu().numpy().view(np.uint32), group=dev["group"].cpu().numpy(),
                   weight=dev["weight"].cpu().numpy(), req_time=dev["req_time"].cpu().numpy(),
                   n_groups=rec.n_groups, tokens_per_granule=rec.tokens_per_granule,
                   granule_bytes=rec.granule_bytes)
    dig = trace_digest(hst.hash, hst.req, hst.group, hst.weight, hst.req_time)
    assert dig == str(gold["trace_sha"]), f"{name}: trace digest differs from the stored one"
    cfgs = tg.configs_for(name, rec)
    assert configs_digest(cfgs) == str(gold["configs_sha"])
    idx = gold["idx"]
    sub = cfgs.subset(idx)
    say(f"  {name}: {hst.n} accesses, evaluating {sub.n} of {cfgs.n} configurations")
    h = K.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                        weight=dev["weight"], n_groups=rec.n_groups,
                        tokens_per_granule=rec.tokens_per_granule,
                        granule_bytes=rec.granule_bytes)
    counts, obj = host.evaluate(h, sub, tg.DEFAULT_COST, rec.n_groups)
    h.free()
    del dev
    ref = gold["counts"]
    assert counts.shape == ref.shape
    assert np.array_equal(counts, ref), f"{name}: " + first_mismatch(counts, ref)
    say(f"  {name}: counts equal; objectives and Pareto fronts")
    # the storage integral of unbounded disk TTL tiers comes with the stored counts
    ref_obj = O.objectives(hst, sub, ref, tg.DEFAULT_COST,
                           store=gold["store"] if "store" in gold else None)
    np.testing.assert_allclose(obj, ref_obj, rtol=1e-6, atol=0)
    for seg in (None, sub.segment):
        flags, n = host.pareto(obj, segment=seg)
        ref_flags = O.pareto(ref_obj, seg)
        assert np.array_equal(flags, ref_flags)
        assert n == int(ref_flags.sum())
    say(f"  {name}: ok")
