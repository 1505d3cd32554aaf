"""GPU parity of the TTL retention curves (Section 4.3) against the oracle.

Hits and hit weights must be identical.  Storage integrals are sums of
w * min(t, delta) in double, added in different orders on the two sides;
for n gaps the rounding differs by at most about n * 2^-53 relative (under
1e-10 at these sizes), so they are held to 1e-9 relative.
"""
import json
import os
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu

RTOL = 1e-9
GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "ttl_hand.json")


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2603_08739_amd import host, kvcfg
    return host, kvcfg


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def check(lib, O, trace, ttl, label):
    host, _ = lib
    say(f"  case {label}: n={trace.n} groups={trace.n_groups} ttl={len(ttl)}")
    h = host.load(trace)
    hits, hitw, store = host.ttl_curves(h, ttl, trace.n_groups)
    h.free()
    rh, rw, rs = O.ttl_curves(trace, ttl)
    np.testing.assert_array_equal(hits, rh, err_msg=label)
    np.testing.assert_array_equal(hitw, rw, err_msg=label)
    np.testing.assert_allclose(store, rs, rtol=RTOL, atol=0, err_msg=label)
    return hits, hitw, store


@pytest.mark.parametrize("name", ["unit", "weighted", "two groups"])
def test_hand_worked_curves(lib, oracle_mod, name):
    gold = json.load(open(GOLD))
    case = [c for c in gold["cases"] if c["name"] == name][0]
    lab = {"A": 0, "B": 1}
    t = tg.from_blocks([lab[b] for b in gold["blocks"]],
                       weights={lab[k]: v for k, v in case["weight"].items()},
                       groups={lab[k]: v for k, v in case["group"].items()},
                       n_groups=case["n_groups"])
    t.req = np.asarray(gold["req"], dtype=np.uint32)
    t.req_time = np.asarray(gold["req_time"], dtype=np.float64)
    hits, hitw, store = check(lib, oracle_mod, t, gold["ttl"], f"hand-{name}")
    assert hits.tolist() == case["hits"] and hitw.tolist() == case["hitw"]
    assert store.tolist() == [[float(x) for x in r] for r in case["store"]]


def ttl_list(rng, trace, k):
    """Zero, repeated values, request-time differences (so that some gaps
    equal a TTL exactly) and random values past the span."""
    rt = trace.req_time
    i = rng.integers(0, len(rt), k)
    j = rng.integers(0, len(rt), k)
    diffs = np.abs(rt[i] - rt[j])
    extra = rng.uniform(0, 1.5 * (rt[-1] - rt[0]) + 1.0, k // 4 + 1)
    vals = np.concatenate([[0.0, 0.0], diffs, diffs[:3], extra])
    return np.sort(vals).tolist()


@pytest.mark.parametrize("seed", range(6))
def test_random_traces(lib, oracle_mod, seed):
    rng = np.random.default_rng(500 + seed)
    t = tg.random_trace(600 + seed, int(rng.integers(5_000, 60_000)),
                        int(rng.integers(200, 8_000)), n_groups=1 + seed % 4,
                        weight_choices=(1,) if seed % 2 else (1, 2, 4),
                        zipf_s=float(rng.choice([0.0, 0.7, 1.1])), reuse_bias=0.3)
    if seed == 3:
        t.req_time = np.floor(t.req_time)   # many equal request times: zero gaps
    check(lib, oracle_mod, t, ttl_list(rng, t, 40), f"rand{seed}")


def test_workload_shaped(lib, oracle_mod):
    rec = tg.recipe("tiny")
    t = rec.to_trace()
    rng = np.random.default_rng(7)
    check(lib, oracle_mod, t, ttl_list(rng, t, 60), "tiny-workload")


def test_most_ttl_values(lib, oracle_mod):
    rng = np.random.default_rng(11)
    t1 = tg.random_trace(700, 20_000, 3_000, n_groups=1, zipf_s=0.9, reuse_bias=0.2)
    check(lib, oracle_mod, t1, ttl_list(rng, t1, 1024)[:1024], "n_ttl=1024 G=1")
    t4 = tg.random_trace(701, 20_000, 3_000, n_groups=4, weight_choices=(1, 3), zipf_s=0.9)
    check(lib, oracle_mod, t4, ttl_list(rng, t4, 1023)[:1023], "n_ttl=1023 G=4")


def test_degenerate_traces(lib, oracle_mod):
    # every block seen once: no gaps, storage = W * t
    w = np.arange(500) % 3 + 1
    t = tg.from_blocks(list(range(500)), weights=w)
    hits, hitw, store = check(lib, oracle_mod, t, [0.0, 1.0, 1e6], "cold")
    assert hits.sum() == 0 and hitw.sum() == 0
    W = float(w.sum())
    assert store[0].tolist() == [0.0, W, W * 1e6]
    # one access
    t = tg.from_blocks([3])
    check(lib, oracle_mod, t, [0.0, 5.0], "single")
    # one block over and over in one request: every gap is zero
    t = tg.from_blocks([9] * 300, per_request=300)
    hits, _, store = check(lib, oracle_mod, t, [0.0], "zero gaps")
    assert hits[0, 0] == 299 and store[0, 0] == 0.0


def test_rejected_arguments(lib):
    import torch
    host, K = lib
    t = tg.random_trace(702, 2_000, 300, n_groups=4)
    h = host.load(t)
    hits = torch.full((4, 1024), 7, dtype=torch.int64, device="cuda")
    hitw = torch.full((4, 1024), 7, dtype=torch.int64, device="cuda")
    store = torch.full((4, 1024), 7.0, dtype=torch.float64, device="cuda")
    bad = [([], K.KV_ERR_INVALID), ([1.0, -1.0], K.KV_ERR_INVALID),
           ([0.0, float("nan")], K.KV_ERR_INVALID), ([0.0, float("inf")], K.KV_ERR_INVALID),
           ([2.0, 1.0], K.KV_ERR_INVALID), ([float(x) for x in range(1024)], K.KV_ERR_UNSUPPORTED)]
    for ttl, status in bad:
        with pytest.raises(K.KvError) as e:
            K.kv_ttl_curves(h, ttl, hits, hitw, store)
        assert e.value.status == status, ttl
    torch.cuda.synchronize()
    assert (hits == 7).all() and (hitw == 7).all() and (store == 7.0).all()
    h.free()
