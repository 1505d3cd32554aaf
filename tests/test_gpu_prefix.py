"""GPU parity of the prefix-reuse hierarchy (inclusive LRU tiers where a
request reuses only a run of its blocks from its first block on) against
the oracle, element by element, in batches mixed with the plain inclusive
mode; and the unsupported combinations."""
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu

P = tg.MODE_INCLUSIVE_PREFIX


@pytest.fixture(scope="module")
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2603_08739_amd import host, kvcfg
    return host, kvcfg


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def compare(lib, O, t, cfgs, label):
    host, _ = lib
    say(f"  case {label}: n={t.n} groups={t.n_groups} configs={cfgs.n}")
    h = host.load(t)
    counts, obj = host.evaluate(h, cfgs, tg.DEFAULT_COST, t.n_groups)
    h.free()
    ref = O.replay(t, cfgs)
    if not np.array_equal(counts, ref):
        bad = np.argwhere(counts != ref)
        c, g, k, f = bad[0]
        raise AssertionError(f"{label}: {len(bad)} mismatches; first cfg={c} group={g} tier={k} "
                             f"field={f}: gpu={counts[c, g, k, f]} oracle={ref[c, g, k, f]} "
                             f"cap={cfgs.cap[c]} mode={cfgs.mode[c]}")
    np.testing.assert_allclose(obj, O.objectives(t, cfgs, ref, tg.DEFAULT_COST), rtol=1e-6,
                               atol=0)
    return counts


def batch(caps):
    items = []
    for c in caps:
        items += [{"cap": c, "mode": 0}, {"cap": c, "mode": P}]
    return tg.from_list(items)


@pytest.mark.parametrize("seed", range(6))
def test_random_traces(lib, oracle_mod, seed):
    rng = np.random.default_rng(800 + seed)
    t = tg.random_trace(900 + seed, int(rng.integers(5_000, 40_000)),
                        int(rng.integers(300, 5_000)), n_groups=1 + seed % 3,
                        weight_choices=(1,) if seed % 2 else (1, 2, 4), zipf_s=0.9,
                        reuse_bias=0.3, per_request=int(rng.integers(1, 40)))
    u = 4
    caps = [(u * int(rng.integers(1, 200)), u * int(rng.integers(0, 800)),
             u * int(rng.integers(0, 3000))) for _ in range(10)]
    caps += [(u * 50, 0, 0), (0, u * 300, 0), (u * 400, u * 100, 0)]
    counts = compare(lib, oracle_mod, t, batch(caps), f"prefix{seed}")
    plain, pref = counts[0::2], counts[1::2]
    # prefix reuse never serves more, and stores the same
    assert (pref[..., 0].sum(axis=-1) <= plain[..., 0].sum(axis=-1)).all()
    np.testing.assert_array_equal(pref[..., 2:4], plain[..., 2:4])


def test_workload_shaped(lib, oracle_mod):
    t = tg.tiny(n_req=800)
    caps = [(c1, c2, c3) for c1 in (512, 4096) for c2 in (0, 8192, 30000) for c3 in (0, 60000)]
    compare(lib, oracle_mod, t, batch(caps), "tiny-prefix")


def test_unsupported(lib):
    host, K = lib
    t = tg.random_trace(950, 2_000, 200, n_groups=2)
    h = host.load(t)
    for bad in [{"cap": (8, 0, 0), "mode": P, "policy": 1},
                {"cap": (8, 0, 0), "mode": P, "policy": 2}]:
        with pytest.raises(K.KvError) as e:
            host.evaluate(h, tg.from_list([bad]), tg.DEFAULT_COST, 2)
        assert e.value.status == K.KV_ERR_UNSUPPORTED, bad
    part = tg.from_list([{"cap": (8, 0, 0), "mode": P}])
    part.partitioned[:] = 1
    part.cap_group[0, 0, :2] = 4
    with pytest.raises(K.KvError) as e:
        host.evaluate(h, part, tg.DEFAULT_COST, 2)
    assert e.value.status == K.KV_ERR_UNSUPPORTED
    h.free()


def test_request_ids_with_gaps(lib, oracle_mod):
    """Request indices may skip values (requests without blocks): every
    request still starts where its first block is."""
    rng = np.random.default_rng(5)
    t = tg.random_trace(960, 6_000, 700, zipf_s=0.8, reuse_bias=0.3, per_request=7)
    gaps = rng.integers(1, 4, int(t.req[-1]) + 1).cumsum()   # request r -> r-th id with gaps
    t.req = gaps[t.req].astype(np.uint32)
    t.req_time = np.sort(rng.uniform(0, 100, int(t.req[-1]) + 3))
    caps = [(c, d, 0) for c in (16, 64, 256) for d in (0, 512)]
    compare(lib, oracle_mod, t, batch(caps), "prefix-gaps")
