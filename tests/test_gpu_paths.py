"""GPU parity on code paths that only large inputs reach, forced on small
ones, plus the library's error and memory-pressure behaviour.

* The block-matrix row of a position block holds one histogram bin per
  earlier block; rows longer than the LDS histogram are built in column
  chunks with a carry, which only traces of more than 1.34e8 accesses need.
  KVCFG_TEST_ROW_CHUNK narrows the chunk so that ~1e5-access traces take
  that path (1, 3 and 8 columns per chunk).
* More thresholds than fit in LDS are binned with global atomics:
  KVCFG_TEST_THR_LDS=0 forces it, and a batch with more than 6,144 distinct
  LRU capacities reaches it without any hook.
* Replay jobs whose state exceeds a budget run in waves sharing one state
  buffer: KVCFG_TEST_REPLAY_BUDGET makes a small batch need several.
* A replay job that fails its state check is reported as KV_ERR_DEVICE by the
  next kv_trace_info on the trace: KVCFG_TEST_FAIL_JOB marks one job as
  failed while every kernel still runs to completion.
Every hook only selects among paths that compute the same result, and each
case is compared with the oracle element by element.
"""
import os
import sys

import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class env:
    def __init__(self, **kw):
        self.kw = {k: str(v) for k, v in kw.items()}

    def __enter__(self):
        self.old = {k: os.environ.get(k) for k in self.kw}
        os.environ.update(self.kw)

    def __exit__(self, *a):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def run(trace, cfgs):
    from paper_2603_08739_amd import host
    h = host.load(trace)
    counts, obj = host.evaluate(h, cfgs, tg.DEFAULT_COST, trace.n_groups)
    h.free()
    return counts, obj


def check(O, trace, cfgs, label, **hooks):
    say(f"  case {label}: n={trace.n} configs={cfgs.n} hooks={hooks}")
    with env(**hooks):
        counts, _ = run(trace, cfgs)
    ref = O.replay_memo(trace, cfgs)
    if not np.array_equal(counts, ref):
        bad = np.argwhere(counts != ref)
        c, g, k, f = bad[0]
        raise AssertionError(f"{label}: {len(bad)} mismatches; first cfg {c} group {g} tier {k} "
                             f"field {f}: gpu {counts[c, g, k, f]} oracle {ref[c, g, k, f]}")
    return counts


@pytest.mark.parametrize("chunk", [1, 3, 8])
def test_row_chunk_path(oracle_mod, chunk):
    t = tg.random_trace(77, 120_000, 30_000, weight_choices=(1, 4), zipf_s=0.6)
    cfgs = tg.from_list([{"cap": (c, d, s)} for c in (16, 600, 5000)
                         for d in (0, 9000) for s in (0, 40000, 200000)])
    check(oracle_mod, t, cfgs, f"rowchunk{chunk}", KVCFG_TEST_ROW_CHUNK=chunk)
    t2 = tg.random_trace(3 * 8192 + 77, 3 * 8192 + 77, 2500, n_groups=2, weight_choices=(1, 4),
                         zipf_s=0.9)
    cfgs2 = tg.random_configs(5, 20, 2, 4, 4000, policies=(0,))
    check(oracle_mod, t2, cfgs2, f"rowchunk{chunk}-groups", KVCFG_TEST_ROW_CHUNK=chunk)


def test_global_binning_forced(oracle_mod):
    t = tg.random_trace(31, 40_000, 6000, n_groups=3, weight_choices=(1, 4), zipf_s=0.8)
    cfgs = tg.random_configs(31, 40, 3, 4, 8000, policies=(0,))
    check(oracle_mod, t, cfgs, "thr-lds-0", KVCFG_TEST_THR_LDS=0)
    pref = tg.from_list([{"cap": (c, d, 0), "mode": tg.MODE_INCLUSIVE_PREFIX}
                         for c in (8, 64, 500) for d in (0, 3000)])
    check(oracle_mod, t, pref, "thr-lds-0-prefix", KVCFG_TEST_THR_LDS=0)


def test_many_distinct_capacities(oracle_mod):
    """More than 6,144 distinct LRU capacities in one batch (no hook)."""
    t = tg.random_trace(41, 30_000, 9000, zipf_s=0.7, reuse_bias=0.2)
    caps = np.arange(1, 2 * 3300 + 1, dtype=np.uint64)        # 6,600 distinct values
    items = [{"cap": (int(caps[2 * i]), int(caps[2 * i + 1]), 0)} for i in range(3300)]
    cfgs = tg.from_list(items)
    check(oracle_mod, t, cfgs, "6600-thresholds")


def test_replay_waves(oracle_mod):
    t = tg.random_trace(51, 20_000, 3000, n_groups=2, weight_choices=(1, 4), zipf_s=0.8)
    cfgs = tg.random_configs(51, 30, 2, 4, 3000, policies=(1, 2))
    one = check(oracle_mod, t, cfgs, "one-wave")
    # an LFU job holds 4 bytes per position: a budget of 1.5 jobs forces one
    # job per wave; a budget of one byte still runs every job (one per wave)
    for b in (6 * t.n, 1):
        two = check(oracle_mod, t, cfgs, f"waves-budget{b}", KVCFG_TEST_REPLAY_BUDGET=b)
        assert np.array_equal(one, two)


def test_replay_failure_is_reported(oracle_mod):
    from paper_2603_08739_amd import host, kvcfg as K
    t = tg.random_trace(61, 5000, 800, zipf_s=0.8)
    cfgs = tg.from_list([{"cap": (c, 0, 0), "policy": tg.POLICY_LFU} for c in (16, 64, 200)])
    h = host.load(t)
    with env(KVCFG_TEST_FAIL_JOB=1):
        host.evaluate(h, cfgs, tg.DEFAULT_COST, 1)
    with pytest.raises(K.KvError) as e:
        h.info()
    assert e.value.status == K.KV_ERR_DEVICE
    assert "replay job 1" in str(e.value) and "LFU" in str(e.value)
    h.info()  # reported once, then cleared
    counts, _ = host.evaluate(h, cfgs, tg.DEFAULT_COST, 1)
    h.info()
    h.free()
    assert np.array_equal(counts, oracle_mod.replay(t, cfgs))


def test_pareto_nan_without_count():
    """Without a count the call stays asynchronous: NaN rows are never on the
    front and never dominate; with a count the NaN is an error."""
    import torch
    from paper_2603_08739_amd import kvcfg as K
    obj = torch.tensor([[1.0, 5.0, 1.0], [float("nan"), 9.0, 0.0], [2.0, 5.0, 1.0],
                        [0.5, 1.0, 3.0]], dtype=torch.float64, device="cuda")
    flags = torch.zeros(4, dtype=torch.uint8, device="cuda")
    assert K.kv_pareto(obj, flags, want_count=False) is None
    torch.cuda.synchronize()
    assert flags.cpu().tolist() == [1, 0, 0, 1]
    with pytest.raises(K.KvError) as e:
        K.kv_pareto(obj, flags)
    assert e.value.status == K.KV_ERR_INVALID
    assert flags.cpu().tolist() == [1, 0, 0, 1]


def test_binding_rejects_bad_outputs():
    import torch
    from paper_2603_08739_amd import host, kvcfg as K
    t = tg.random_trace(3, 500, 100, n_groups=2)
    h = host.load(t)
    arr, n = host.config_array(tg.from_list([{"cap": (8, 0, 0)}] * 4))
    model = host.cost_model(tg.DEFAULT_COST)
    bad = [torch.zeros((4, 1, 3, 8), dtype=torch.int64, device="cuda"),      # one group short
           torch.zeros((4, 2, 3, 8), dtype=torch.int32, device="cuda"),      # dtype
           torch.zeros((4, 2, 8, 3), dtype=torch.int64, device="cuda").transpose(2, 3),
           torch.zeros((4, 2, 3, 8), dtype=torch.int64)]                     # host memory
    for c in bad:
        with pytest.raises(ValueError):
            K.kv_eval_configs(h, arr, n, model, c)
    good = torch.zeros((4, 2, 3, 8), dtype=torch.int64, device="cuda")
    with pytest.raises(ValueError):
        K.kv_eval_configs(h, arr, n, model, good, torch.zeros((4, 2), dtype=torch.float64,
                                                              device="cuda"))
    K.kv_eval_configs(h, arr, n, model, good)
    h.free()


def test_maximum_trace_size():
    """A trace of exactly 2^29 accesses, the library's limit (the position
    range every kernel's 32-bit positions and the stack pass's block matrix
    are sized for), checked by facts that hold exactly at any size: at
    capacity 1 an LRU cache hits exactly the immediate repeats; a capacity
    holding every block misses only the first accesses; LRU hits never fall
    as the capacity grows; inclusive tiers split the single-cache hits of
    their capacities; an exclusive LRU hierarchy of unit blocks hits like
    one LRU cache of the summed capacity in total and like its top tier's
    capacity at the top; FIFO and LFU replays conserve their counts."""
    import torch
    from paper_2603_08739_amd import host, kvcfg as K
    n = 1 << 29
    say(f"  case max-size: n={n}")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(29)
    pool = 1 << 22
    u = torch.rand(n, device="cuda", generator=gen)
    ids = (u.pow(3.0) * pool).long().clamp_(max=pool - 1)  # low ids hot
    del u
    # distinct ids -> distinct 64-bit hashes (an odd multiplier is a bijection mod 2^64)
    mult = 0x9E3779B97F4A7C15 - (1 << 64)
    hashes = ids * mult + 0x2545F4914F6CDD1D
    req = (torch.arange(n, device="cuda", dtype=torch.int64) // 64).to(torch.int32)
    req_time = torch.arange(n // 64, device="cuda", dtype=torch.float64) * 0.01
    distinct = int(torch.unique(ids).numel())
    repeats = int((ids[1:] == ids[:-1]).sum())
    del ids
    torch.cuda.synchronize()
    h = K.kv_trace_load(hashes, req, req_time)
    del hashes, req
    st = h.info()
    assert st.n == n and st.n_distinct == distinct
    say(f"  {distinct} distinct blocks, {repeats} immediate repeats")
    caps = [1, 16, 4096, 65536, 1 << 20, distinct]
    items = [{"cap": (c, 0, 0)} for c in caps]
    items += [{"cap": (4096, 65536, 1 << 20)},
              {"cap": (4096, 61440, 0), "mode": tg.MODE_EXCLUSIVE_DEMOTE},
              {"cap": (65536, 0, 0), "policy": tg.POLICY_FIFO},
              {"cap": (65536, 0, 0), "policy": tg.POLICY_LFU},
              {"cap": (distinct, 0, 0), "policy": tg.POLICY_LFU}]
    cfgs = tg.from_list(items)
    counts, _ = host.evaluate(h, cfgs, tg.DEFAULT_COST, 1)
    h.free()
    c = counts[:, 0].astype(np.int64)
    lru = c[:len(caps), 0, 0]
    assert lru[0] == repeats
    assert lru[-1] == n - distinct
    assert np.all(np.diff(lru) >= 0)
    hit = dict(zip(caps, lru))
    inc = c[len(caps)]
    assert inc[0, 0] == hit[4096] and inc[1, 0] == hit[65536] - hit[4096]
    assert inc[2, 0] == hit[1 << 20] - hit[65536]
    exc = c[len(caps) + 1]
    assert exc[0, 0] == hit[4096] and exc[0, 0] + exc[1, 0] == hit[65536]
    for r in c[len(caps) + 2:]:
        top = r[0]
        assert top[0] + top[1] == n and top[2] == top[1]      # hits + misses; every miss inserts
        assert 0 <= top[2] - top[3] <= 65536 or top[3] == 0   # what stays fits
        assert repeats <= top[0] <= n - distinct
    assert c[-1, 0, 0] == n - distinct and c[-1, 0, 3] == 0   # holds every block
    torch.cuda.empty_cache()
