"""kv_ttl_curves_noalloc against kv_ttl_curves, through the C ABI.

The variant keeps its TTL values and gap histograms in the library's
per-device scratch array instead of the trace's workspace, and allocates no
device memory.  Two calls in a row, the second with a smaller input (fewer
groups, fewer TTLs, a shorter trace), must each give the existing entry
point's results: hits and hit weights exactly, storage to 1e-9 relative (the
double sums of weight * gap are accumulated in a scheduling-dependent
order).  Sizes beyond the scratch array are refused.
"""
import numpy as np
import pytest

import tracegen as tg

pytestmark = pytest.mark.gpu


def curves(K, h, ttl, G, noalloc):
    import torch
    k = len(ttl)
    hits = torch.zeros((G, k), dtype=torch.int64, device="cuda")
    hitw = torch.zeros((G, k), dtype=torch.int64, device="cuda")
    store = torch.full((G, k), -1.0, dtype=torch.float64, device="cuda")
    if noalloc:
        keep = K.kv_ttl_curves_noalloc(h, ttl, hits, hitw, store)
    else:
        K.kv_ttl_curves(h, ttl, hits, hitw, store)
    torch.cuda.synchronize()
    if noalloc:
        del keep
    return hits.cpu().numpy(), hitw.cpu().numpy(), store.cpu().numpy()


def test_noalloc_matches_ttl_curves():
    from paper_2603_08739_amd import host, kvcfg as K
    cases = [
        (tg.random_trace(11, 60_000, 9000, n_groups=4, weight_choices=(1, 4), zipf_s=0.8),
         list(np.linspace(0.0, 80_000.0, 1000))),   # 4 x 1001 = 4,004 bins (near the limit)
        (tg.random_trace(12, 7_000, 900, n_groups=2, weight_choices=(1,), zipf_s=0.5),
         [0.0, 1.0, 5.0, 30.0, 600.0]),
    ]
    for t, ttl in cases:
        h = host.load(t)
        a = curves(K, h, ttl, t.n_groups, noalloc=False)
        b = curves(K, h, ttl, t.n_groups, noalloc=True)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        np.testing.assert_allclose(b[2], a[2], rtol=1e-9, atol=0)
        h.free()


def test_noalloc_rejects_oversize():
    from paper_2603_08739_amd import host, kvcfg as K
    t = tg.random_trace(13, 2_000, 300, n_groups=5)
    h = host.load(t)
    with pytest.raises(K.KvError) as e:
        curves(K, h, list(range(1000)), 5, noalloc=True)          # 5 x 1001 > 4,096 bins
    assert e.value.status == K.KV_ERR_UNSUPPORTED
    h.free()
