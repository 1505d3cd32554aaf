"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments before touching the device (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvcfg.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:kv_status|const char\*)\s+(kv_\w+)\s*\(", text,
                                 re.M)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(["kv_trace_load", "kv_trace_free", "kv_trace_info",
                                           "kv_eval_configs", "kv_pareto", "kv_ttl_curves",
                                           "kv_ttl_curves_noalloc",
                                           "kv_last_error", "kv_timing_enable",
                                           "kv_timing_read"])


def test_library_exports_every_declared_symbol():
    from paper_2603_08739_amd import kvcfg
    for name in declared_functions():
        assert hasattr(kvcfg.LIB, name), name
        assert name in kvcfg.EXPORTS
    assert ctypes.sizeof(kvcfg.kv_config) == 560


def test_struct_layouts_match_header():
    """Field offsets of the ctypes mirrors agree with the C compiler's."""
    import subprocess
    import tempfile
    src = r'''
#include <stddef.h>
#include <stdio.h>
#include "kvcfg.h"
int main(void) {
  printf("%zu %zu %zu %zu\n", sizeof(kv_trace_desc), sizeof(kv_trace_stats),
         sizeof(kv_config), sizeof(kv_cost_model));
  printf("%zu %zu %zu %zu\n", offsetof(kv_trace_desc, n_req), offsetof(kv_trace_desc, req_time),
         offsetof(kv_trace_desc, granule_bytes), offsetof(kv_trace_stats, span));
  printf("%zu %zu %zu\n", offsetof(kv_config, mode), offsetof(kv_config, policy),
         offsetof(kv_cost_model, t_prefill_per_token));
  printf("%zu %zu %zu %zu %zu\n", offsetof(kv_config, disk_ttl), offsetof(kv_config, medium),
         offsetof(kv_config, ttl), offsetof(kv_cost_model, n_media),
         offsetof(kv_cost_model, media));
  return 0;
}
'''
    from paper_2603_08739_amd import kvcfg as K
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        exe = os.path.join(d, "t")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), c, "-o", exe], check=True)
        out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split()
    got = [int(x) for x in out]
    want = [ctypes.sizeof(K.kv_trace_desc), ctypes.sizeof(K.kv_trace_stats),
            ctypes.sizeof(K.kv_config), ctypes.sizeof(K.kv_cost_model),
            K.kv_trace_desc.n_req.offset, K.kv_trace_desc.req_time.offset,
            K.kv_trace_desc.granule_bytes.offset, K.kv_trace_stats.span.offset,
            K.kv_config.mode.offset, K.kv_config.policy.offset,
            K.kv_cost_model.t_prefill_per_token.offset, K.kv_config.disk_ttl.offset,
            K.kv_config.medium.offset, K.kv_config.ttl.offset, K.kv_cost_model.n_media.offset,
            K.kv_cost_model.media.offset]
    assert got == want


def test_host_side_validation_without_device():
    from paper_2603_08739_amd import kvcfg as K
    lib = K.LIB
    h = ctypes.c_void_p()
    assert lib.kv_trace_load(None, None, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert "desc" in K.kv_last_error()
    d = K.kv_trace_desc()
    d.n = 0
    assert lib.kv_trace_load(ctypes.byref(d), None, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert h.value is None
    d.n = 10
    d.n_req = 1
    d.n_groups = 17
    d.hash = d.req = d.req_time = ctypes.c_void_p(16)
    d.tokens_per_granule = 16
    d.granule_bytes = 1
    assert lib.kv_trace_load(ctypes.byref(d), None, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert "n_groups" in K.kv_last_error()
    d.n = (1 << 29) + 1
    d.n_groups = 1
    assert lib.kv_trace_load(ctypes.byref(d), None, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert lib.kv_trace_free(None) == K.KV_OK
    # a pointer that is not a live handle is refused, never dereferenced
    assert lib.kv_trace_free(ctypes.c_void_p(0x1000)) == K.KV_ERR_INVALID
    st = K.kv_trace_stats()
    assert lib.kv_trace_info(ctypes.c_void_p(0x1000), ctypes.byref(st)) == K.KV_ERR_INVALID
    m = K.cost_model(1.0, (0, 0, 0), 1.0, 1.0, 0.0, 1.0, 1.0)
    assert lib.kv_eval_configs(None, None, 0, ctypes.byref(m), None, None, None) == K.KV_ERR_INVALID
    assert lib.kv_eval_configs(ctypes.c_void_p(0x1000), None, 1, ctypes.byref(m), None, None,
                               None) == K.KV_ERR_INVALID
    n = ctypes.c_uint32(7)
    assert lib.kv_pareto(None, None, 0, None, None, ctypes.byref(n), None) == K.KV_OK
    assert n.value == 0
    assert lib.kv_pareto(None, None, 5, None, None, None, None) == K.KV_ERR_INVALID
    assert lib.kv_pareto(ctypes.c_void_p(16), None, (1 << 26) + 1, None, ctypes.c_void_p(16),
                         None, None) == K.KV_ERR_INVALID
    ttl = (ctypes.c_double * 2)(0.0, 1.0)
    assert lib.kv_ttl_curves(None, ttl, 2, ctypes.c_void_p(16), ctypes.c_void_p(16),
                             ctypes.c_void_p(16), None) == K.KV_ERR_INVALID
    assert lib.kv_ttl_curves(ctypes.c_void_p(0x1000), ttl, 2, ctypes.c_void_p(16),
                             ctypes.c_void_p(16), ctypes.c_void_p(16), None) == K.KV_ERR_INVALID
    assert "live" in K.kv_last_error()
