"""ctypes binding of libkvcfg (include/kvcfg.h): argument marshalling only.

Every computation runs in the HIP library; this module converts torch device
tensors and numpy host arrays into the C structs and pointers of the ABI.
PyTorch serves as the device allocator and the source of the current HIP
stream.  If the compiled library is missing the import fails: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvcfg.so")

KV_OK, KV_ERR_INVALID, KV_ERR_NOMEM, KV_ERR_DEVICE, KV_ERR_UNSUPPORTED = 0, -1, -2, -3, -4
KV_MAX_GROUPS, KV_TIERS, KV_FIELDS = 16, 3, 8
KV_MODE_INCLUSIVE, KV_MODE_EXCLUSIVE_DEMOTE, KV_MODE_INCLUSIVE_PREFIX = 0, 1, 2
KV_POLICY_LRU, KV_POLICY_FIFO, KV_POLICY_LFU, KV_POLICY_LEAF = 0, 1, 2, 3
FIELDS = ("hit", "miss", "ins", "evict", "hit_w", "miss_w", "ins_w", "evict_w")

_u64, _u32, _u8, _f64, _vp = (ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint8,
                              ctypes.c_double, ctypes.c_void_p)


class kv_trace_desc(ctypes.Structure):
    _fields_ = [("n", _u64), ("hash", _vp), ("req", _vp), ("group", _vp), ("weight", _vp),
                ("n_req", _u32), ("req_time", _vp), ("n_groups", _u32),
                ("tokens_per_granule", _u32), ("granule_bytes", _u64)]


class kv_trace_stats(ctypes.Structure):
    _fields_ = [("n", _u64), ("n_distinct", _u64), ("n_w", _u64), ("distinct_w", _u64),
                ("n_g", _u64 * KV_MAX_GROUPS), ("n_w_g", _u64 * KV_MAX_GROUPS),
                ("u_g", _u64 * KV_MAX_GROUPS), ("u_w_g", _u64 * KV_MAX_GROUPS),
                ("max_multiplicity", _u64), ("n_req", _u32), ("n_groups", _u32),
                ("w_min", _u32), ("w_max", _u32), ("span", _f64)]


KV_MAX_MEDIA = 4
CONFIG_BYTES = 560


class kv_config(ctypes.Structure):
    _fields_ = [("cap", _u64 * KV_TIERS), ("cap_group", (_u64 * KV_MAX_GROUPS) * KV_TIERS),
                ("mode", _u8), ("partitioned", _u8), ("policy", _u8 * KV_MAX_GROUPS),
                ("disk_ttl", _u8), ("medium", _u8), ("reserved", _u8 * 4),
                ("ttl", _f64 * KV_MAX_GROUPS)]


class kv_disk_medium(ctypes.Structure):
    _fields_ = [("price_per_gib_hour", _f64), ("bw_base", _f64), ("bw_per_gib", _f64),
                ("bw_max", _f64)]


class kv_cost_model(ctypes.Structure):
    _fields_ = [("price_gpu_per_hour", _f64), ("price_per_gib_hour", _f64 * KV_TIERS),
                ("bw_dram", _f64), ("ssd_bw_base", _f64), ("ssd_bw_per_gib", _f64),
                ("ssd_bw_max", _f64), ("t_prefill_per_token", _f64), ("n_media", _u32),
                ("reserved", _u32), ("media", kv_disk_medium * KV_MAX_MEDIA)]


KV_STAGES = 17
STAGE_NAMES = ("load_validate", "load_sort", "load_links", "partition", "stack_matrix",
               "stack_local", "stack_assemble", "stack_final", "lru_counts", "replay_init",
               "replay_lfu", "replay_combine", "objectives", "pareto", "replay_fifo",
               "ttl_curves", "replay_excl")


class kv_timing(ctypes.Structure):
    _fields_ = [("calls", _u64 * KV_STAGES), ("ms", _f64 * KV_STAGES)]


assert ctypes.sizeof(kv_config) == CONFIG_BYTES


class KvError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"[{status}] {msg}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2603_08739_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    lib.kv_trace_load.restype = ctypes.c_int
    lib.kv_trace_load.argtypes = [ctypes.POINTER(kv_trace_desc), _vp, ctypes.POINTER(_vp)]
    lib.kv_trace_free.restype = ctypes.c_int
    lib.kv_trace_free.argtypes = [_vp]
    lib.kv_trace_info.restype = ctypes.c_int
    lib.kv_trace_info.argtypes = [_vp, ctypes.POINTER(kv_trace_stats)]
    lib.kv_eval_configs.restype = ctypes.c_int
    lib.kv_eval_configs.argtypes = [_vp, _vp, _u32, ctypes.POINTER(kv_cost_model), _vp, _vp, _vp]
    lib.kv_pareto.restype = ctypes.c_int
    lib.kv_pareto.argtypes = [_vp, _vp, _u32, _vp, _vp, ctypes.POINTER(_u32), _vp]
    lib.kv_ttl_curves.restype = ctypes.c_int
    lib.kv_ttl_curves.argtypes = [_vp, _vp, _u32, _vp, _vp, _vp, _vp]
    lib.kv_ttl_curves_noalloc.restype = ctypes.c_int
    lib.kv_ttl_curves_noalloc.argtypes = [_vp, _vp, _u32, _vp, _vp, _vp, _vp]
    lib.kv_last_error.restype = ctypes.c_char_p
    lib.kv_last_error.argtypes = []
    lib.kv_timing_enable.restype = ctypes.c_int
    lib.kv_timing_enable.argtypes = [ctypes.c_int]
    lib.kv_timing_read.restype = ctypes.c_int
    lib.kv_timing_read.argtypes = [ctypes.POINTER(kv_timing), ctypes.c_int]
    return lib


LIB = _load()
EXPORTS = ("kv_trace_load", "kv_trace_free", "kv_trace_info", "kv_eval_configs", "kv_pareto",
           "kv_ttl_curves", "kv_ttl_curves_noalloc", "kv_last_error", "kv_timing_enable",
           "kv_timing_read")


def kv_timing_enable(on: bool = True):
    _check(LIB.kv_timing_enable(1 if on else 0))


def kv_timing_read(reset: bool = True) -> dict:
    """{stage name: (launches, device ms)} since the last reset."""
    t = kv_timing()
    _check(LIB.kv_timing_read(ctypes.byref(t), 1 if reset else 0))
    return {STAGE_NAMES[i]: (int(t.calls[i]), float(t.ms[i])) for i in range(KV_STAGES)}


def kv_last_error() -> str:
    return LIB.kv_last_error().decode()


def _check(status: int):
    if status != KV_OK:
        raise KvError(status, kv_last_error())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t, name, dtypes, numel, optional=False):
    """Checks that a tensor the library writes or reads on the device is a
    contiguous CUDA tensor of an allowed dtype holding at least `numel`
    elements (the library trusts the pointer it is given)."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}; expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements; the call needs {numel}")
    return _ptr(t)


def _dt():
    import torch
    i64 = (torch.int64, torch.uint64) if hasattr(torch, "uint64") else (torch.int64,)
    i32 = (torch.int32, torch.uint32) if hasattr(torch, "uint32") else (torch.int32,)
    return i64, i32, (torch.uint8,), (torch.float64,)


class Trace:
    """A device-resident canonical trace (owns the kv_trace handle)."""

    def __init__(self, handle):
        self.handle = handle
        self.n_groups = int(self.info().n_groups)

    def info(self) -> kv_trace_stats:
        st = kv_trace_stats()
        _check(LIB.kv_trace_info(self.handle, ctypes.byref(st)))
        return st

    def free(self):
        if self.handle is not None:
            _check(LIB.kv_trace_free(self.handle))
            self.handle = None

    def __del__(self):
        try:
            if self.handle is not None:
                LIB.kv_trace_free(self.handle)
        except Exception:
            pass


def kv_trace_load(hash, req, req_time, group=None, weight=None, n_groups=1,
                  tokens_per_granule=16, granule_bytes=128 * 1024, stream=None) -> Trace:
    """hash: int64/uint64 device tensor [n]; req: int32 [n]; req_time: float64 [n_req];
    group, weight: uint8 [n] or None."""
    i64, i32, u8, f64 = _dt()
    n = int(hash.numel())
    d = kv_trace_desc()
    d.n = n
    d.hash = _dev(hash, "hash", i64, n)
    d.req = _dev(req, "req", i32, n)
    d.group = _dev(group, "group", u8, n, optional=True)
    d.weight = _dev(weight, "weight", u8, n, optional=True)
    d.n_req = int(req_time.numel())
    d.req_time = _dev(req_time, "req_time", f64, d.n_req)
    d.n_groups = int(n_groups)
    d.tokens_per_granule = int(tokens_per_granule)
    d.granule_bytes = int(granule_bytes)
    h = ctypes.c_void_p()
    _check(LIB.kv_trace_load(ctypes.byref(d), _stream(stream), ctypes.byref(h)))
    return Trace(h)


def config_array(cap, cap_group, mode, partitioned, policy, disk_ttl=None, medium=None,
                 ttl=None):
    """numpy arrays (n,3) (n,3,16) (n,) (n,) (n,16) [(n,) (n,) (n,16)] -> ctypes kv_config[n]."""
    n = int(np.asarray(cap).shape[0])
    arr = (kv_config * max(n, 1))()
    raw = np.frombuffer(arr, dtype=np.uint8).reshape(max(n, 1), CONFIG_BYTES)
    if n:
        raw[:n, 0:24] = np.ascontiguousarray(cap, dtype=np.uint64).view(np.uint8).reshape(n, 24)
        raw[:n, 24:408] = np.ascontiguousarray(cap_group, dtype=np.uint64).view(
            np.uint8).reshape(n, 384)
        raw[:n, 408] = np.asarray(mode, dtype=np.uint8)
        raw[:n, 409] = np.asarray(partitioned, dtype=np.uint8)
        raw[:n, 410:426] = np.asarray(policy, dtype=np.uint8)
        raw[:n, 426] = 0 if disk_ttl is None else np.asarray(disk_ttl, dtype=np.uint8)
        raw[:n, 427] = 0 if medium is None else np.asarray(medium, dtype=np.uint8)
        raw[:n, 428:432] = 0
        if ttl is not None:
            raw[:n, 432:560] = np.ascontiguousarray(ttl, dtype=np.float64).view(
                np.uint8).reshape(n, 128)
    return arr, n


def cost_model(price_gpu_per_hour, price_per_gib_hour, bw_dram, ssd_bw_base, ssd_bw_per_gib,
               ssd_bw_max, t_prefill_per_token, media=()) -> kv_cost_model:
    """media: sequence of (price_per_gib_hour, bw_base, bw_per_gib, bw_max) tuples."""
    m = kv_cost_model()
    if len(media) > KV_MAX_MEDIA:
        raise ValueError("too many disk media")
    m.n_media = len(media)
    for i, md in enumerate(media):
        m.media[i].price_per_gib_hour, m.media[i].bw_base, m.media[i].bw_per_gib, \
            m.media[i].bw_max = [float(x) for x in md]
    m.price_gpu_per_hour = price_gpu_per_hour
    for k in range(3):
        m.price_per_gib_hour[k] = price_per_gib_hour[k]
    m.bw_dram = bw_dram
    m.ssd_bw_base = ssd_bw_base
    m.ssd_bw_per_gib = ssd_bw_per_gib
    m.ssd_bw_max = ssd_bw_max
    m.t_prefill_per_token = t_prefill_per_token
    return m


def kv_eval_configs(trace: Trace, cfg_arr, n_cfg: int, model: kv_cost_model, counts, obj=None,
                    stream=None):
    """counts: int64/uint64 device tensor [n_cfg, n_groups, 3, 8]; obj: float64 [n_cfg, 3]."""
    i64, _, _, f64 = _dt()
    n_cfg = int(n_cfg)
    if n_cfg > len(cfg_arr):
        raise ValueError("n_cfg exceeds the configuration array")
    pc = _dev(counts, "counts", i64, n_cfg * trace.n_groups * KV_TIERS * KV_FIELDS)
    po = _dev(obj, "obj", f64, n_cfg * 3, optional=True)
    _check(LIB.kv_eval_configs(trace.handle, ctypes.cast(cfg_arr, _vp), n_cfg,
                               ctypes.byref(model), pc, po, _stream(stream)))


def kv_pareto(obj, on_front, segment=None, bounds=None, want_count=True, stream=None):
    """obj: float64 device [n,3]; on_front: uint8 device [n]; segment: int32/uint32 device [n]."""
    _, i32, u8, f64 = _dt()
    n = int(obj.shape[0])
    if obj.dim() != 2 or obj.shape[1] != 3:
        raise ValueError("obj must have shape [n, 3]")
    po = _dev(obj, "obj", f64, 3 * n)
    pf = _dev(on_front, "on_front", u8, n)
    ps = _dev(segment, "segment", i32, n, optional=True)
    b = None
    if bounds is not None:
        barr = (ctypes.c_double * 3)(*[float(x) for x in bounds])
        b = ctypes.cast(barr, _vp)
    cnt = _u32(0)
    _check(LIB.kv_pareto(po, ps, n, b, pf, ctypes.byref(cnt) if want_count else None,
                         _stream(stream)))
    return int(cnt.value) if want_count else None


def kv_ttl_curves(trace: Trace, ttl, hits, hitw, store, stream=None):
    """ttl: host sequence of float seconds (non-decreasing); hits, hitw: int64/uint64
    device tensors [n_groups, n_ttl]; store: float64 device [n_groups, n_ttl]."""
    i64, _, _, f64 = _dt()
    vals = [float(x) for x in ttl]
    arr = (ctypes.c_double * max(len(vals), 1))(*vals)
    m = trace.n_groups * len(vals)
    ph = _dev(hits, "hits", i64, m)
    pw = _dev(hitw, "hitw", i64, m)
    pst = _dev(store, "store", f64, m)
    _check(LIB.kv_ttl_curves(trace.handle, ctypes.cast(arr, _vp), len(vals), ph, pw, pst,
                             _stream(stream)))


def kv_ttl_curves_noalloc(trace: Trace, ttl, hits, hitw, store, stream=None):
    """kv_ttl_curves without device allocation (the library's scratch array);
    the TTL values are staged in a host array that lives until the stream
    has completed the call."""
    i64, _, _, f64 = _dt()
    vals = [float(x) for x in ttl]
    arr = (ctypes.c_double * max(len(vals), 1))(*vals)
    m = trace.n_groups * len(vals)
    ph = _dev(hits, "hits", i64, m)
    pw = _dev(hitw, "hitw", i64, m)
    pst = _dev(store, "store", f64, m)
    _check(LIB.kv_ttl_curves_noalloc(trace.handle, ctypes.cast(arr, _vp), len(vals), ph, pw, pst,
                                     _stream(stream)))
    return arr
