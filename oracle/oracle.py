"""Python entry to the CPU oracle (``kvoracle.cpp``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg call this module; the GPU library never does, and this
module never imports the GPU library.

* :func:`replay`     literal per-configuration tiered replay -> counts
                     uint64[n_cfg, n_groups, 3, 8] with fields
                     (hit, miss, ins, evict, hit_w, miss_w, ins_w, evict_w).
* :func:`objectives` (cost, throughput, latency) per configuration.
* :func:`pareto`     non-dominated flags by brute force.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liboracle.so")
SRC = os.path.join(HERE, "kvoracle.cpp")

FIELDS = ("hit", "miss", "ins", "evict", "hit_w", "miss_w", "ins_w", "evict_w")
HIT, MISS, INS, EVICT, HIT_W, MISS_W, INS_W, EVICT_W = range(8)

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (no GPU compiler involved)."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        cmd = ["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fPIC", "-shared",
               "-pthread", SRC, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        p = ctypes.c_void_p
        lib.oracle_replay.restype = ctypes.c_int
        lib.oracle_replay.argtypes = [ctypes.c_uint64, p, p, p, ctypes.c_uint32,
                                      ctypes.c_uint32, p, p, p, p, p, ctypes.c_uint32, p]
        lib.oracle_objectives.restype = ctypes.c_int
        lib.oracle_objectives.argtypes = [ctypes.c_uint32, p, p, ctypes.c_uint32, p,
                                          ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                          ctypes.c_double, ctypes.c_uint64, p]
        lib.oracle_pareto.restype = ctypes.c_int64
        lib.oracle_pareto.argtypes = [ctypes.c_uint32, p, p, p, p]
        _lib = lib
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def replay(trace, cfgs, threads: int | None = None) -> np.ndarray:
    """Literal replay of every configuration of ``cfgs`` over ``trace``."""
    lib = _load()
    n_cfg = cfgs.n
    g = trace.n_groups
    out = np.zeros((n_cfg, g, 3, 8), dtype=np.uint64)
    h = np.ascontiguousarray(trace.hash, dtype=np.uint64)
    gr = np.ascontiguousarray(trace.group, dtype=np.uint8)
    w = np.ascontiguousarray(trace.weight, dtype=np.uint8)
    cap = np.ascontiguousarray(cfgs.cap, dtype=np.uint64)
    cg = np.ascontiguousarray(cfgs.cap_group, dtype=np.uint64)
    mode = np.ascontiguousarray(cfgs.mode, dtype=np.uint8)
    part = np.ascontiguousarray(cfgs.partitioned, dtype=np.uint8)
    pol = np.ascontiguousarray(cfgs.policy, dtype=np.uint8)
    rc = lib.oracle_replay(trace.n, _ptr(h), _ptr(gr), _ptr(w), g, n_cfg, _ptr(cap), _ptr(cg),
                           _ptr(mode), _ptr(part), _ptr(pol),
                           threads or default_threads(), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_replay rejected the batch (code {rc})")
    return out


def cost_vector(cost: dict) -> np.ndarray:
    return np.array([cost["price_gpu_per_hour"], *cost["price_per_gib_hour"],
                     cost["bw_dram"], cost["ssd_bw_base"], cost["ssd_bw_per_gib"],
                     cost["ssd_bw_max"], cost["t_prefill_per_token"]], dtype=np.float64)


def objectives(trace, cfgs, counts, cost: dict) -> np.ndarray:
    lib = _load()
    n_cfg = cfgs.n
    obj = np.zeros((n_cfg, 3), dtype=np.float64)
    cap = np.ascontiguousarray(cfgs.cap, dtype=np.uint64)
    cnt = np.ascontiguousarray(counts, dtype=np.uint64)
    cm = cost_vector(cost)
    n_w = int(trace.weight.astype(np.uint64).sum())
    span = float(trace.req_time[-1] - trace.req_time[0])
    lib.oracle_objectives(n_cfg, _ptr(cap), _ptr(cnt), trace.n_groups, _ptr(cm),
                          float(trace.granule_bytes), float(trace.tokens_per_granule),
                          span, float(trace.n_req), n_w, _ptr(obj))
    return obj


def pareto(obj, segment=None, bounds=None) -> np.ndarray:
    lib = _load()
    o = np.ascontiguousarray(obj, dtype=np.float64)
    n = o.shape[0]
    seg = None if segment is None else np.ascontiguousarray(segment, dtype=np.uint32)
    b = None if bounds is None else np.ascontiguousarray(bounds, dtype=np.float64)
    flag = np.zeros(n, dtype=np.uint8)
    rc = lib.oracle_pareto(n, _ptr(o), _ptr(seg), _ptr(b), _ptr(flag))
    if rc < 0:
        raise ValueError("NaN objective")
    return flag
