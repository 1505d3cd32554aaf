"""Marshalling helpers around the binding: host arrays <-> device tensors.

Nothing here computes any part of the evaluation; it moves inputs to the
device, calls the library and brings results back.
"""
from __future__ import annotations

import numpy as np
import torch

from . import kvcfg


def to_device(trace, device="cuda"):
    """Device tensors for a trace object with hash/req/group/weight/req_time arrays."""
    return {
        "hash": torch.from_numpy(np.ascontiguousarray(trace.hash).view(np.int64)).to(device),
        "req": torch.from_numpy(np.ascontiguousarray(trace.req).view(np.int32)).to(device),
        "group": torch.from_numpy(np.ascontiguousarray(trace.group)).to(device),
        "weight": torch.from_numpy(np.ascontiguousarray(trace.weight)).to(device),
        "req_time": torch.from_numpy(np.ascontiguousarray(trace.req_time)).to(device),
    }


def load(trace, dev=None, stream=None):
    dev = dev or to_device(trace)
    return kvcfg.kv_trace_load(dev["hash"], dev["req"], dev["req_time"], group=dev["group"],
                               weight=dev["weight"], n_groups=trace.n_groups,
                               tokens_per_granule=trace.tokens_per_granule,
                               granule_bytes=trace.granule_bytes, stream=stream)


def config_array(cfgs):
    return kvcfg.config_array(cfgs.cap, cfgs.cap_group, cfgs.mode, cfgs.partitioned,
                              cfgs.policy, cfgs.disk_ttl, cfgs.medium, cfgs.ttl)


def cost_model(cost: dict):
    return kvcfg.cost_model(cost["price_gpu_per_hour"], cost["price_per_gib_hour"],
                            cost["bw_dram"], cost["ssd_bw_base"], cost["ssd_bw_per_gib"],
                            cost["ssd_bw_max"], cost["t_prefill_per_token"],
                            cost.get("media", ()))


def evaluate(handle, cfgs, cost: dict, n_groups: int, device="cuda", stream=None):
    """Returns (counts uint64 [n,G,3,8], obj float64 [n,3]) as numpy arrays."""
    arr, n = config_array(cfgs)
    counts = torch.zeros((n, n_groups, 3, 8), dtype=torch.int64, device=device)
    obj = torch.zeros((n, 3), dtype=torch.float64, device=device)
    kvcfg.kv_eval_configs(handle, arr, n, cost_model(cost), counts, obj, stream=stream)
    torch.cuda.synchronize()
    return counts.cpu().numpy().view(np.uint64), obj.cpu().numpy()


def pareto(obj_np, segment=None, bounds=None, device="cuda"):
    obj = torch.from_numpy(np.ascontiguousarray(obj_np, dtype=np.float64)).to(device)
    flags = torch.zeros(obj.shape[0], dtype=torch.uint8, device=device)
    seg = None
    if segment is not None:
        seg = torch.from_numpy(np.ascontiguousarray(segment, dtype=np.uint32).view(np.int32)).to(device)
    n = kvcfg.kv_pareto(obj, flags, segment=seg, bounds=bounds)
    torch.cuda.synchronize()
    return flags.cpu().numpy(), n


def ttl_curves(handle, ttl, n_groups: int, device="cuda", stream=None):
    """Returns (hits uint64 [G,K], hitw uint64 [G,K], store float64 [G,K]) as numpy arrays."""
    k = len(ttl)
    hits = torch.zeros((n_groups, k), dtype=torch.int64, device=device)
    hitw = torch.zeros((n_groups, k), dtype=torch.int64, device=device)
    store = torch.zeros((n_groups, k), dtype=torch.float64, device=device)
    kvcfg.kv_ttl_curves(handle, ttl, hits, hitw, store, stream=stream)
    torch.cuda.synchronize()
    return (hits.cpu().numpy().view(np.uint64), hitw.cpu().numpy().view(np.uint64),
            store.cpu().numpy())
