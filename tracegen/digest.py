"""Digests of generated inputs, so that stored expected values can be
matched to the exact trace and configuration batch they were computed from
(a change of generator, seed or batch changes the digest)."""
from __future__ import annotations

import hashlib

import numpy as np


def _feed(h, name: str, a) -> None:
    a = np.ascontiguousarray(a)
    h.update(f"{name}:{a.dtype.str}:{a.shape}".encode())
    h.update(memoryview(a).cast("B"))


def trace_digest(hash, req, group, weight, req_time) -> str:
    """sha256 over the per-access arrays and the request times (host arrays)."""
    h = hashlib.sha256()
    _feed(h, "hash", np.asarray(hash).view(np.uint64))
    _feed(h, "req", np.asarray(req).view(np.uint32))
    _feed(h, "group", np.asarray(group, dtype=np.uint8))
    _feed(h, "weight", np.asarray(weight, dtype=np.uint8))
    _feed(h, "req_time", np.asarray(req_time, dtype=np.float64))
    return h.hexdigest()


def configs_digest(cfgs) -> str:
    h = hashlib.sha256()
    for f in ("cap", "cap_group", "mode", "partitioned", "policy", "segment"):
        _feed(h, f, getattr(cfgs, f))
    return h.hexdigest()
