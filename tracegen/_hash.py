"""64-bit block-hash chains for synthetic KV-block traces.

A trace names each 16-token (or 64-token) KV block by a salted 64-bit hash of
its whole prefix, as the paper's traces do (Section 3.3, trace description:
salted hash blocks of 16 tokens).  The chain used here is

    h[-1] = salt,   h[j] = mix(h[j-1] XOR mix(content[j]))

where ``mix`` is the splitmix64 output finaliser (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014) and
``content[j]`` packs (generator tag, stream entity, block index) into one
word.  Two accesses carry the same hash exactly when they read the same block
of the same prefix stream, so shared prefixes share hashes.

This module is input generation only: it holds none of the cache-evaluation
arithmetic, and both the GPU library and the CPU oracle consume its output.
"""
from __future__ import annotations

import numpy as np

_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_S30 = np.uint64(30)
_S27 = np.uint64(27)
_S31 = np.uint64(31)


def mix64(z: np.ndarray) -> np.ndarray:
    """splitmix64 finaliser, element-wise on a uint64 array (wraps mod 2^64)."""
    z = np.asarray(z, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z ^= z >> _S30
        z *= _M1
        z ^= z >> _S27
        z *= _M2
        z ^= z >> _S31
    return z


def content_word(tag: int, entity: np.ndarray, j) -> np.ndarray:
    """(tag:8 | entity:36 | block index:20) packed into one uint64 word."""
    ent = np.asarray(entity, dtype=np.uint64)
    jj = np.asarray(j, dtype=np.uint64)
    if np.any(ent >= np.uint64(1 << 36)):
        raise ValueError("entity id exceeds 36 bits")
    if np.any(jj >= np.uint64(1 << 20)):
        raise ValueError("block index exceeds 20 bits")
    return (np.uint64(tag) << np.uint64(56)) | (ent << np.uint64(20)) | jj


def chain_streams(tag: int, entity: np.ndarray, length: np.ndarray,
                  start: np.ndarray, first_index: np.ndarray | None = None
                  ) -> tuple[np.ndarray, np.ndarray]:
    """Hash chains for many streams at once.

    Stream ``s`` has ``length[s]`` blocks whose block indices run from
    ``first_index[s]`` (default 0); its chain starts from ``start[s]`` (the
    salt, or the hash of the block before the stream).  Returns the flat hash
    array (streams concatenated in input order) and the per-stream offsets.
    """
    entity = np.asarray(entity, dtype=np.uint64)
    length = np.asarray(length, dtype=np.int64)
    n = len(length)
    if first_index is None:
        first_index = np.zeros(n, dtype=np.int64)
    first_index = np.asarray(first_index, dtype=np.int64)
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(length, out=offsets[1:])
    out = np.empty(int(offsets[-1]), dtype=np.uint64)
    if n == 0 or offsets[-1] == 0:
        return out, offsets
    # Walk block index j over streams sorted by decreasing length so that the
    # active streams at step j are always a prefix of the sorted order.
    order = np.argsort(-length, kind="stable")
    ls = length[order]
    ent = entity[order]
    off = offsets[:-1][order]
    fi = first_index[order]
    h = np.asarray(start, dtype=np.uint64)[order].copy()
    maxlen = int(ls[0])
    # number of streams with length > j, for every j
    active_counts = n - np.searchsorted(ls[::-1], np.arange(maxlen), side="right")
    for j in range(maxlen):
        k = int(active_counts[j])
        c = mix64(content_word(tag, ent[:k], fi[:k] + j))
        h[:k] = mix64(h[:k] ^ c)
        out[off[:k] + j] = h[:k]
    return out, offsets
