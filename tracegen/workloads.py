"""Seeded synthetic KV-block access traces shaped like the paper's workloads.

The paper's traces A/B/C (chatbot, API, agent; two hours each, 40k-170k
requests, salted hashes of 16-token blocks; Section 3.3) are not public, so
five generators stand in for them, one per benchmark workload:

* ``tiny``     - 2,000 requests, Poisson 20/s, shared system-prompt prefix
                 (Zipf 1.1 over 100 prompts of U{256..2048} tokens) plus a
                 unique lognormal(6, 1) suffix.
* ``chat``     - 20,000 multi-turn sessions; Geometric(0.3) turns, each turn
                 re-reads the whole history plus a lognormal(5.5, 0.8) user
                 turn; exponential think time, mean 30 s.
* ``tenant``   - 8 tenant groups, each with its own Zipf prompt pool
                 (500 prompts, s from 0.8 to 1.4) and arrival rate.
* ``longctx``  - 100,000 requests reading the first U{8192..131072} tokens of
                 one of 2,000 documents (Zipf 1.0), 64-token blocks.
* ``full``     - 1M requests mixing chat/tenant/long-context 40/30/30.

Distributions: Zipf(s) over n items draws rank k with probability
proportional to k^-s (item id k-1); lognormal token counts are
max(1, rint(exp(N(mu, sigma^2)))); geometric counts live on {1, 2, ...};
Poisson arrivals are cumulative exponential gaps.  All draws come from
``numpy.random.default_rng`` (PCG64), so a (workload, seed) pair fixes the
trace bit for bit.

Requests are ordered by (arrival time, generator tag, request id); the blocks
of one request are accessed in block-index order; only full blocks are
accesses.  Output tokens are not modelled; a chat turn's history is the
concatenation of the earlier user turns.

This module generates inputs only and holds none of the evaluation
arithmetic.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from ._hash import chain_streams, mix64

# Bumped whenever a generator's output changes; stored expected values are
# keyed by it (and by a digest of the generated arrays).
GENERATOR_VERSION = 1

GRANULE_128K = 128 * 1024
GRANULE_512K = 512 * 1024
SPAN_2H = 7200.0

TAG_PROMPT = 1
TAG_SUFFIX = 2
TAG_CHAT = 3
TAG_TENANT_PROMPT = 4
TAG_DOC = 5
TAG_RANDOM = 6


@dataclass
class Trace:
    """One synthetic trace, laid out as the C ABI expects it (host copy)."""
    name: str
    hash: np.ndarray          # uint64[N] chained block hash per access
    req: np.ndarray           # uint32[N] request index per access (non-decreasing)
    group: np.ndarray         # uint8[N]  tenant group per access
    weight: np.ndarray        # uint8[N]  block size in granules per access
    req_time: np.ndarray      # float64[R] arrival time per request, non-decreasing
    n_groups: int = 1
    tokens_per_granule: int = 16
    granule_bytes: int = GRANULE_128K
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.hash.shape[0])

    @property
    def n_req(self) -> int:
        return int(self.req_time.shape[0])


# --------------------------------------------------------------------------
# distribution helpers
# --------------------------------------------------------------------------

def zipf_choice(rng: np.random.Generator, n_items: int, s: float, size: int) -> np.ndarray:
    """Zipf(s) over ``n_items``: P(rank k) proportional to k^-s; returns k-1."""
    k = np.arange(1, n_items + 1, dtype=np.float64)
    p = k ** (-float(s))
    p /= p.sum()
    return rng.choice(n_items, size=size, p=p)


def lognormal_tokens(rng: np.random.Generator, mu: float, sigma: float, size: int) -> np.ndarray:
    return np.maximum(1, np.rint(np.exp(rng.normal(mu, sigma, size)))).astype(np.int64)


def poisson_arrivals(rng: np.random.Generator, n: int, mean_gap: float) -> np.ndarray:
    return np.cumsum(rng.exponential(mean_gap, n))


# --------------------------------------------------------------------------
# per-generator request sets
# --------------------------------------------------------------------------

@dataclass
class _Requests:
    """Requests of one generator, in the generator's own id order.

    Request r reads ``len0[r]`` hashes of ``table`` from ``start0[r]``, then
    ``len1[r]`` hashes from ``start1[r]`` (a shared prefix, then its own
    continuation).
    """
    time: np.ndarray          # float64[r]
    tag: int
    table: np.ndarray         # uint64[t] hash streams of this generator
    start0: np.ndarray        # int64[r]
    len0: np.ndarray          # int64[r]
    start1: np.ndarray        # int64[r]
    len1: np.ndarray          # int64[r]
    group: np.ndarray         # uint8[r]
    weight: int


def _prompt_suffix_requests(rng, salt, tag_prompt, n_prompts, prompt_ent_base,
                            zipf_s, n_req, mean_gap, suffix_mu, suffix_sigma,
                            tokens_per_block, req_ent_base, group_id, out_tag):
    """Shared system prompt (Zipf over a prompt pool) + unique suffix."""
    prompt_len = rng.integers(256, 2048, size=n_prompts, endpoint=True)
    t = poisson_arrivals(rng, n_req, mean_gap)
    choice = zipf_choice(rng, n_prompts, zipf_s, n_req)
    suffix = lognormal_tokens(rng, suffix_mu, suffix_sigma, n_req)
    pblk = prompt_len // tokens_per_block
    p_hash, p_off = chain_streams(tag_prompt, prompt_ent_base + np.arange(n_prompts),
                                  pblk, np.full(n_prompts, salt, dtype=np.uint64))
    total = (prompt_len[choice] + suffix) // tokens_per_block
    shared = np.minimum(pblk[choice], total)
    nsuf = total - shared
    # the suffix chain continues from the last shared prompt block
    last = p_hash[p_off[choice] + shared - 1]
    s_hash, s_off = chain_streams(TAG_SUFFIX, req_ent_base + np.arange(n_req), nsuf,
                                  last, first_index=shared)
    table = np.concatenate([p_hash, s_hash])
    return _Requests(time=t, tag=out_tag, table=table, start0=p_off[choice], len0=shared,
                     start1=len(p_hash) + s_off[:-1], len1=nsuf,
                     group=np.full(n_req, group_id, dtype=np.uint8), weight=1)


def _chat_requests(rng, salt, n_sessions, n_turns_cap, span, ent_base, tag):
    """Multi-turn chat: each turn re-reads the session history."""
    start = poisson_arrivals(rng, n_sessions, span / n_sessions)
    turns = rng.geometric(0.3, n_sessions).astype(np.int64)
    if n_turns_cap is not None:
        c = np.cumsum(turns)
        keep = int(np.searchsorted(c, n_turns_cap, side="left")) + 1
        keep = min(keep, n_sessions)
        turns = turns[:keep].copy()
        start = start[:keep]
        over = int(turns.sum()) - n_turns_cap
        if over > 0:
            turns[-1] -= over
        n_sessions = keep
    n_t = int(turns.sum())
    tokens = lognormal_tokens(rng, 5.5, 0.8, n_t)
    think = rng.exponential(30.0, n_t)
    sess = np.repeat(np.arange(n_sessions), turns)
    first = np.cumsum(turns) - turns                       # first turn index per session
    tpos = np.arange(n_t) - np.repeat(first, turns)        # turn number inside the session
    cum_tok = np.cumsum(tokens)
    base_tok = np.repeat(cum_tok[first] - tokens[first], turns)
    hist_tok = cum_tok - base_tok
    gap_before = np.where(tpos == 0, 0.0, think[np.maximum(np.arange(n_t) - 1, 0)])
    cum_gap = np.cumsum(gap_before)
    base_gap = np.repeat(cum_gap[first], turns)
    t = np.repeat(start, turns) + (cum_gap - base_gap)
    nblk = hist_tok // 16
    # session stream length = blocks read by the session's last turn
    slen = nblk[first + turns - 1]
    s_hash, s_off = chain_streams(tag, ent_base + np.arange(n_sessions), slen,
                                  np.full(n_sessions, salt, dtype=np.uint64))
    z = np.zeros(n_t, dtype=np.int64)
    return _Requests(time=t, tag=tag, table=s_hash, start0=s_off[sess], len0=nblk,
                     start1=z, len1=z, group=np.zeros(n_t, dtype=np.uint8), weight=1)


def _longctx_requests(rng, salt, n_req, n_docs, span, ent_base, tag, weight):
    """Long-context reads: a prefix of a Zipf(1.0)-chosen document, 64-token blocks."""
    t = poisson_arrivals(rng, n_req, span / n_req)
    doc = zipf_choice(rng, n_docs, 1.0, n_req)
    ln = rng.integers(8192, 131072, size=n_req, endpoint=True)
    nblk = ln // 64
    dlen = np.zeros(n_docs, dtype=np.int64)
    np.maximum.at(dlen, doc, nblk)
    d_hash, d_off = chain_streams(tag, ent_base + np.arange(n_docs), dlen,
                                  np.full(n_docs, salt, dtype=np.uint64))
    z = np.zeros(n_req, dtype=np.int64)
    return _Requests(time=t, tag=tag, table=d_hash, start0=d_off[doc], len0=nblk,
                     start1=z, len1=z, group=np.zeros(n_req, dtype=np.uint8), weight=weight)


@dataclass
class Recipe:
    """A trace before expansion: hash streams plus per-request segments.

    Requests are already in trace order; request r reads table[start0[r]:
    start0[r]+len0[r]] then table[start1[r]: start1[r]+len1[r]].
    ``expand`` materialises the per-access arrays with torch, on the CPU or
    directly on a GPU; both give the same integers.
    """
    name: str
    table: np.ndarray
    start0: np.ndarray
    len0: np.ndarray
    start1: np.ndarray
    len1: np.ndarray
    group: np.ndarray       # uint8 per request
    weight: np.ndarray      # uint8 per request
    req_time: np.ndarray
    n_groups: int
    tokens_per_granule: int
    granule_bytes: int
    meta: dict

    @property
    def n(self) -> int:
        return int(self.len0.sum() + self.len1.sum())

    def expand(self, device="cpu", max_requests=None):
        """Per-access tensors: hash (int64 bits of the uint64 hash), req (int32),
        group (uint8), weight (uint8); plus req_time (float64)."""
        import torch
        R = len(self.len0) if max_requests is None else min(max_requests, len(self.len0))
        dev = torch.device(device)
        L0 = torch.from_numpy(self.len0[:R]).to(dev)
        L1 = torch.from_numpy(self.len1[:R]).to(dev)
        S0 = torch.from_numpy(self.start0[:R]).to(dev)
        S1 = torch.from_numpy(self.start1[:R]).to(dev)
        tot = L0 + L1
        off = torch.zeros(R + 1, dtype=torch.int64, device=dev)
        torch.cumsum(tot, 0, out=off[1:])
        n = int(off[-1])
        if n >= (1 << 32) - 1:
            raise ValueError("trace too long for 32-bit positions")
        rid = torch.repeat_interleave(torch.arange(R, device=dev), tot, output_size=n)
        pos = torch.arange(n, device=dev) - off[:-1][rid]
        first = pos < L0[rid]
        src = torch.where(first, S0[rid] + pos, S1[rid] + (pos - L0[rid]))
        table = torch.from_numpy(self.table.view(np.int64)).to(dev)
        out = {
            "hash": table[src],
            "req": rid.to(torch.int32),
            "group": torch.from_numpy(self.group[:R]).to(dev)[rid],
            "weight": torch.from_numpy(self.weight[:R]).to(dev)[rid],
            "req_time": torch.from_numpy(self.req_time[:R].copy()).to(dev),
        }
        return out

    def to_trace(self, max_requests=None) -> "Trace":
        d = self.expand("cpu", max_requests)
        return Trace(name=self.name, hash=d["hash"].numpy().view(np.uint64),
                     req=d["req"].numpy().view(np.uint32), group=d["group"].numpy(),
                     weight=d["weight"].numpy(), req_time=d["req_time"].numpy(),
                     n_groups=self.n_groups, tokens_per_granule=self.tokens_per_granule,
                     granule_bytes=self.granule_bytes, meta=dict(self.meta))


def _merge(name, parts, n_groups, tokens_per_granule, granule_bytes, meta) -> Recipe:
    """Order all requests by (time, tag, id) and concatenate the hash tables."""
    toff = np.cumsum([0] + [len(p.table) for p in parts])
    table = np.concatenate([p.table for p in parts]) if len(parts) > 1 else parts[0].table
    times = np.concatenate([p.time for p in parts])
    tags = np.concatenate([np.full(len(p.time), p.tag, dtype=np.int64) for p in parts])
    ids = np.concatenate([np.arange(len(p.time), dtype=np.int64) for p in parts])
    s0 = np.concatenate([p.start0 + toff[i] for i, p in enumerate(parts)])
    s1 = np.concatenate([p.start1 + toff[i] for i, p in enumerate(parts)])
    l0 = np.concatenate([p.len0 for p in parts])
    l1 = np.concatenate([p.len1 for p in parts])
    grp = np.concatenate([p.group for p in parts])
    wts = np.concatenate([np.full(len(p.time), p.weight, dtype=np.uint8) for p in parts])
    order = np.lexsort((ids, tags, times))
    return Recipe(name=name, table=np.ascontiguousarray(table, dtype=np.uint64),
                  start0=s0[order].astype(np.int64), len0=l0[order].astype(np.int64),
                  start1=s1[order].astype(np.int64), len1=l1[order].astype(np.int64),
                  group=grp[order].astype(np.uint8), weight=wts[order],
                  req_time=times[order].astype(np.float64), n_groups=n_groups,
                  tokens_per_granule=tokens_per_granule, granule_bytes=granule_bytes,
                  meta=meta)


def _salt(seed: int, which: int) -> np.uint64:
    return mix64(np.array([(seed << 8) | which], dtype=np.uint64))[0]


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

def tiny_recipe(seed: int = 0, n_req: int = 2000) -> Recipe:
    """2,000 requests, Poisson 20/s, Zipf(1.1) over 100 system prompts + unique suffix."""
    rng = np.random.default_rng(seed)
    part = _prompt_suffix_requests(rng, _salt(seed, 1), TAG_PROMPT, 100, 0, 1.1,
                                   n_req, 1.0 / 20.0, 6.0, 1.0, 16, 0, 0, TAG_PROMPT)
    return _merge("tiny", [part], 1, 16, GRANULE_128K, {"seed": seed, "n_req": n_req})


def chat_recipe(seed: int = 1, n_sessions: int = 20000) -> Recipe:
    """Multi-turn chat: 20,000 sessions over two hours."""
    rng = np.random.default_rng(seed)
    part = _chat_requests(rng, _salt(seed, 3), n_sessions, None, SPAN_2H, 0, TAG_CHAT)
    return _merge("chat", [part], 1, 16, GRANULE_128K, {"seed": seed, "n_sessions": n_sessions})


def _tenant_parts(rng, seed, total_req, n_groups=8, span=SPAN_2H, ent_base=0, req_base=0,
                  group_ids=True):
    parts = []
    svals = np.linspace(0.8, 1.4, n_groups)
    tri = n_groups * (n_groups + 1) // 2
    rb = req_base
    for g in range(n_groups):
        n_g = int(round(total_req * (g + 1) / tri))
        if n_g == 0:
            continue
        p = _prompt_suffix_requests(rng, _salt(seed, 16 + g), TAG_TENANT_PROMPT, 500,
                                    ent_base + g * 500, float(svals[g]), n_g,
                                    span / n_g, 6.0, 1.0, 16, rb,
                                    g if group_ids else 0, TAG_TENANT_PROMPT)
        rb += n_g
        parts.append(p)
    return parts


def tenant_recipe(seed: int = 2, total_req: int = 100000, n_groups: int = 8) -> Recipe:
    """Mixed-tenant trace: 8 groups with their own Zipf prompt pools and rates."""
    rng = np.random.default_rng(seed)
    parts = _tenant_parts(rng, seed, total_req, n_groups)
    return _merge("tenant", parts, n_groups, 16, GRANULE_128K,
                  {"seed": seed, "total_req": total_req})


def longctx_recipe(seed: int = 3, n_req: int = 100000, n_docs: int = 2000) -> Recipe:
    """Long-context/agentic trace: 64-token blocks, one granule = one 512 KiB block."""
    rng = np.random.default_rng(seed)
    part = _longctx_requests(rng, _salt(seed, 5), n_req, n_docs, SPAN_2H, 0, TAG_DOC, 1)
    return _merge("longctx", [part], 1, 64, GRANULE_512K,
                  {"seed": seed, "n_req": n_req, "n_docs": n_docs})


def full_recipe(seed: int = 4, n_req: int = 1_000_000) -> Recipe:
    """Full-scale sweep: chat/tenant/long-context mixed 40/30/30 over two hours.

    Granules are 128 KiB (16 tokens); the long-context 64-token blocks weigh
    4 granules.  All accesses share one group.
    """
    rng = np.random.default_rng(seed)
    n_chat = int(round(0.4 * n_req))
    n_ten = int(round(0.3 * n_req))
    n_long = n_req - n_chat - n_ten
    # enough sessions for the requested number of turns (mean 1/0.3 turns each)
    n_sess = int(n_chat * 0.3 * 1.3) + 16
    chat_p = _chat_requests(rng, _salt(seed, 3), n_sess, n_chat, SPAN_2H, 0, TAG_CHAT)
    ten_p = _tenant_parts(rng, seed, n_ten, 8, SPAN_2H, ent_base=0, req_base=0,
                          group_ids=False)
    long_p = _longctx_requests(rng, _salt(seed, 5), n_long, 2000, SPAN_2H, 0, TAG_DOC, 4)
    return _merge("full", [chat_p] + ten_p + [long_p], 1, 16, GRANULE_128K,
                  {"seed": seed, "n_req": n_req})


RECIPES = {
    "tiny": tiny_recipe,
    "chat": chat_recipe,
    "tenant": tenant_recipe,
    "longctx": longctx_recipe,
    "full": full_recipe,
}
WORKLOADS = tuple(RECIPES)


def recipe(name: str, seed: int | None = None, **kw) -> Recipe:
    fn = RECIPES[name]
    return fn(**kw) if seed is None else fn(seed=seed, **kw)


def make(name: str, seed: int | None = None, **kw) -> Trace:
    """Host copy of a workload trace (expanded on the CPU)."""
    return recipe(name, seed, **kw).to_trace()


def tiny(seed: int = 0, n_req: int = 2000) -> Trace:
    return tiny_recipe(seed, n_req).to_trace()


def chat(seed: int = 1, n_sessions: int = 20000) -> Trace:
    return chat_recipe(seed, n_sessions).to_trace()


def tenant(seed: int = 2, total_req: int = 100000, n_groups: int = 8) -> Trace:
    return tenant_recipe(seed, total_req, n_groups).to_trace()


def longctx(seed: int = 3, n_req: int = 100000, n_docs: int = 2000) -> Trace:
    return longctx_recipe(seed, n_req, n_docs).to_trace()


def full(seed: int = 4, n_req: int = 1_000_000) -> Trace:
    return full_recipe(seed, n_req).to_trace()


# --------------------------------------------------------------------------
# small traces for correctness tests
# --------------------------------------------------------------------------

def from_blocks(blocks, weights=None, groups=None, n_groups=1, name="hand",
                per_request=1, seed=7) -> Trace:
    """A trace from a sequence of small integer block labels.

    Label ``b`` becomes hash mix(b + salt); ``weights`` / ``groups`` give a
    per-label weight / group (dicts or arrays indexed by label).
    """
    b = np.asarray(blocks, dtype=np.int64)
    n = b.size
    salt = np.uint64((seed * 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF)
    h = mix64(b.astype(np.uint64) ^ salt)
    if weights is None:
        w = np.ones(n, dtype=np.uint8)
    else:
        wl = np.asarray([weights[int(x)] for x in b] if isinstance(weights, dict)
                        else np.asarray(weights)[b])
        w = wl.astype(np.uint8)
    if groups is None:
        g = np.zeros(n, dtype=np.uint8)
    else:
        gl = np.asarray([groups[int(x)] for x in b] if isinstance(groups, dict)
                        else np.asarray(groups)[b])
        g = gl.astype(np.uint8)
    n_req = max(1, (n + per_request - 1) // per_request)
    req = (np.arange(n) // per_request).astype(np.uint32)
    rt = np.arange(n_req, dtype=np.float64) * 0.5
    return Trace(name=name, hash=h, req=req, group=g, weight=w, req_time=rt,
                 n_groups=n_groups, tokens_per_granule=16, granule_bytes=GRANULE_128K,
                 meta={"labels": b})


def random_trace(seed: int, n: int, n_blocks: int, n_groups: int = 1,
                 weight_choices=(1,), zipf_s: float = 0.0, reuse_bias: float = 0.0,
                 per_request: int = 8) -> Trace:
    """Random trace over ``n_blocks`` labels with per-label weight and group.

    ``zipf_s`` > 0 skews label popularity; ``reuse_bias`` in [0, 1) is the
    chance that an access repeats one of the last few labels (short reuse).
    """
    rng = np.random.default_rng(seed)
    if zipf_s > 0:
        lab = zipf_choice(rng, n_blocks, zipf_s, n)
    else:
        lab = rng.integers(0, n_blocks, n)
    if reuse_bias > 0 and n > 1:
        rep = rng.random(n) < reuse_bias
        back = rng.integers(1, 6, n)
        for i in np.nonzero(rep)[0]:
            if i - back[i] >= 0:
                lab[i] = lab[i - back[i]]
    wl = rng.choice(np.asarray(weight_choices), size=n_blocks)
    gl = rng.integers(0, n_groups, n_blocks)
    t = from_blocks(lab, weights=wl, groups=gl, n_groups=n_groups, name=f"rand{seed}",
                    per_request=per_request, seed=seed + 101)
    t.req_time = np.cumsum(rng.exponential(1.0, t.n_req))
    return t
