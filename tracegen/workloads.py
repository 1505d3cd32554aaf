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
    """Requests of one generator, in the generator's own id order."""
    time: np.ndarray          # float64[r]
    tag: int
    nblk: np.ndarray          # int64[r] blocks read by each request
    flat: np.ndarray          # uint64[sum nblk] hashes, request after request
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
    # suffix chain continues from the last shared prompt block
    last = p_hash[p_off[choice] + shared - 1]
    s_hash, s_off = chain_streams(TAG_SUFFIX, req_ent_base + np.arange(n_req), nsuf,
                                  last, first_index=shared)
    # assemble request-major flat hashes
    r_off = np.zeros(n_req + 1, dtype=np.int64)
    np.cumsum(total, out=r_off[1:])
    flat = np.empty(int(r_off[-1]), dtype=np.uint64)
    # shared part: gather from the prompt table
    rid_sh = np.repeat(np.arange(n_req), shared)
    pos_sh = np.arange(rid_sh.size) - np.repeat(np.cumsum(shared) - shared, shared)
    flat[r_off[rid_sh] + pos_sh] = p_hash[p_off[choice[rid_sh]] + pos_sh]
    rid_sf = np.repeat(np.arange(n_req), nsuf)
    pos_sf = np.arange(rid_sf.size) - np.repeat(s_off[:-1], nsuf)
    flat[r_off[rid_sf] + shared[rid_sf] + pos_sf] = s_hash
    return _Requests(time=t, tag=out_tag, nblk=total, flat=flat,
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
    # cumulative tokens and times inside each session
    cum_tok = np.cumsum(tokens)
    base_tok = np.repeat(cum_tok[first] - tokens[first], turns)
    hist_tok = cum_tok - base_tok
    cum_think = np.cumsum(think)
    gap_before = np.where(tpos == 0, 0.0, think[np.maximum(np.arange(n_t) - 1, 0)])
    cum_gap = np.cumsum(gap_before)
    base_gap = np.repeat(cum_gap[first], turns)
    t = np.repeat(start, turns) + (cum_gap - base_gap)
    del cum_think
    nblk = hist_tok // 16
    # session stream length = blocks read by the session's last turn
    last_turn = first + turns - 1
    slen = nblk[last_turn]
    s_hash, s_off = chain_streams(tag, ent_base + np.arange(n_sessions), slen,
                                  np.full(n_sessions, salt, dtype=np.uint64))
    r_off = np.zeros(n_t + 1, dtype=np.int64)
    np.cumsum(nblk, out=r_off[1:])
    rid = np.repeat(np.arange(n_t), nblk)
    pos = np.arange(rid.size) - np.repeat(r_off[:-1], nblk)
    flat = s_hash[s_off[sess[rid]] + pos]
    return _Requests(time=t, tag=tag, nblk=nblk, flat=flat,
                     group=np.zeros(n_t, dtype=np.uint8), weight=1)


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
    r_off = np.zeros(n_req + 1, dtype=np.int64)
    np.cumsum(nblk, out=r_off[1:])
    total = int(r_off[-1])
    flat = np.empty(total, dtype=np.uint64)
    # chunked gather keeps peak memory bounded on large traces
    step = 1 << 22
    for a in range(0, n_req, step):
        b = min(n_req, a + step)
        nb = nblk[a:b]
        rid = np.repeat(np.arange(a, b), nb)
        pos = np.arange(rid.size, dtype=np.int64) - np.repeat(r_off[a:b] - r_off[a], nb)
        flat[r_off[a]:r_off[b]] = d_hash[d_off[doc[rid]] + pos]
    return _Requests(time=t, tag=tag, nblk=nblk, flat=flat,
                     group=np.zeros(n_req, dtype=np.uint8), weight=weight)


def _merge(name, parts, n_groups, tokens_per_granule, granule_bytes, meta):
    """Order all requests by (time, tag, id) and lay out the access arrays."""
    times = np.concatenate([p.time for p in parts])
    tags = np.concatenate([np.full(len(p.time), p.tag, dtype=np.int64) for p in parts])
    ids = np.concatenate([np.arange(len(p.time), dtype=np.int64) for p in parts])
    nblk = np.concatenate([p.nblk for p in parts])
    grp = np.concatenate([p.group for p in parts])
    wts = np.concatenate([np.full(len(p.time), p.weight, dtype=np.uint8) for p in parts])
    src = np.concatenate([p.flat for p in parts]) if len(parts) > 1 else parts[0].flat
    src_off = np.zeros(len(nblk) + 1, dtype=np.int64)
    np.cumsum(nblk, out=src_off[1:])
    order = np.lexsort((ids, tags, times))
    n_req = len(order)
    o_nblk = nblk[order]
    o_off = np.zeros(n_req + 1, dtype=np.int64)
    np.cumsum(o_nblk, out=o_off[1:])
    n = int(o_off[-1])
    if n >= (1 << 32) - 1:
        raise ValueError("trace too long for 32-bit positions")
    hashes = np.empty(n, dtype=np.uint64)
    req = np.empty(n, dtype=np.uint32)
    group = np.empty(n, dtype=np.uint8)
    weight = np.empty(n, dtype=np.uint8)
    step = 1 << 20
    for a in range(0, n_req, step):
        b = min(n_req, a + step)
        nb = o_nblk[a:b]
        loc = np.repeat(np.arange(a, b), nb)
        pos = np.arange(loc.size, dtype=np.int64) - np.repeat(o_off[a:b] - o_off[a], nb)
        sl = slice(o_off[a], o_off[b])
        hashes[sl] = src[src_off[order[loc]] + pos]
        req[sl] = loc.astype(np.uint32)
        group[sl] = grp[order[loc]]
        weight[sl] = wts[order[loc]]
    return Trace(name=name, hash=hashes, req=req, group=group, weight=weight,
                 req_time=times[order].astype(np.float64), n_groups=n_groups,
                 tokens_per_granule=tokens_per_granule, granule_bytes=granule_bytes,
                 meta=meta)


def _salt(seed: int, which: int) -> np.uint64:
    return mix64(np.array([(seed << 8) | which], dtype=np.uint64))[0]


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

def tiny(seed: int = 0, n_req: int = 2000) -> Trace:
    """2,000 requests, Poisson 20/s, Zipf(1.1) over 100 system prompts + unique suffix."""
    rng = np.random.default_rng(seed)
    part = _prompt_suffix_requests(rng, _salt(seed, 1), TAG_PROMPT, 100, 0, 1.1,
                                   n_req, 1.0 / 20.0, 6.0, 1.0, 16, 0, 0, TAG_PROMPT)
    return _merge("tiny", [part], 1, 16, GRANULE_128K, {"seed": seed, "n_req": n_req})


def chat(seed: int = 1, n_sessions: int = 20000) -> Trace:
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


def tenant(seed: int = 2, total_req: int = 100000, n_groups: int = 8) -> Trace:
    """Mixed-tenant trace: 8 groups with their own Zipf prompt pools and rates."""
    rng = np.random.default_rng(seed)
    parts = _tenant_parts(rng, seed, total_req, n_groups)
    return _merge("tenant", parts, n_groups, 16, GRANULE_128K,
                  {"seed": seed, "total_req": total_req})


def longctx(seed: int = 3, n_req: int = 100000, n_docs: int = 2000) -> Trace:
    """Long-context/agentic trace: 64-token blocks, one granule = one 512 KiB block."""
    rng = np.random.default_rng(seed)
    part = _longctx_requests(rng, _salt(seed, 5), n_req, n_docs, SPAN_2H, 0, TAG_DOC, 1)
    return _merge("longctx", [part], 1, 64, GRANULE_512K,
                  {"seed": seed, "n_req": n_req, "n_docs": n_docs})


def full(seed: int = 4, n_req: int = 1_000_000) -> Trace:
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


WORKLOADS = {
    "tiny": tiny,
    "chat": chat,
    "tenant": tenant,
    "longctx": longctx,
    "full": full,
}


def make(name: str, seed: int | None = None, **kw) -> Trace:
    fn = WORKLOADS[name]
    return fn(**kw) if seed is None else fn(seed=seed, **kw)


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
