"""Candidate tier-configuration batches and cost-model inputs.

A configuration is an (HBM, DRAM, SSD) capacity vector in granules (0 means
the tier is absent), an organisation mode and an eviction policy per tenant
group.  The planner in the paper emits such candidates on a grid (Section
4.1); the grids here are the benchmark workloads' grids.

Encodings (shared input format of the library and the oracle):

* mode:   0 = inclusive (every tier an independent cache over all
          accesses), 1 = exclusive with write-back demotion (LRU only),
          2 = inclusive with prefix reuse (a request reuses a run of its
          blocks from its first block on; LRU, shared caches only).
* policy: 0 = LRU, 1 = FIFO, 2 = LFU, 3 = radix-tree leaf-first LRU.
* partitioned: 0 = one cache per tier shared by all groups (policy[0]);
               1 = tier capacity split per group (cap_group[k][g], policy[g]).

Units: GiB = 2^30 bytes, TiB = 2^40 bytes; a capacity in bytes becomes
granules by exact division by the trace's granule size.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass

import numpy as np

MAX_GROUPS = 16

MODE_INCLUSIVE = 0
MODE_EXCLUSIVE_DEMOTE = 1
MODE_INCLUSIVE_PREFIX = 2

POLICY_LRU = 0
POLICY_FIFO = 1
POLICY_LFU = 2
POLICY_LEAF = 3

GIB = 1 << 30
TIB = 1 << 40


_FIELDS = ("cap", "cap_group", "mode", "partitioned", "policy", "segment", "disk_ttl",
           "medium", "ttl")


@dataclass
class ConfigBatch:
    cap: np.ndarray          # uint64[n,3] granules per tier (0 = absent)
    cap_group: np.ndarray    # uint64[n,3,16] per-group granules (partitioned configs)
    mode: np.ndarray         # uint8[n]
    partitioned: np.ndarray  # uint8[n]
    policy: np.ndarray       # uint8[n,16]
    segment: np.ndarray      # uint32[n] Pareto segment id
    disk_ttl: np.ndarray = None  # uint8[n]: 1 = the disk tier is a TTL tier
    medium: np.ndarray = None    # uint8[n]: disk medium index of the cost model
    ttl: np.ndarray = None       # float64[n,16]: disk TTL (s) by the block's group

    def __post_init__(self):
        n = self.cap.shape[0]
        if self.disk_ttl is None:
            self.disk_ttl = np.zeros(n, np.uint8)
        if self.medium is None:
            self.medium = np.zeros(n, np.uint8)
        if self.ttl is None:
            self.ttl = np.zeros((n, MAX_GROUPS), np.float64)

    @property
    def n(self) -> int:
        return int(self.cap.shape[0])

    def subset(self, idx) -> "ConfigBatch":
        idx = np.asarray(idx)
        return ConfigBatch(*[getattr(self, f)[idx].copy() for f in _FIELDS])

    @staticmethod
    def concat(parts) -> "ConfigBatch":
        return ConfigBatch(*[np.concatenate([getattr(p, f) for p in parts]) for f in _FIELDS])


def empty(n: int) -> ConfigBatch:
    return ConfigBatch(cap=np.zeros((n, 3), np.uint64),
                       cap_group=np.zeros((n, 3, MAX_GROUPS), np.uint64),
                       mode=np.zeros(n, np.uint8), partitioned=np.zeros(n, np.uint8),
                       policy=np.zeros((n, MAX_GROUPS), np.uint8),
                       segment=np.zeros(n, np.uint32))


def from_list(items) -> ConfigBatch:
    """Build a batch from dicts: {cap:(h,d,s), mode, policy, partitioned, cap_group, segment}."""
    b = empty(len(items))
    for i, it in enumerate(items):
        b.cap[i] = np.asarray(it["cap"], dtype=np.uint64)
        b.mode[i] = it.get("mode", MODE_INCLUSIVE)
        b.partitioned[i] = it.get("partitioned", 0)
        pol = it.get("policy", POLICY_LRU)
        if np.isscalar(pol):
            b.policy[i, :] = pol
        else:
            pol = np.asarray(pol, dtype=np.uint8)
            b.policy[i, :len(pol)] = pol
        if "cap_group" in it:
            cg = np.asarray(it["cap_group"], dtype=np.uint64)
            b.cap_group[i, :, :cg.shape[1]] = cg
        b.segment[i] = it.get("segment", 0)
        if "ttl" in it:
            b.disk_ttl[i] = 1
            t = it["ttl"]
            if np.isscalar(t):
                b.ttl[i, :] = float(t)
            else:
                t = np.asarray(t, dtype=np.float64)
                b.ttl[i, :len(t)] = t
        b.medium[i] = it.get("medium", 0)
    return b


def _granules(nbytes: float, granule_bytes: int) -> int:
    q = nbytes / granule_bytes
    if q != int(q):
        raise ValueError("capacity is not a whole number of granules")
    return int(q)


def grid(hbm_gib, dram_gib, ssd_tib, granule_bytes, mode=MODE_INCLUSIVE,
         policy=POLICY_LRU, segment=0) -> ConfigBatch:
    pts = list(itertools.product(hbm_gib, dram_gib, ssd_tib))
    b = empty(len(pts))
    for i, (h, d, s) in enumerate(pts):
        b.cap[i] = (_granules(h * GIB, granule_bytes), _granules(d * GIB, granule_bytes),
                    _granules(s * TIB, granule_bytes))
    b.mode[:] = mode
    b.policy[:, :] = policy
    b.segment[:] = segment
    return b


def split_capacity(c: int, n_groups: int) -> np.ndarray:
    """floor(C/G) granules per group, remainder +1 to the lowest-index groups."""
    q, r = divmod(int(c), n_groups)
    out = np.full(n_groups, q, dtype=np.uint64)
    out[:r] += 1
    return out


def tiny_configs(granule_bytes) -> ConfigBatch:
    """64 = HBM {1,2,4,8} GiB x DRAM {0,64,256,1024} GiB x SSD {0,1,2,4} TiB, LRU."""
    return grid([1, 2, 4, 8], [0, 64, 256, 1024], [0, 1, 2, 4], granule_bytes)


def chat_configs(granule_bytes) -> ConfigBatch:
    """512 = 8 x 8 x 8 capacity grid, LRU on every tier."""
    return grid([1, 2, 4, 8, 16, 32, 64, 128], [0, 16, 32, 64, 128, 256, 512, 1024],
                [0, 0.25, 0.5, 1, 2, 4, 8, 16], granule_bytes)


def tenant_configs(granule_bytes, n_groups=8, seed=2, n_assign=100) -> ConfigBatch:
    """10 capacity points x 100 per-group policy assignments, partitioned.

    The assignments are the three uniform ones plus distinct random draws
    from {LRU, FIFO, LFU}^8.
    """
    rng = np.random.default_rng([seed, 1])
    assign = [tuple([p] * n_groups) for p in (POLICY_LRU, POLICY_FIFO, POLICY_LFU)]
    seen = set(assign)
    while len(assign) < n_assign:
        a = tuple(int(x) for x in rng.integers(0, 3, n_groups))
        if a not in seen:
            seen.add(a)
            assign.append(a)
    caps = list(itertools.product([1, 2, 4, 8, 16], [0, 128], [0.5]))
    items = []
    for (h, d, s) in caps:
        c = (_granules(h * GIB, granule_bytes), _granules(d * GIB, granule_bytes),
             _granules(s * TIB, granule_bytes))
        cg = np.stack([split_capacity(x, n_groups) for x in c])
        for a in assign:
            items.append({"cap": c, "cap_group": cg, "partitioned": 1, "policy": a})
    return from_list(items)


def longctx_configs(granule_bytes) -> ConfigBatch:
    """2,048 = 8 x 16 x 16 grid up to TB scale, LRU with write-back demotion."""
    hbm = [1, 2, 4, 8, 16, 32, 64, 128]
    dram = [0, 64, 128, 256, 384, 512, 768, 1024, 1536, 2048, 3072, 4096, 6144, 8192,
            12288, 16384]
    ssd = [0, 1, 2, 4, 6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 192, 256]
    return grid(hbm, dram, ssd, granule_bytes, mode=MODE_EXCLUSIVE_DEMOTE)


def full_configs(granule_bytes, seed=4, n_replay=1000) -> ConfigBatch:
    """10,000 LRU grid points (25 x 20 x 20) + 1,000 FIFO/LFU replay points.

    The replay points are grid points sampled without replacement; the first
    half run FIFO, the second half LFU; all inclusive and shared.  Segment id
    = policy code, so a segmented Pareto pass gives one front per policy.
    """
    hbm = [4 * (i + 1) for i in range(25)]
    dram = [128 * i for i in range(20)]
    ssd = [0.5 * i for i in range(20)]
    lru = grid(hbm, dram, ssd, granule_bytes, policy=POLICY_LRU, segment=POLICY_LRU)
    rng = np.random.default_rng([seed, 1])
    pick = rng.choice(lru.n, size=n_replay, replace=False)
    rep = lru.subset(pick)
    half = n_replay // 2
    rep.policy[:half, :] = POLICY_FIFO
    rep.policy[half:, :] = POLICY_LFU
    rep.segment[:half] = POLICY_FIFO
    rep.segment[half:] = POLICY_LFU
    return ConfigBatch.concat([lru, rep])


def chat_leaf_configs(granule_bytes) -> ConfigBatch:
    """The chat grid under radix-tree (leaf-first) eviction on every tier."""
    return grid([1, 2, 4, 8, 16, 32, 64, 128], [0, 16, 32, 64, 128, 256, 512, 1024],
                [0, 0.25, 0.5, 1, 2, 4, 8, 16], granule_bytes, policy=POLICY_LEAF)


def chat_ttl_configs(granule_bytes) -> ConfigBatch:
    """64 = HBM {1, 4, 16, 64} GiB x DRAM {0, 64, 256, 1024} GiB x disk TTL
    {0, 60, 600, 3600} s: LRU HBM and DRAM over an unbounded TTL disk tier."""
    items = []
    for h, d, t in itertools.product([1, 4, 16, 64], [0, 64, 256, 1024], [0.0, 60.0, 600.0, 3600.0]):
        items.append({"cap": (_granules(h * GIB, granule_bytes), _granules(d * GIB, granule_bytes), 0),
                      "ttl": t})
    return from_list(items)


def chat_excl_configs(granule_bytes) -> ConfigBatch:
    """32 = HBM {1, 4, 16, 64} GiB x DRAM {16, 256} GiB x SSD {0, 1} TiB x
    {FIFO, LFU}: write-back-demotion (exclusive) hierarchies, which have no
    stack property under these policies and are replayed access by access."""
    parts = []
    for p in (POLICY_FIFO, POLICY_LFU):
        parts.append(grid([1, 4, 16, 64], [16, 256], [0, 1], granule_bytes,
                          mode=MODE_EXCLUSIVE_DEMOTE, policy=p, segment=p))
    return ConfigBatch.concat(parts)


def full_ttl_configs(granule_bytes) -> ConfigBatch:
    """16 = HBM {4, 40} GiB x DRAM {0, 512} GiB x disk TTL {0, 60, 600, 3600} s:
    LRU HBM and DRAM over an unbounded TTL disk tier."""
    items = []
    for h, d, t in itertools.product([4, 40], [0, 512], [0.0, 60.0, 600.0, 3600.0]):
        items.append({"cap": (_granules(h * GIB, granule_bytes), _granules(d * GIB, granule_bytes), 0),
                      "ttl": t})
    return from_list(items)


def longctx_leaf_configs(granule_bytes) -> ConfigBatch:
    """64 = HBM {1, 8, 32, 128} GiB x DRAM {0, 512, 4096, 16384} GiB x SSD
    {0, 8, 64, 256} TiB of the long-context grid, inclusive tiers under
    radix-tree (leaf-first) eviction."""
    return grid([1, 8, 32, 128], [0, 512, 4096, 16384], [0, 8, 64, 256], granule_bytes,
                policy=POLICY_LEAF)


# Workload variants: the same trace under other configuration batches.
VARIANTS = {"chat_leaf": "chat", "chat_ttl": "chat", "chat_excl": "chat", "full_ttl": "full",
            "longctx_leaf": "longctx"}


def trace_of(name: str) -> str:
    """The workload whose trace a (variant) name evaluates."""
    return VARIANTS.get(name, name)


def configs_for(name: str, trace) -> ConfigBatch:
    gb = trace.granule_bytes
    if name == "chat_leaf":
        return chat_leaf_configs(gb)
    if name == "chat_ttl":
        return chat_ttl_configs(gb)
    if name == "chat_excl":
        return chat_excl_configs(gb)
    if name == "full_ttl":
        return full_ttl_configs(gb)
    if name == "longctx_leaf":
        return longctx_leaf_configs(gb)
    if name == "tiny":
        return tiny_configs(gb)
    if name == "chat":
        return chat_configs(gb)
    if name == "tenant":
        return tenant_configs(gb, trace.n_groups)
    if name == "longctx":
        return longctx_configs(gb)
    if name == "full":
        return full_configs(gb)
    raise KeyError(name)


# Cost-model inputs (all rates per hour, bandwidths in bytes/s).  The paper's
# objective model needs profiles that are not available, so these constants
# parameterise a stated proxy: DRAM bandwidth at 20 GB/s, where the paper's
# DRAM-bandwidth sweep stops improving TTFT much (Table 1); cloud-disk
# bandwidth that grows with provisioned capacity up to a cap (Observation 5).
DEFAULT_COST = {
    "price_gpu_per_hour": 40.0,
    "price_per_gib_hour": (0.02, 0.004, 0.0002),
    "bw_dram": 20.0e9,
    "ssd_bw_base": 0.35e9,
    "ssd_bw_per_gib": 0.5e6,
    "ssd_bw_max": 4.0e9,
    "t_prefill_per_token": 1.0 / 20000.0,
}


def random_configs(seed: int, n: int, n_groups: int, w_max: int, cap_hi: int,
                   policies=(POLICY_LRU, POLICY_FIFO, POLICY_LFU), exclusive: bool = False,
                   partitioned_frac: float = 0.5, zero_frac: float = 0.25,
                   exclusive_policies=(POLICY_LRU,)) -> ConfigBatch:
    """Random candidate configurations for correctness tests.

    Capacities are 0 (absent, with probability ``zero_frac``) or uniform in
    [w_max, cap_hi]; with ``exclusive`` every configuration uses the
    exclusive hierarchy with group policies drawn from ``exclusive_policies``
    (LRU only by default), otherwise the inclusive one with random policies.
    """
    rng = np.random.default_rng([seed, 7])
    b = empty(n)

    def cap():
        if rng.random() < zero_frac:
            return 0
        return int(rng.integers(w_max, max(w_max, cap_hi) + 1))

    for i in range(n):
        caps = [cap() for _ in range(3)]
        if not any(caps):
            caps[int(rng.integers(0, 3))] = int(rng.integers(w_max, max(w_max, cap_hi) + 1))
        part = n_groups > 1 and rng.random() < partitioned_frac
        if exclusive:
            b.mode[i] = MODE_EXCLUSIVE_DEMOTE
            if len(exclusive_policies) == 1:
                pol = [exclusive_policies[0]] * MAX_GROUPS
            else:
                pol = [int(rng.choice(exclusive_policies)) for _ in range(MAX_GROUPS)]
        else:
            pol = [int(rng.choice(policies)) for _ in range(MAX_GROUPS)]
        b.policy[i] = pol
        if part:
            b.partitioned[i] = 1
            for k in range(3):
                tot = 0
                for g in range(n_groups):
                    x = cap() if caps[k] else 0
                    b.cap_group[i, k, g] = x
                    tot += x
                caps[k] = max(caps[k], tot) if tot else caps[k]
        b.cap[i] = caps
    return b
