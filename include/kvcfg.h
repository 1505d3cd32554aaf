/* kvcfg.h - batched KV-cache tier-configuration evaluation on one MI355X.
 *
 * Kareto (arXiv 2603.08739) searches storage configurations for an LLM
 * service's KV cache by replaying a historical trace of KV-block hashes
 * through a model of the HBM / DRAM / disk hierarchy and comparing the
 * candidates on (cost, throughput, latency) (Eq. 1, Eq. 2; Section 4.1).
 * This library is that inner loop, batched: it evaluates many candidate
 * configurations over one device-resident trace and filters the
 * non-dominated ones.
 *
 *   kv_trace_load    canonicalise a trace of block hashes (once per trace)
 *   kv_eval_configs  per configuration: exact per-tier hit / miss / insert /
 *                    eviction counts, then (cost, throughput, latency)
 *   kv_pareto        non-dominated filter under optional bounds
 *   kv_ttl_curves    per group, hits and storage cost of a disk tier that
 *                    keeps blocks for a time-to-live, for many TTLs at once
 *
 * Conventions for every call:
 *   - Return KV_OK or a negative kv_status; kv_last_error() then describes
 *     the failure (thread-local).  No C++ exception crosses this interface.
 *   - Arguments are validated before any device work; on a validation
 *     failure no output is touched and nothing is allocated or leaked.
 *   - "device" pointers are HIP device allocations on the current device;
 *     "host" pointers are ordinary process memory.  The library keeps no
 *     pointer to caller memory after a call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Device work is
 *     enqueued on it; device outputs are valid once the stream has completed.
 *   - Capacities and weights are in granules; a granule is the unit KV block
 *     size of the trace (e.g. 16 tokens = 128 KiB).
 */
#ifndef KVCFG_H
#define KVCFG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum kv_status {
  KV_OK = 0,
  KV_ERR_INVALID = -1,     /* argument or data violates this contract        */
  KV_ERR_NOMEM = -2,       /* device memory exhausted (nothing left allocated) */
  KV_ERR_DEVICE = -3,      /* a HIP runtime or kernel-launch error            */
  KV_ERR_UNSUPPORTED = -4  /* well-formed request outside the supported set   */
} kv_status;

enum { KV_MAX_GROUPS = 16, KV_TIERS = 3, KV_FIELDS = 8 };

/* Tier organisation of a configuration. */
enum {
  /* Every tier is an independent cache that sees every access; an access is
   * served by the fastest tier holding its block, then each tier applies its
   * own hit or insert (with eviction) rule. */
  KV_MODE_INCLUSIVE = 0,
  /* Hierarchy with write-back demotion: a block lives in at most one tier;
   * a hit in a lower tier promotes the block to the top tier, and an
   * overfull tier demotes its victim to the next tier (dropping it past the
   * last tier).  A block entering a tier (a miss, a promotion, a demotion)
   * is that tier's newest member - LRU: most recently used; FIFO: newest
   * insertion; LFU: count 1, touched now (one touch sequence per
   * hierarchy) - and the tier passes its own victims down, each entering
   * the next tier the same way, before it admits the block.  LRU over blocks
   * of one weight is evaluated as a split stack; FIFO, LFU and LRU over
   * mixed weights replay the trace once per configuration, one access after
   * another (about a microsecond per access and configuration: meant for
   * traces of up to some millions of accesses).  Not with LEAF, prefix
   * reuse or a disk TTL tier. */
  KV_MODE_EXCLUSIVE_DEMOTE = 1,
  /* The inclusive hierarchy with prefix reuse, as in a radix-tree KV cache
   * (blocks are prefix-chained, Section 3.2): contents evolve exactly as in
   * KV_MODE_INCLUSIVE, but a request reuses only a run of its blocks from
   * its first block on.  Per tier, block j of a request is available iff
   * the tier holds it and block j-1 of the same request was available there
   * (the first block needs only presence); the access is served by the
   * fastest tier where it is available.  Insert and evict counts are those
   * of KV_MODE_INCLUSIVE.  Requires LRU and a shared (non-partitioned)
   * configuration. */
  KV_MODE_INCLUSIVE_PREFIX = 2
};

/* Eviction policy of a tier cache.  A miss inserts the block after evicting
 * victims until used + w <= capacity.  LRU evicts the least recently used
 * block (Section 2.1 names LRU); FIFO the oldest insertion; LFU the smallest
 * (in-cache access count, last access position) - the count starts at 1 on
 * insertion and is forgotten on eviction.  LEAF is the eviction of a radix
 * (prefix-tree) KV cache (Section 3.2): a request's blocks form a chain, the
 * parent of a block being the block accessed just before it in the same
 * request; a cached block is a leaf when no cached block has it as parent,
 * and the victim is the leaf whose latest access is the oldest.  LEAF needs
 * a trace whose requests are prefix chains (a block is re-accessed only in a
 * later request, always after the same parent block) and tier capacities
 * that each hold the heaviest request; it is supported in the inclusive
 * mode on shared tiers, without a disk TTL tier. */
enum { KV_POLICY_LRU = 0, KV_POLICY_FIFO = 1, KV_POLICY_LFU = 2, KV_POLICY_LEAF = 3 };

/* Record fields of kv_eval_configs' counts, per (config, group, tier).
 *   hit    accesses served by this tier
 *   miss   accesses that reached this tier (no faster tier served them) and
 *          were not served by it
 *   ins    blocks inserted into this tier (tier-local misses in the
 *          inclusive mode; arrivals by promotion or demotion otherwise)
 *   evict  blocks that left this tier for lack of room (demotions count),
 *          charged to the evicted block's group
 *   *_w    the same, summed in granules
 * A tier of capacity 0 is absent and records zeros. */
enum {
  KV_F_HIT = 0, KV_F_MISS = 1, KV_F_INS = 2, KV_F_EVICT = 3,
  KV_F_HIT_W = 4, KV_F_MISS_W = 5, KV_F_INS_W = 6, KV_F_EVICT_W = 7
};

/* A trace of KV-block accesses in time order: the paper's traces carry, per
 * request, its arrival time and the salted hashes of its KV blocks
 * (Section 3.3 and Section 4.1).  All arrays are device pointers.  Blocks of
 * one request are listed in block-index order; each distinct hash must carry
 * one weight and one group throughout. */
typedef struct kv_trace_desc {
  uint64_t n;                  /* accesses; 1 <= n <= 2^29                   */
  const uint64_t* hash;        /* [n] block hash per access                  */
  const uint32_t* req;         /* [n] request index, non-decreasing, < n_req */
  const uint8_t* group;        /* [n] tenant group < n_groups, or NULL (= 0) */
  const uint8_t* weight;       /* [n] block size in granules >= 1, or NULL (= 1) */
  uint32_t n_req;              /* requests; >= 1                             */
  const double* req_time;      /* [n_req] arrival time in seconds, non-decreasing */
  uint32_t n_groups;           /* 1..16                                      */
  uint32_t tokens_per_granule; /* >= 1                                       */
  uint64_t granule_bytes;      /* >= 1                                       */
} kv_trace_desc;

typedef struct kv_trace kv_trace; /* opaque, device-resident canonical trace */

typedef struct kv_trace_stats {
  uint64_t n;                        /* accesses                              */
  uint64_t n_distinct;               /* distinct blocks U                     */
  uint64_t n_w;                      /* total weight of all accesses          */
  uint64_t distinct_w;               /* total weight of distinct blocks       */
  uint64_t n_g[KV_MAX_GROUPS];       /* accesses per group                    */
  uint64_t n_w_g[KV_MAX_GROUPS];     /* weight per group                      */
  uint64_t u_g[KV_MAX_GROUPS];       /* distinct blocks per group             */
  uint64_t u_w_g[KV_MAX_GROUPS];     /* distinct weight per group             */
  uint64_t max_multiplicity;         /* most accesses to one block            */
  uint32_t n_req, n_groups;
  uint32_t w_min, w_max;             /* smallest / largest block weight       */
  double span;                       /* req_time[n_req-1] - req_time[0]       */
} kv_trace_stats;

/* One candidate configuration (the planner's candidates, Section 4.1). */
typedef struct kv_config {
  uint64_t cap[KV_TIERS];            /* granules per tier, HBM/DRAM/SSD; 0 = absent.
                                        Each nonzero capacity must be >= the
                                        trace's largest block weight.         */
  uint64_t cap_group[KV_TIERS][KV_MAX_GROUPS]; /* partitioned: per-group capacity of
                                        each tier; sum over groups <= cap[k]  */
  uint8_t mode;                      /* KV_MODE_*                             */
  uint8_t partitioned;               /* 0: one cache per tier shared by all groups,
                                        policy[0]; 1: group g owns cap_group[k][g]
                                        of tier k and uses policy[g]          */
  uint8_t policy[KV_MAX_GROUPS];     /* KV_POLICY_* (same policy on every tier) */
  uint8_t disk_ttl;                  /* 1: tier 2 (disk) is a TTL tier (below);
                                        0: an ordinary capacity tier           */
  uint8_t medium;                    /* disk medium: index into the cost model's
                                        media (0 when it has none)            */
  uint8_t reserved[4];               /* must be 0                             */
  double ttl[KV_MAX_GROUPS];         /* disk TTL tier: seconds a block stays on
                                        disk after each access, by the block's
                                        group (shared configurations too)     */
} kv_config;

/* The disk TTL tier (Section 4.1 planner: a TTL for KV blocks on disk;
 * Section 4.3: a block is kept for the TTL after each access).  With
 * disk_ttl = 1, tier 2 holds a block while the time since its latest access
 * is at most ttl[g] (g = the block's group; a re-access at a gap delta hits
 * iff delta <= ttl[g]):
 *   - cap[2] == 0: unbounded; the tier's storage is billed as its mean
 *     occupancy over the trace span, S / span granules, where S is the
 *     storage-time integral sum over blocks of w_b * (ttl + sum of
 *     min(ttl, gap) over the block's re-access gaps) (C_g(t) of Section 4.3);
 *   - cap[2] > 0: also bounded by cap[2] granules, least recently accessed
 *     block first (with one TTL the blocks expire in that order too), billed
 *     as provisioned capacity; every group needs the same ttl.
 * Its records: hit / miss as for any tier; ins = accesses that found the
 * block absent from the tier (it is written again); evict = blocks that left
 * the tier before the trace's last access (expired or displaced), i.e. ins
 * minus the blocks still held at the time of the last access's request.
 * Requires KV_MODE_INCLUSIVE, LRU on every tier and a shared configuration. */

/* A disk medium (e.g. cloud SSD classes that differ in price and I/O
 * bandwidth, Section 4.1 planner). */
typedef struct kv_disk_medium {
  double price_per_gib_hour;         /* >= 0                                  */
  double bw_base;                    /* bytes/s at zero capacity, > 0         */
  double bw_per_gib;                 /* extra bytes/s per provisioned GiB, >= 0 */
  double bw_max;                     /* bytes/s cap, > 0                      */
} kv_disk_medium;

enum { KV_MAX_MEDIA = 4 };

/* Inputs of the objective proxy (all > 0). */
typedef struct kv_cost_model {
  double price_gpu_per_hour;         /* compute price per wall-clock hour     */
  double price_per_gib_hour[KV_TIERS]; /* capacity price per GiB per hour (>= 0) */
  double bw_dram;                    /* DRAM -> HBM bytes/s                   */
  double ssd_bw_base;                /* disk bytes/s at zero capacity         */
  double ssd_bw_per_gib;             /* extra disk bytes/s per provisioned GiB */
  double ssd_bw_max;                 /* disk bytes/s cap                      */
  double t_prefill_per_token;        /* seconds to recompute one token's KV   */
  uint32_t n_media;                  /* 0: the disk is priced by the fields
                                        above; else media[kv_config.medium]
                                        replaces price_per_gib_hour[2] and the
                                        ssd_bw_* fields                       */
  uint32_t reserved;                 /* must be 0                             */
  kv_disk_medium media[KV_MAX_MEDIA];
} kv_cost_model;

/* Canonicalise a trace (Section 4.1: the simulator replays request arrival
 * times and token-level KV-block hashes).  Reads the caller's device arrays
 * during the call only and builds, on the device, dense block ids and the
 * previous/next occurrence of every access.  On success *out owns device
 * memory until kv_trace_free.  Errors: KV_ERR_INVALID for bad sizes, a group
 * >= n_groups, a zero weight, a hash seen with two weights or two groups, or
 * a non-monotone req / req_time; *out is then NULL. */
kv_status kv_trace_load(const kv_trace_desc* desc, void* stream, kv_trace** out);

/* Free a trace (NULL is accepted).  A handle already freed is detected and
 * rejected with KV_ERR_INVALID while its memory has not been reused. */
kv_status kv_trace_free(kv_trace* t);

/* Copy the trace's summary statistics into a host struct (synchronous).
 * Also waits for the latest kv_eval_configs call on the trace and returns
 * KV_ERR_DEVICE (with *out filled) if one of its FIFO/LFU replay jobs failed
 * the replay's internal state check, in which case that call's counts are
 * invalid; kv_last_error() names the job (policy, capacity, group).  A
 * failure is reported once, by whichever call on the trace sees it first. */
kv_status kv_trace_info(const kv_trace* t, kv_trace_stats* out);

/* Evaluate n_cfg configurations over the trace (the simulator's per-candidate
 * evaluation, Section 4.1; objectives after Eq. 1 and Eq. 2).
 *   cfg     host [n_cfg]
 *   model   host
 *   counts  device uint64 [n_cfg][n_groups][3][8], fields KV_F_* (required)
 *   obj     device double [n_cfg][3] = (cost, throughput, latency), or NULL
 * Counts are exact.  Objectives, per configuration, with H_w[k] = granules
 * served by tier k (all groups), I_w = granules inserted into the disk tier,
 * R_w = N_w - sum H_w, gb = granule bytes, tpg = tokens per granule:
 *   capGiB[k] = cap[k]*gb/2^30;  bw_ssd = min(ssd_bw_base + ssd_bw_per_gib*capGiB[2], ssd_bw_max)
 *   T_busy = R_w*tpg*t_prefill_per_token + H_w[1]*gb/bw_dram + (H_w[2]+I_w)*gb/bw_ssd
 *   T_wall = max(span, T_busy)
 *   cost = (price_gpu_per_hour + sum_k capGiB[k]*price_per_gib_hour[k]) * T_wall/3600
 *   throughput = N_w*tpg/T_wall (tokens/s);  latency = T_busy/n_req (s)
 * evaluated left to right in IEEE double without contraction.  An unbounded
 * disk TTL tier takes capGiB[2] = (S*gb/2^30)/span (its mean occupancy; 0
 * when span is 0), S its storage-time integral summed in double in an order
 * of the library's choosing; with media, price_per_gib_hour[2] and the
 * ssd_bw_* terms are those of media[cfg.medium].
 * FIFO/LFU tiers are replayed once per distinct (order, group, policy,
 * capacity); when the replay state of all of them (4 bytes per access per LFU
 * job, 4 bytes per distinct block per FIFO job) does not fit in device
 * memory, the jobs run in consecutive waves that share one state buffer.
 * Errors: KV_ERR_INVALID for a capacity in (0, w_max), partitioned capacities
 * that exceed cap[k], an unknown mode or policy, nonzero reserved bytes, a
 * nonpositive cost-model rate, n_media > KV_MAX_MEDIA, a medium >= n_media
 * (when n_media > 0, else nonzero), disk_ttl > 1, or a disk TTL that is
 * negative or not finite; KV_ERR_UNSUPPORTED for a disk TTL tier outside
 * the inclusive LRU shared mode or bounded with unequal group TTLs, for more
 * than 1,024 distinct TTLs per group in one call, for LEAF outside the
 * inclusive shared mode, on a trace whose requests are not prefix chains,
 * of more than 2^28 accesses or of total weight 2^31 granules or more, or
 * with a nonzero capacity below the heaviest request, for the exclusive
 * mode with FIFO/LFU or with blocks of different weights, and for the
 * prefix-reuse mode with FIFO/LFU or partitioned capacities; KV_ERR_NOMEM when not even
 * one replay job's state fits; KV_ERR_DEVICE when an earlier call's replay
 * failure (see kv_trace_info) has already arrived.  n_cfg == 0 is a no-op. */
kv_status kv_eval_configs(const kv_trace* t, const kv_config* cfg, uint32_t n_cfg,
                          const kv_cost_model* model, uint64_t* counts, double* obj,
                          void* stream);

/* Pareto-based selection (Section 4.1): on_front[i] = 1 iff row i satisfies
 * the bounds and no other bounded row of the same segment dominates it, where
 * a dominates b when a.cost <= b.cost, a.throughput >= b.throughput and
 * a.latency <= b.latency with at least one strict.  Equal rows are all kept.
 *   obj       device double [n][3]
 *   segment   device uint32 [n] or NULL (one segment)
 *   bounds    host double [3] or NULL: cost <= b0, throughput >= b1,
 *             latency <= b2; NaN disables a bound
 *   on_front  device uint8 [n]
 *   n_front   host, or NULL; when non-NULL the call waits for the stream and
 *             stores the number of flagged rows
 * A row with a NaN objective is never on the front and never dominates.
 * Without n_front the call is asynchronous and cannot report a NaN: such rows
 * simply get flag 0 and dominate nothing.  Calls on different streams of one
 * device take turns (they share the device's result counters).
 * Errors: KV_ERR_INVALID for NULL obj/on_front with n > 0, or n > 2^26; when
 * n_front is non-NULL, also KV_ERR_INVALID if any objective is NaN (flags are
 * still written).  n == 0 is a no-op (n_front = 0). */
kv_status kv_pareto(const double* obj, const uint32_t* segment, uint32_t n,
                    const double* bounds, uint8_t* on_front, uint32_t* n_front,
                    void* stream);

/* TTL retention curves of the disk tier (Section 4.3: the cumulative hits
 * H_g(t) and storage cost C_g(t) of a group under a time-to-live t, the
 * inputs of the ROI-aware group TTL).  A block stays on disk for ttl seconds
 * after each access, so an access hits iff its block's previous access lies
 * at most ttl seconds before it (inclusive).  With delta_i = req_time[req[i]]
 * - req_time[req[p]] for the previous access p of the same block (an access
 * without one has no delta), per group g and TTL ttl[k]:
 *   hits[g][k]  = #{ accesses i of g with a delta : delta_i <= ttl[k] }
 *   hitw[g][k]  = sum of w_i over those accesses (granules)
 *   store[g][k] = W_g*ttl[k] + sum over accesses i of g with a delta of
 *                 w_i*min(ttl[k], delta_i)
 * in granule-seconds: the storage-time integral of g's blocks, each kept ttl
 * after every access including its last (W_g = u_w_g of kv_trace_stats).
 * With unit weights hits and store are the paper's H_g(t) and C_g(t).
 *   ttl    host double [n_ttl]: finite, >= 0, non-decreasing
 *   hits   device uint64 [n_groups][n_ttl]
 *   hitw   device uint64 [n_groups][n_ttl]
 *   store  device double [n_groups][n_ttl]
 * hits and hitw are exact.  store is evaluated as
 * W_g*t + S + t*(P_g - hitw[g][k]), S the sum of w_i*delta_i over the hits
 * and P_g the summed weight of g's accesses with a delta, the sums of
 * w_i*delta_i in double in an order of the library's choosing.  Device
 * outputs are valid once the stream has completed.
 * Errors: KV_ERR_INVALID for a NULL argument, n_ttl == 0, or a ttl value
 * that is negative, not finite or below its predecessor;
 * KV_ERR_UNSUPPORTED when n_groups * (n_ttl + 1) > 4096. */
kv_status kv_ttl_curves(const kv_trace* t, const double* ttl, uint32_t n_ttl, uint64_t* hits,
                        uint64_t* hitw, double* store, void* stream);

/* kv_ttl_curves for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, checks and results, but the TTL values and the gap
 * histograms live in a fixed per-device scratch array of the library (about
 * 104 KiB, held by every device the library runs on until the process ends),
 * so the call makes no hipMalloc, hipFree or other allocating call.
 *   - At most 4096 histogram bins: n_groups * (n_ttl + 1) <= 4096 and
 *     n_ttl <= 1024, else KV_ERR_UNSUPPORTED.
 *   - ttl (host) is copied to the device through `stream`; keep it unchanged
 *     until the stream has reached this call.
 *   - Every call on one device shares that device's scratch array: calls
 *     that overlap on one device (concurrent streams or threads) race and
 *     must be serialised by the caller.  Each call clears what it needs. */
kv_status kv_ttl_curves_noalloc(const kv_trace* t, const double* ttl, uint32_t n_ttl,
                                uint64_t* hits, uint64_t* hitw, double* store, void* stream);

/* Message describing the calling thread's most recent failure ("" if none). */
const char* kv_last_error(void);

/* Device-time observability.  While enabled, every call records a pair of
 * HIP events on its stream around each stage below; kv_timing_read waits for
 * the recorded events and returns, per stage, the number of launches and the
 * summed device milliseconds between each pair.  Process-wide; not meant for
 * concurrent callers.  Stages:
 *   0 load: validation        1 load: radix sort       2 load: links and ids
 *   3 group-partitioned order 4 stack: block matrix    5 stack: in-block sort
 *   6 stack: assembly, bins   7 stack: final depths    8 LRU records
 *   9 replay: job setup       10 replay: LFU jobs      11 replay: combine
 *   12 objectives             13 Pareto filter         14 replay: FIFO jobs
 *   15 TTL curves             16 replay: exclusive hierarchies
 * The replay kernels run on streams of their own, concurrently with the LRU
 * stages, so stage times may overlap. */
enum { KV_STAGES = 17 };
typedef struct kv_timing {
  uint64_t calls[KV_STAGES];
  double ms[KV_STAGES];
} kv_timing;

kv_status kv_timing_enable(int on);
/* Fill *out (host) with the totals since the last reset; reset if `reset`. */
kv_status kv_timing_read(kv_timing* out, int reset);

#ifdef __cplusplus
}
#endif

#endif /* KVCFG_H */
