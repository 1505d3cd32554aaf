// k_excl.hip - exclusive (write-back demotion) hierarchies replayed access by
// access: FIFO and LFU tiers, and LRU tiers over blocks of mixed weights.
//
// In the tier hierarchy of a KV cache (Section 4.1's DRAM and disk below
// HBM) a block can live in one tier at a time: a hit in a lower tier
// promotes the block to the top tier, and a tier that overflows demotes its
// victim to the next tier, dropping it past the last one.  With LRU tiers
// and blocks of one weight the hierarchy is a split stack (one stack pass
// serves it); with other policies, or with mixed weights (a tier evicts
// until the block fits), it is not, and each configuration is replayed in
// trace order here.  A block entering a tier (a miss, a promotion, a
// demotion) is that tier's newest member - LRU: most recently used; FIFO:
// newest insertion; LFU: count 1, touched now - and the tier passes its own
// victims down before it admits the block.
//
// One wavefront per configuration: its lanes stage slices of the trace
// (block id, weight, group) in LDS, and its first lane walks them in order.
// The block state (tier, list links, LFU bucket of the block) is indexed by
// the trace's dense block ids in device memory; the list ends, the used
// weight of every (hierarchy, tier), the counters and the records of the
// first 2,048 LFU buckets stay in LDS.  The walk records which live tier
// served each access; all lanes turn a slice's records into hit, miss and
// insertion counts at once, so the walk itself counts only evictions.  LRU and FIFO
// tiers are doubly linked lists, oldest first; an LFU tier is a list of
// count buckets in increasing count, each a list of its blocks oldest touch
// first, so that the victim (least count, then least recent touch) heads the
// first bucket and every update takes a constant number of steps.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr uint32_t kNil = 0xFFFFFFFFu;
constexpr uint8_t kNoTier = 0xFF;
constexpr uint32_t kNoServe = 0xFF;  // an access of a hierarchy with no live tier, or not replayed here
constexpr int kXNT = 64;        // one wavefront per configuration
constexpr int kXStage = 1024;   // trace positions staged in LDS at a time
constexpr int kXH = KV_MAX_GROUPS * KV_TIERS;  // (hierarchy, tier) slots
constexpr uint32_t kXPool = 2048;  // LFU buckets whose records sit in LDS (40 KB)
// the five fields of an LFU bucket record
enum BucketField { kBF = 0, kBH, kBT, kBP, kBN, kBFields };

struct ExclJobDev {
  uint32_t cfg;    // configuration
  uint32_t mask;   // replayed hierarchies: bit g = group g (partitioned), bit 0 = the shared one
  uint64_t off;    // byte offset of the job's block state in the state buffer
};

struct ExclArgs {
  const kv_config* cfg;
  const ExclJobDev* jobs;
  const uint32_t* bid;   // [n] dense block id, trace order
  const uint8_t* w8;     // [n]
  const uint8_t* g8;     // [n]
  const uint8_t* blk_w;  // [U]
  const uint8_t* blk_g;  // [U]
  uint64_t n;
  uint32_t u;            // distinct blocks
  uint32_t n_groups;
  uint8_t* state;
  uint64_t* counts;      // [n_cfg][n_groups][3][8]
  uint32_t* err;         // {code, configuration} of the first failed job
};

// Byte layout of one job's block state (U = distinct blocks, P = U + 1 LFU
// buckets): tier u8[U] (padded to 4 bytes), prv/nxt u32[U], and with an LFU
// hierarchy node u32[U] plus the buckets' count, first, last, previous and
// next u32[P].
struct ExclLayout {
  uint64_t tier, prv, nxt, node, bf, bh, bt, bp, bn, bytes;
  __host__ __device__ ExclLayout(uint32_t u, bool lfu) {
    const uint64_t U = u, P = U + 1;
    tier = 0;
    prv = (U + 3) & ~3ull;
    nxt = prv + 4 * U;
    node = nxt + 4 * U;
    bf = node + (lfu ? 4 * U : 0);
    bh = bf + (lfu ? 4 * P : 0);
    bt = bh + (lfu ? 4 * P : 0);
    bp = bt + (lfu ? 4 * P : 0);
    bn = bp + (lfu ? 4 * P : 0);
    bytes = ((bn + (lfu ? 4 * P : 0)) + 255) & ~255ull;
  }
};

// Bucket records past the LDS pool.  Kept out of line: merged with the LDS
// access into one access through a selected pointer, the pair does not
// compile for gfx950.
__host__ __device__ __attribute__((noinline)) uint32_t dev_get(const uint32_t* p, uint32_t x) {
  return p[x];
}
__host__ __device__ __attribute__((noinline)) void dev_set(uint32_t* p, uint32_t x, uint32_t v) {
  p[x] = v;
}

// One job's replay state.  The walk (`access`, `finish`) runs in one lane;
// `tally` runs in every lane over a slice's served tiers.  Buckets are taken
// from the free list (last freed first) before a new index is used, so the
// live buckets keep low indices: the records of the first kXPool buckets
// sit in LDS, the others in device memory.
struct XWalk {
  uint8_t* tier;
  uint32_t *prv, *nxt, *node;
  uint32_t* bdev[kBFields];  // bucket records in device memory, by field
  uint32_t* blds[kBFields];  // the first kXPool of them in LDS
  uint32_t* lh;             // [kXH] first list member / first bucket
  uint32_t* lt;             // [kXH] last list member / last bucket
  unsigned long long* used; // [kXH]
  unsigned long long* cnt;  // [KV_MAX_GROUPS][3][8]
  const uint64_t* cap;      // [kXH]
  const uint8_t* pol;       // [KV_MAX_GROUPS] policy of each hierarchy
  const uint8_t* live;      // [KV_MAX_GROUPS][3] live tiers, fastest first
  const uint8_t* nlive;     // [KV_MAX_GROUPS]
  const uint8_t* blk_w;
  const uint8_t* blk_g;
  uint32_t free_b, bump, limit;  // LFU bucket pool: free list, next unused, size
  bool bad;

  __host__ __device__ void count(uint32_t g, uint32_t k, int f, uint32_t w) {
    cnt[(g * KV_TIERS + k) * 8 + f] += 1;
    cnt[(g * KV_TIERS + k) * 8 + f + 4] += w;
  }
  // ---- LRU / FIFO lists (first = oldest)
  // unlinks b, whose neighbours are p and q
  __host__ __device__ void list_unlink(uint32_t hk, uint32_t p, uint32_t q) {
    if (p != kNil) nxt[p] = q; else lh[hk] = q;
    if (q != kNil) prv[q] = p; else lt[hk] = p;
  }
  __host__ __device__ void list_append(uint32_t hk, uint32_t b) {
    const uint32_t p = lt[hk];
    prv[b] = p;
    nxt[b] = kNil;
    if (p != kNil) nxt[p] = b; else lh[hk] = b;
    lt[hk] = b;
  }
  // ---- LFU count buckets: count, first and last block, previous and next
  // bucket
  __host__ __device__ uint32_t bget(int k, uint32_t x) const {
    if (x < kXPool) return blds[k][x];
    return dev_get(bdev[k], x);
  }
  __host__ __device__ void bset(int k, uint32_t x, uint32_t v) {
    if (x < kXPool) blds[k][x] = v;
    else dev_set(bdev[k], x, v);
  }
  __host__ __device__ uint32_t bucket_new(uint32_t f) {
    uint32_t r = free_b;
    if (r != kNil) {
      free_b = bget(kBN, r);
    } else if (bump < limit) {
      r = bump++;
    } else {
      bad = true;  // more buckets than blocks: never with a consistent state
      return kNil;
    }
    bset(kBF, r, f);
    bset(kBH, r, kNil);
    bset(kBT, r, kNil);
    return r;
  }
  __host__ __device__ void bucket_free(uint32_t hk, uint32_t x) {
    const uint32_t p = bget(kBP, x), q = bget(kBN, x);
    if (p != kNil) bset(kBN, p, q); else lh[hk] = q;
    if (q != kNil) bset(kBP, q, p); else lt[hk] = p;
    bset(kBN, x, free_b);
    free_b = x;
  }
  __host__ __device__ void bucket_push(uint32_t x, uint32_t b) {
    const uint32_t p = bget(kBT, x);
    prv[b] = p;
    nxt[b] = kNil;
    if (p != kNil) nxt[p] = b; else bset(kBH, x, b);
    bset(kBT, x, b);
    node[b] = x;
  }
  // takes a block out of its bucket x, between blocks p and q, freeing the
  // bucket when it empties
  __host__ __device__ void bucket_pull(uint32_t hk, uint32_t x, uint32_t p, uint32_t q) {
    if (p != kNil) nxt[p] = q; else bset(kBH, x, q);
    if (q != kNil) prv[q] = p; else bset(kBT, x, p);
    if (p == kNil && q == kNil) bucket_free(hk, x);  // it was the bucket's only block
  }
  // ---- policy-level operations on tier slot hk
  __host__ __device__ uint32_t victim(uint32_t hk, uint32_t pol) const {
    const uint32_t f = lh[hk];
    if (pol != KV_POLICY_LFU || f == kNil) return f;
    return bget(kBH, f);
  }
  // A block's links: its bucket (LFU only) and its list neighbours.  All are
  // indexed by the block alone, so their loads go out together.
  struct Links {
    uint32_t x, p, q;
  };
  __host__ __device__ Links links(uint32_t pol, uint32_t b) const {
    return Links{pol == KV_POLICY_LFU ? node[b] : kNil, prv[b], nxt[b]};
  }
  // What an access reads of its block before it is known whether it hits,
  // all in one round of loads: the tier, and the links a top-tier hit moves
  // (none for FIFO, whose hits move nothing).
  struct Fields {
    uint32_t t;
    Links l;
  };
  __host__ __device__ Fields fields(uint32_t pol, uint32_t b) const {
    Fields f;
    f.t = tier[b];
    f.l = pol == KV_POLICY_FIFO ? Links{kNil, kNil, kNil} : links(pol, b);
    return f;
  }
  __host__ __device__ void take(uint32_t hk, uint32_t pol, const Links& l) {
    if (pol == KV_POLICY_LFU) bucket_pull(hk, l.x, l.p, l.q);
    else list_unlink(hk, l.p, l.q);
  }
  __host__ __device__ void admit(uint32_t hk, uint32_t pol, uint32_t b) {
    if (pol != KV_POLICY_LFU) {
      list_append(hk, b);
      return;
    }
    uint32_t x = lh[hk];
    if (x == kNil || bget(kBF, x) != 1u) {
      const uint32_t y = bucket_new(1u);
      if (y == kNil) return;
      bset(kBP, y, kNil);
      bset(kBN, y, x);
      if (x != kNil) bset(kBP, x, y); else lt[hk] = y;
      lh[hk] = y;
      x = y;
    }
    bucket_push(x, b);
  }
  // a hit in the top tier
  __host__ __device__ void touch(uint32_t hk, uint32_t pol, uint32_t b, const Links& l) {
    if (pol == KV_POLICY_LRU) {
      list_unlink(hk, l.p, l.q);
      list_append(hk, b);
    } else if (pol == KV_POLICY_LFU) {
      const uint32_t x = l.x, f = bget(kBF, x), q = bget(kBN, x);
      uint32_t y = q;
      if (q == kNil || bget(kBF, q) != f + 1u) {
        y = bucket_new(f + 1u);
        if (y == kNil) return;
        bset(kBP, y, x);
        bset(kBN, y, q);
        bset(kBN, x, y);
        if (q != kNil) bset(kBP, q, y); else lt[hk] = y;
      }
      bucket_pull(hk, x, l.p, l.q);
      bucket_push(y, b);
    }
  }
  // Block b (weight w, group g) enters live tier number D of hierarchy h,
  // whose policy is P: the tier first passes victims to live tier D + 1 (or
  // drops them).
  template <int D, uint32_t P>
  __host__ __device__ void enter(uint32_t h, uint32_t b, uint32_t w, uint32_t g) {
    const uint32_t k = live[h * KV_TIERS + D], hk = h * KV_TIERS + k, p = P;
    while (used[hk] + w > cap[hk]) {
      const uint32_t v = victim(hk, p);
      if (v == kNil) {  // an empty tier holds any block: never with a consistent state
        bad = true;
        return;
      }
      const uint32_t vw = blk_w[v], vg = blk_g[v];
      take(hk, p, links(p, v));
      used[hk] -= vw;
      tier[v] = kNoTier;
      count(vg, k, KV_F_EVICT, vw);  // its insertion below follows from this count
      if constexpr (D + 1 < KV_TIERS) {
        if (D + 1 < nlive[h]) enter<D + 1, P>(h, v, vw, vg);
      }
      if (bad) return;
    }
    admit(hk, p, b);
    used[hk] += w;
    tier[b] = (uint8_t)k;
  }
  // One access of hierarchy h.  Returns what served it: live tier number d
  // (fastest first), the number of live tiers for a miss in every tier, or
  // kNoServe with no live tier.  Its hit, miss and top-tier insertion
  // counts are left to `tally`.  The policy is dispatched once per access:
  // the walk below it is compiled for each policy.
  __host__ __device__ uint32_t access(uint32_t h, uint32_t b, uint32_t w, uint32_t g) {
    const uint32_t nl = nlive[h];
    if (nl == 0) return kNoServe;
    switch (pol[h]) {
      case KV_POLICY_FIFO: return access_p<KV_POLICY_FIFO>(h, b, w, g, nl);
      case KV_POLICY_LFU: return access_p<KV_POLICY_LFU>(h, b, w, g, nl);
      default: return access_p<KV_POLICY_LRU>(h, b, w, g, nl);
    }
  }
  template <uint32_t P>
  __host__ __device__ uint32_t access_p(uint32_t h, uint32_t b, uint32_t w, uint32_t g,
                                        uint32_t nl) {
    const uint32_t p = P;
    const Fields f = fields(p, b);  // in bounds either way; the links go unused after a miss
    const uint32_t t = f.t;
    const Links& l = f.l;
    uint32_t d = 0;
    while (d < nl && live[h * KV_TIERS + d] != t) ++d;
    if (d == 0) {
      touch(h * KV_TIERS + t, p, b, l);
      return 0;
    }
    if (t != kNoTier) {  // a hit below the top: taken out for promotion
      take(h * KV_TIERS + t, p, p == KV_POLICY_FIFO ? links(p, b) : l);
      used[h * KV_TIERS + t] -= w;
      tier[b] = kNoTier;
    }
    enter<0, P>(h, b, w, g);
    return d;
  }
  // The counts of an access that `access` left out: a miss in each live tier
  // faster than the one that served it, its hit, and its insertion into the
  // top tier unless the top tier served it.  `add(p, v)` adds v to *p.
  template <class Add>
  __host__ __device__ void tally(uint32_t h, uint32_t d, uint32_t g, uint32_t w, Add add) const {
    if (d == kNoServe) return;
    const uint32_t nl = nlive[h];
    unsigned long long* c = cnt + g * KV_TIERS * 8;
    for (uint32_t j = 0; j < nl && j <= d; ++j) {
      const uint32_t k = live[h * KV_TIERS + j];
      const int f = j == d ? KV_F_HIT : KV_F_MISS;
      add(&c[k * 8 + f], 1ull);
      add(&c[k * 8 + f + 4], (unsigned long long)w);
    }
    if (d != 0) {
      const uint32_t k = live[h * KV_TIERS];
      add(&c[k * 8 + KV_F_INS], 1ull);
      add(&c[k * 8 + KV_F_INS + 4], (unsigned long long)w);
    }
  }
  // After the walk: every block a live tier demotes enters the next live
  // tier, so that tier's insertions are the evictions above it.
  __host__ __device__ void finish(uint32_t n_groups, bool part, uint32_t mask) {
    for (uint32_t g = 0; g < n_groups; ++g) {
      const uint32_t h = part ? g : 0u;
      if (!((mask >> h) & 1u)) continue;
      unsigned long long* c = cnt + g * KV_TIERS * 8;
      for (uint32_t d = 1; d < nlive[h]; ++d) {
        const uint32_t k = live[h * KV_TIERS + d], a = live[h * KV_TIERS + d - 1];
        c[k * 8 + KV_F_INS] += c[a * 8 + KV_F_EVICT];
        c[k * 8 + KV_F_INS + 4] += c[a * 8 + KV_F_EVICT + 4];
      }
    }
  }
};

// Marks every block of every job of the wave absent (the lists need no
// initialisation: a block's links are written when it enters a tier).
__global__ __launch_bounds__(256) void k_excl_fill(uint8_t* __restrict__ state,
                                                   const ExclJobDev* __restrict__ jobs,
                                                   uint32_t n_jobs, uint32_t tier_words) {
  const uint64_t total = (uint64_t)n_jobs * tier_words;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t j = (uint32_t)(i / tier_words), q = (uint32_t)(i % tier_words);
    reinterpret_cast<uint32_t*>(state + jobs[j].off)[q] = 0xFFFFFFFFu;
  }
}

__global__ __launch_bounds__(kXNT) void k_excl_replay(ExclArgs a) {
  const ExclJobDev job = a.jobs[blockIdx.x];
  const kv_config& C = a.cfg[job.cfg];
  const uint32_t G = a.n_groups;
  const bool part = C.partitioned != 0;
  __shared__ uint32_t lh[kXH], lt[kXH];
  __shared__ unsigned long long used[kXH];
  __shared__ uint64_t cap[kXH];
  __shared__ unsigned long long cnt[KV_MAX_GROUPS * KV_TIERS * 8];
  __shared__ uint8_t pol[KV_MAX_GROUPS], live[KV_MAX_GROUPS * KV_TIERS], nlive[KV_MAX_GROUPS];
  __shared__ uint32_t sb[kXStage];
  __shared__ uint8_t sw[kXStage], sg[kXStage], sv[kXStage];
  __shared__ uint32_t sbf[kXPool], sbh[kXPool], sbt[kXPool], sbp[kXPool], sbn[kXPool];
  const uint32_t lane = threadIdx.x;
  for (uint32_t i = lane; i < (uint32_t)kXH; i += kXNT) {
    const uint32_t h = i / KV_TIERS, k = i % KV_TIERS;
    lh[i] = lt[i] = kNil;
    used[i] = 0;
    cap[i] = part ? C.cap_group[k][h] : C.cap[k];
  }
  for (uint32_t i = lane; i < (uint32_t)(KV_MAX_GROUPS * KV_TIERS * 8); i += kXNT) cnt[i] = 0;
  if (lane < (uint32_t)KV_MAX_GROUPS) {
    const uint32_t h = lane;
    pol[h] = part ? C.policy[h] : C.policy[0];
    uint32_t m = 0;
    for (uint32_t k = 0; k < (uint32_t)KV_TIERS; ++k) {
      const uint64_t x = part ? C.cap_group[k][h] : C.cap[k];
      if (x) live[h * KV_TIERS + m++] = (uint8_t)k;
    }
    nlive[h] = (uint8_t)m;
  }
  bool lfu = false;
  for (uint32_t h = 0; h < (part ? G : 1u); ++h)
    lfu |= ((job.mask >> h) & 1u) && (part ? C.policy[h] : C.policy[0]) == KV_POLICY_LFU;
  const ExclLayout L(a.u, lfu);
  uint8_t* base = a.state + job.off;
  XWalk x;
  x.tier = base + L.tier;
  x.prv = reinterpret_cast<uint32_t*>(base + L.prv);
  x.nxt = reinterpret_cast<uint32_t*>(base + L.nxt);
  x.node = reinterpret_cast<uint32_t*>(base + L.node);
  x.bdev[kBF] = reinterpret_cast<uint32_t*>(base + L.bf);
  x.bdev[kBH] = reinterpret_cast<uint32_t*>(base + L.bh);
  x.bdev[kBT] = reinterpret_cast<uint32_t*>(base + L.bt);
  x.bdev[kBP] = reinterpret_cast<uint32_t*>(base + L.bp);
  x.bdev[kBN] = reinterpret_cast<uint32_t*>(base + L.bn);
  x.blds[kBF] = sbf;
  x.blds[kBH] = sbh;
  x.blds[kBT] = sbt;
  x.blds[kBP] = sbp;
  x.blds[kBN] = sbn;
  x.lh = lh;
  x.lt = lt;
  x.used = used;
  x.cnt = cnt;
  x.cap = cap;
  x.pol = pol;
  x.live = live;
  x.nlive = nlive;
  x.blk_w = a.blk_w;
  x.blk_g = a.blk_g;
  x.free_b = kNil;
  x.bump = 0;
  x.limit = lfu ? a.u + 1 : 0;
  x.bad = false;
  __syncthreads();
  for (uint64_t base_p = 0; base_p < a.n; base_p += kXStage) {
    const uint32_t m = (uint32_t)std::min<uint64_t>(kXStage, a.n - base_p);
    for (uint32_t i = lane; i < m; i += kXNT) {
      sb[i] = a.bid[base_p + i];
      sw[i] = a.w8[base_p + i];
      sg[i] = a.g8[base_p + i];
    }
    __syncthreads();
    if (lane == 0 && !x.bad) {
      // the next access's staged fields are read before this access runs
      uint32_t nb = sb[0], nw = sw[0], ng = sg[0];
      for (uint32_t i = 0; i < m; ++i) {
        const uint32_t b = nb, w = nw, g = ng, h = part ? g : 0u;
        if (i + 1 < m) {
          nb = sb[i + 1];
          nw = sw[i + 1];
          ng = sg[i + 1];
        }
        sv[i] = (uint8_t)(((job.mask >> h) & 1u) ? x.access(h, b, w, g) : kNoServe);
        if (x.bad) break;
      }
    }
    __syncthreads();
    // the slice's hit, miss and top-tier insertion counts, by every lane
    for (uint32_t i = lane; i < m; i += kXNT) {
      const uint32_t g = sg[i];
      x.tally(part ? g : 0u, sv[i], g, sw[i],
              [](unsigned long long* p, unsigned long long v) { atomicAdd(p, v); });
    }
  }
  __syncthreads();
  if (lane == 0) x.finish(G, part, job.mask);
  // the records this job owns: every group of a shared hierarchy, the
  // replayed groups of a partitioned one
  if (lane == 0 && x.bad && atomicCAS(&a.err[0], 0u, 2u) == 0u) atomicExch(&a.err[1], job.cfg);
  __syncthreads();
  for (uint32_t i = lane; i < G * KV_TIERS * 8; i += kXNT) {
    const uint32_t g = i / (KV_TIERS * 8);
    if (part && !((job.mask >> g) & 1u)) continue;
    a.counts[((uint64_t)job.cfg * G) * KV_TIERS * 8 + i] = cnt[i];
  }
}

uint64_t excl_test_budget() {
  const char* e = std::getenv("KVCFG_TEST_REPLAY_BUDGET");
  return e ? std::strtoull(e, nullptr, 10) : 0;
}

}  // namespace

bool excl_replayed(const kv_config& C, uint32_t g, bool mixed) {
  if (C.mode != KV_MODE_EXCLUSIVE_DEMOTE) return false;
  const uint32_t pol = C.partitioned ? C.policy[g] : C.policy[0];
  return pol != KV_POLICY_LRU || mixed;
}

kv_status excl_run(Trace& t, const kv_config* cfg_host, const kv_config* cfg_dev,
                   uint32_t n_cfg, uint64_t* counts, hipStream_t s) {
  const uint32_t G = t.n_groups;
  const bool mixed = t.st.w_min != t.st.w_max;
  std::vector<ExclJobDev> jobs;
  std::vector<uint64_t> bytes;
  for (uint32_t c = 0; c < n_cfg; ++c) {
    const kv_config& C = cfg_host[c];
    if (C.mode != KV_MODE_EXCLUSIVE_DEMOTE) continue;
    uint32_t mask = 0;
    bool lfu = false;
    for (uint32_t h = 0; h < (C.partitioned ? G : 1u); ++h)
      if (excl_replayed(C, h, mixed)) {
        mask |= 1u << h;
        lfu |= (C.partitioned ? C.policy[h] : C.policy[0]) == KV_POLICY_LFU;
      }
    if (!mask) continue;
    jobs.push_back(ExclJobDev{c, mask, 0});
    bytes.push_back(ExclLayout((uint32_t)t.u, lfu).bytes);
  }
  if (jobs.empty()) return KV_OK;
  StageTimer tm(kStReplayExcl, s);
  // waves of jobs whose states fit one buffer (all at once when they fit)
  uint64_t total = 0, largest = 0;
  for (uint64_t b : bytes) {
    total += b;
    largest = std::max(largest, b);
  }
  uint64_t budget = total;
  if (const uint64_t tb = excl_test_budget()) budget = std::max<uint64_t>(tb, 1);
  DevBuf& bstate = t.ws[20];
  DevBuf& bjobs = t.ws[21];
  kv_status st;
  std::vector<uint32_t> lo;
  uint64_t wave_bytes = 0;
  for (;;) {
    lo.assign(1, 0);
    wave_bytes = 0;
    uint64_t cur = 0;
    for (size_t i = 0; i < jobs.size(); ++i) {
      if (cur && cur + bytes[i] > std::max(budget, largest)) {
        lo.push_back((uint32_t)i);
        cur = 0;
      }
      jobs[i].off = cur;
      cur += bytes[i];
      wave_bytes = std::max(wave_bytes, cur);
    }
    if ((st = bstate.reserve(wave_bytes)) == KV_OK) break;
    if (st != KV_ERR_NOMEM || budget <= largest) return st;
    budget /= 2;
  }
  lo.push_back((uint32_t)jobs.size());
  if ((st = bjobs.reserve(jobs.size() * sizeof(ExclJobDev))) != KV_OK) return st;
  t.excl_stage.resize(jobs.size() * sizeof(ExclJobDev));
  std::memcpy(t.excl_stage.data(), jobs.data(), t.excl_stage.size());
  KV_HIP(hipMemcpyAsync(bjobs.p, t.excl_stage.data(), t.excl_stage.size(),
                        hipMemcpyHostToDevice, s));
  ExclArgs a{};
  a.cfg = cfg_dev;
  a.bid = t.shared.bid.as<uint32_t>();
  a.w8 = t.shared.w.as<uint8_t>();
  a.g8 = t.shared.g.as<uint8_t>();
  a.blk_w = t.blk_w.as<uint8_t>();
  a.blk_g = t.blk_g.as<uint8_t>();
  a.n = t.n;
  a.u = (uint32_t)t.u;
  a.n_groups = G;
  a.state = bstate.as<uint8_t>();
  a.counts = counts;
  a.err = t.err.as<uint32_t>();
  const uint32_t tier_words = (uint32_t)((t.u + 3) / 4);
  for (size_t w = 0; w + 1 < lo.size(); ++w) {
    const uint32_t j0 = lo[w], nj = lo[w + 1] - lo[w];
    a.jobs = bjobs.as<ExclJobDev>() + j0;
    const uint64_t fill = (uint64_t)nj * tier_words;
    hipLaunchKernelGGL(k_excl_fill, dim3((uint32_t)std::min<uint64_t>((fill + 255) / 256, 16384)),
                       dim3(256), 0, s, a.state, a.jobs, nj, tier_words);
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_excl_replay, dim3(nj), dim3(kXNT), 0, s, a);
    KV_HIP(hipGetLastError());
  }
  // a failed state check is reported by the next call on this trace
  KV_HIP(hipMemcpyAsync(t.err_host, t.err.p, 2 * sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  KV_HIP(hipEventRecord(t.err_ev, s));
  t.err_pending = true;
  return KV_OK;
}

}  // namespace kv
