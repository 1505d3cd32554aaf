// k_replay.hip - tiers whose policy has no stack property (FIFO, LFU).
//
// The paper's simulator replays the trace through each candidate's tiers
// (Section 3.2, Section 4.1).  FIFO and LFU caches are not inclusive across
// capacities (FIFO shows Belady's anomaly), so each distinct (access order,
// group, policy, capacity) is replayed once as a "job"; inclusive tiers are
// independent caches, so a configuration's records follow from its tiers'
// per-access hit bits:
//   served by tier k  = hit_k and not hit in any faster tier,
//   miss of tier k    = not hit in tiers 0..k.
// A job whose capacity holds every distinct block of its accesses needs no
// replay: it hits exactly on re-accesses.
//
// Job state lives in HBM, indexed by dense block id.
//  FIFO: S[b] = total weight inserted before b's latest insertion.  The FIFO
//        queue always holds the longest suffix of the insertion sequence that
//        fits, so b is resident iff (weight inserted so far) - S[b] <= C.
//  LFU:  (frequency, last access position) per block.  Victims are the
//        minimum (frequency, last access); the members of one frequency class
//        are ordered by the position at which they entered it, which is
//        their last access, so each class is a queue over trace positions
//        and a per-class head pointer that only moves forward finds the
//        oldest live member.
#include <cstdio>
#include <cstring>
#include <map>
#include <optional>
#include <tuple>

#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr uint64_t kNoIns = ~0ull;

struct JobDev {
  uint32_t order, group, policy, closed;
  uint64_t cap, begin, end;
  uint64_t state_off;   // u64 words into the state pool
  uint64_t class_off;   // u32 words into the class pool (LFU)
  uint64_t bits_off;    // u64 words into the bitmap pool
  uint64_t word0;       // first bitmap word index (begin / 64)
  uint32_t kind;        // kJobFifoChunk, kJobFifoSerial, kJobLfu
  uint32_t chunk;       // chunk length (multiple of 64)
};

enum : uint32_t { kJobFifoChunk = 0, kJobFifoSerial = 1, kJobLfu = 2 };

struct JobArgs {
  const uint32_t* bid[2];
  const uint32_t* key[2];
  const uint32_t* nxt[2];
  const uint8_t* w8[2];
  const uint8_t* g8[2];
  const uint8_t* blk_w;
  const uint8_t* blk_g;
  uint64_t u;           // distinct blocks
  uint32_t n_groups;
  uint32_t n_class;     // LFU classes per job (max multiplicity + 2)
};

constexpr int kRNT = 1024;                 // threads of a replay workgroup
constexpr int kRIt = 4;                    // accesses per thread per chunk
constexpr uint32_t kRChunk = kRNT * kRIt;  // longest chunk
constexpr uint32_t kCand = 4096;           // LFU eviction candidates per chunk
constexpr uint32_t kMinFast = 256;         // shorter LFU chunks go serial
constexpr uint16_t kInf16 = 0xFFFF;

// Optional per-job replay statistics (diagnostics build only).
#ifdef KV_REPLAY_STATS
enum { kStFastOk = 0, kStFailPool, kStFailElig, kStFailConv, kStSerialAcc, kStIters,
       kStScanned, kStFastAcc, kStats };
__device__ unsigned long long g_rstats[256][kStats];
#define RSTAT(j, k, v) do { if (threadIdx.x == 0) atomicAdd(&g_rstats[(j) & 255][k], (unsigned long long)(v)); } while (0)
#else
#define RSTAT(j, k, v) do { } while (0)
#endif

__device__ __forceinline__ uint32_t ld_acq(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_acq64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// per-job counters: [job][group][4] = ins, ins_w, evict, evict_w
struct GroupCounters {
  unsigned long long ins[KV_MAX_GROUPS], insw[KV_MAX_GROUPS], ev[KV_MAX_GROUPS],
      evw[KV_MAX_GROUPS];
};

__global__ __launch_bounds__(256) void k_replay_init(const JobDev* __restrict__ jobs,
                                                     uint64_t* __restrict__ state,
                                                     uint32_t* __restrict__ cls, JobArgs a) {
  const JobDev j = jobs[blockIdx.y];
  if (j.closed) return;
  const uint64_t fill = (j.policy == KV_POLICY_FIFO) ? kNoIns : 0ull;
  uint64_t* st = state + j.state_off;
  for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < a.u;
       b += (uint64_t)gridDim.x * blockDim.x)
    st[b] = fill;
  if (j.policy == KV_POLICY_LFU) {
    // head[n_class] u32 | cnt[n_class] u32 | nz[(n_class+63)/64] u64
    uint32_t* head = cls + j.class_off;
    uint32_t* cnt = head + a.n_class;
    uint64_t* nz = reinterpret_cast<uint64_t*>(cnt + a.n_class);
    const uint32_t nw = (a.n_class + 63) / 64;
    for (uint32_t f = blockIdx.x * blockDim.x + threadIdx.x; f < a.n_class;
         f += gridDim.x * blockDim.x) {
      head[f] = (uint32_t)j.begin;
      cnt[f] = 0;
    }
    for (uint32_t f = blockIdx.x * blockDim.x + threadIdx.x; f < nw; f += gridDim.x * blockDim.x)
      nz[f] = 0;
  }
}

__device__ __forceinline__ void write_counters(const GroupCounters& c, uint32_t G,
                                               unsigned long long* cnt) {
  if (threadIdx.x < G) {
    unsigned long long* o = cnt + (uint64_t)threadIdx.x * 4;
    o[0] = c.ins[threadIdx.x];
    o[1] = c.insw[threadIdx.x];
    o[2] = c.ev[threadIdx.x];
    o[3] = c.evw[threadIdx.x];
  }
}

// Build the hit-bit words of [a, a + len) (a multiple of 64) from LDS flags.
__device__ __forceinline__ void store_bits(const uint8_t* s_hit, uint64_t a, uint32_t len,
                                           const JobDev& j, uint64_t* __restrict__ bits) {
  const uint32_t nwords = (len + 63) / 64;
  for (uint32_t wd = threadIdx.x; wd < nwords; wd += kRNT) {
    uint64_t word = 0;
    for (uint32_t k = 0; k < 64; ++k) {
      const uint32_t loc = wd * 64 + k;
      if (loc < len && s_hit[loc]) word |= 1ull << k;
    }
    const uint64_t base = a + (uint64_t)wd * 64;
    if (base < j.end && base + 64 > j.begin) bits[(base >> 6) - j.word0] = word;
  }
}

// ---------------------------------------------------------------------------
// FIFO by chunks.  With C >= chunk * w_max a block inserted inside a chunk
// cannot leave the queue before the chunk ends, so each block misses at most
// once per chunk: at its first access whose insertion total W(i) exceeds
// S[b] + C.  W depends on the misses before i, and more misses only raise W,
// so iterating "misses -> W -> misses" from "no misses" rises monotonically
// to the exact answer.
// ---------------------------------------------------------------------------
__device__ void fifo_chunked(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ S,
                             uint64_t* __restrict__ bits, unsigned long long* cnt) {
  __shared__ uint8_t s_ex[kRChunk];
  __shared__ uint8_t s_hit[kRChunk];
  __shared__ uint64_t s_red[kRNT / 64 + 1];
  __shared__ GroupCounters gc;
  const uint32_t tid = threadIdx.x;
  const uint32_t o = j.order;
  if (tid < KV_MAX_GROUPS) gc.ins[tid] = gc.insw[tid] = gc.ev[tid] = gc.evw[tid] = 0;
  __syncthreads();
  const uint32_t L = j.chunk;
  uint64_t W0 = 0;
  for (uint64_t c0 = j.begin & ~63ull; c0 < j.end; c0 += L) {
    const uint64_t c1 = min(c0 + L, j.end);
    uint32_t bb[kRIt], ww[kRIt], gg[kRIt];
    int lp[kRIt];
    uint64_t ss[kRIt], wi[kRIt];
    bool v[kRIt], miss[kRIt];
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t loc = tid * kRIt + e;
      const uint64_t p = c0 + loc;
      v[e] = loc < L && p >= j.begin && p < c1;
      bb[e] = v[e] ? a.bid[o][p] : 0u;
      ww[e] = v[e] ? a.w8[o][p] : 0u;
      gg[e] = v[e] ? a.g8[o][p] : 0u;
      const uint32_t k = v[e] ? a.key[o][p] : 0u;
      lp[e] = (k != 0 && (uint64_t)(k - 1) >= c0) ? (int)((uint64_t)(k - 1) - c0) : -1;
      ss[e] = v[e] ? S[bb[e]] : kNoIns;
      miss[e] = false;
    }
    uint64_t tot = 0;
    for (uint32_t it = 0; it < L + 2; ++it) {
      uint64_t x = 0;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) x += miss[e] ? ww[e] : 0u;
      const uint64_t pre = block_excl_scan<kRNT>(x, s_red, &tot);
      uint64_t run = W0 + pre;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) {
        wi[e] = run;
        const bool ex = v[e] && (ss[e] == kNoIns || run - ss[e] > j.cap);
        s_ex[tid * kRIt + e] = ex ? 1 : 0;
        run += miss[e] ? ww[e] : 0u;
      }
      __syncthreads();
      bool changed = false;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) {
        const bool ex = s_ex[tid * kRIt + e] != 0;
        const bool nm = ex && (lp[e] < 0 || s_ex[lp[e]] == 0);
        changed |= nm != miss[e];
        miss[e] = nm;
      }
      if (!__syncthreads_or(changed)) break;
    }
    // tot and wi belong to the final miss set
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      if (v[e] && miss[e]) {
        S[bb[e]] = wi[e];
        atomicAdd(&gc.ins[gg[e]], 1ull);
        atomicAdd(&gc.insw[gg[e]], (unsigned long long)ww[e]);
      }
      s_hit[tid * kRIt + e] = (v[e] && !miss[e]) ? 1 : 0;
    }
    W0 += tot;
    __syncthreads();
    store_bits(s_hit, c0, L, j, bits);
    __syncthreads();
  }
  // evictions = insertions - blocks still queued at the end
  __shared__ unsigned long long sfin[KV_MAX_GROUPS], sfinw[KV_MAX_GROUPS];
  if (tid < KV_MAX_GROUPS) sfin[tid] = sfinw[tid] = 0;
  __syncthreads();
  for (uint64_t b = tid; b < a.u; b += kRNT) {
    const uint64_t s = S[b];
    if (s != kNoIns && W0 - s <= j.cap) {
      const uint32_t g = a.blk_g[b];
      atomicAdd(&sfin[g], 1ull);
      atomicAdd(&sfinw[g], (unsigned long long)a.blk_w[b]);
    }
  }
  __syncthreads();
  if (tid < KV_MAX_GROUPS) {
    gc.ev[tid] = gc.ins[tid] - sfin[tid];
    gc.evw[tid] = gc.insw[tid] - sfinw[tid];
  }
  __syncthreads();
  write_counters(gc, a.n_groups, cnt);
}

// FIFO for capacities below 64 blocks: lanes of wave 0 gather a batch of 64
// accesses, one lane resolves them in trace order.
__device__ void fifo_serial(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ S,
                            uint64_t* __restrict__ bits, unsigned long long* cnt) {
  __shared__ uint32_t sb[64], sw[64], sg[64];
  __shared__ int sdup[64];
  __shared__ uint64_t ss[64], snew[64];
  __shared__ GroupCounters gc;
  const uint32_t lane = threadIdx.x;
  const uint32_t o = j.order;
  if (lane < KV_MAX_GROUPS) gc.ins[lane] = gc.insw[lane] = gc.ev[lane] = gc.evw[lane] = 0;
  uint64_t wcur = 0;
  for (uint64_t base = j.begin & ~63ull; base < j.end; base += 64) {
    const uint64_t i = base + lane;
    const bool in = lane < 64 && i >= j.begin && i < j.end;
    if (lane < 64) {
      const uint32_t b = in ? a.bid[o][i] : 0u;
      sb[lane] = b;
      sw[lane] = in ? a.w8[o][i] : 0u;
      sg[lane] = in ? a.g8[o][i] : 0u;
      ss[lane] = in ? S[b] : 0ull;
    }
    __syncthreads();
    if (lane < 64) {
      int dup = -1;
      if (in)
        for (int l = (int)lane - 1; l >= 0; --l)
          if (base + l >= j.begin && sb[l] == sb[lane]) {
            dup = l;
            break;
          }
      sdup[lane] = dup;
    }
    __syncthreads();
    if (lane == 0) {
      uint64_t word = 0;
      for (uint32_t l = 0; l < 64; ++l) {
        const uint64_t p = base + l;
        if (p < j.begin || p >= j.end) continue;
        const uint64_t s = sdup[l] >= 0 ? snew[sdup[l]] : ss[l];
        const bool hit = s != kNoIns && wcur - s <= j.cap;
        if (hit) {
          word |= 1ull << l;
          snew[l] = s;
        } else {
          snew[l] = wcur;
          S[sb[l]] = wcur;
          wcur += sw[l];
          gc.ins[sg[l]] += 1;
          gc.insw[sg[l]] += sw[l];
        }
      }
      bits[(base >> 6) - j.word0] = word;
    }
    __syncthreads();
  }
  __shared__ uint64_t swfin;
  __shared__ unsigned long long sfin[KV_MAX_GROUPS], sfinw[KV_MAX_GROUPS];
  if (lane == 0) swfin = wcur;
  if (lane < KV_MAX_GROUPS) sfin[lane] = sfinw[lane] = 0;
  __syncthreads();
  const uint64_t wf = swfin;
  for (uint64_t b = lane; b < a.u; b += kRNT) {
    const uint64_t s = S[b];
    if (s != kNoIns && wf - s <= j.cap) {
      const uint32_t g = a.blk_g[b];
      atomicAdd(&sfin[g], 1ull);
      atomicAdd(&sfinw[g], (unsigned long long)a.blk_w[b]);
    }
  }
  __syncthreads();
  if (lane < KV_MAX_GROUPS) {
    gc.ev[lane] = gc.ins[lane] - sfin[lane];
    gc.evw[lane] = gc.insw[lane] - sfinw[lane];
  }
  __syncthreads();
  write_counters(gc, a.n_groups, cnt);
}

// ---------------------------------------------------------------------------
// LFU.  State per block: (last access position << 32) | in-cache count (0 =
// absent).  The members of count class f in victim order are the positions
// of their last accesses, so class f is a queue over positions scanned by a
// head pointer head[f]; cnt[f] counts members, nz has a bit per nonempty class.
// ---------------------------------------------------------------------------
struct LfuShared {
  uint64_t used;
  uint32_t fmin;
  uint32_t head1;
};

__device__ __forceinline__ uint32_t next_class(const uint64_t* nz, uint32_t nw, uint32_t f) {
  uint32_t wi = f >> 6;
  if (wi >= nw) return 0xFFFFFFFFu;
  uint64_t m = ld_acq64(&nz[wi]) & (~0ull << (f & 63));
  while (m == 0) {
    if (++wi >= nw) return 0xFFFFFFFFu;
    m = ld_acq64(&nz[wi]);
  }
  return (wi << 6) + (uint32_t)__ffsll((long long)m) - 1u;
}

__device__ __forceinline__ void class_add(uint32_t* cnt, uint64_t* nz, uint32_t f, int d) {
  if (d > 0) {
    if (atomicAdd(&cnt[f], 1u) == 0u) atomicOr((unsigned long long*)&nz[f >> 6], 1ull << (f & 63));
  } else {
    if (atomicSub(&cnt[f], 1u) == 1u)
      atomicAnd((unsigned long long*)&nz[f >> 6], ~(1ull << (f & 63)));
  }
}

// Exact replay of [p0, p1) by one thread (thread 0); returns false if the
// state is found inconsistent.
__device__ bool lfu_serial_range(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ st,
                                 uint32_t* head, uint32_t* ccount, uint64_t* nz, uint32_t nw,
                                 LfuShared& ls, GroupCounters& gc, uint64_t* __restrict__ bits,
                                 uint64_t p0, uint64_t p1) {
  const uint32_t o = j.order;
  const uint32_t* __restrict__ bid = a.bid[o];
  head[1] = ls.head1;
  uint64_t used = ls.used;
  uint32_t fmin = ls.fmin;
  uint64_t word = 0;
  bool ok = true;
  for (uint64_t i = p0; i < p1 && ok; ++i) {
    if (i >= j.begin) {
      const uint32_t b = bid[i];
      const uint32_t w = a.w8[o][i];
      const uint64_t s = st[b];
      const uint32_t f = (uint32_t)s;
      if (f) {
        word |= 1ull << (i & 63);
        const uint32_t f1 = f + 1;
        class_add(ccount, nz, f, -1);
        class_add(ccount, nz, f1, +1);
        if (f == fmin && ld_acq(&ccount[f]) == 0) fmin = f1;
        st[b] = ((uint64_t)i << 32) | f1;
      } else {
        while (used + w > j.cap) {
          uint32_t q = head[fmin];
          uint32_t v = 0;
          // the oldest live member of class fmin lies before position i; the
          // bound only guards against corrupted state
          for (; q < i; ++q) {
            v = bid[q];
            const uint64_t sv = st[v];
            if ((uint32_t)sv == fmin && (uint32_t)(sv >> 32) == q) break;
          }
          if (q >= i) {
            ok = false;
            break;
          }
          head[fmin] = q + 1;
          st[v] = 0;
          const uint32_t vw = a.blk_w[v], vg = a.blk_g[v];
          used -= vw;
          gc.ev[vg] += 1;
          gc.evw[vg] += vw;
          class_add(ccount, nz, fmin, -1);
          if (ld_acq(&ccount[fmin]) == 0) {
            const uint32_t nf = next_class(nz, nw, fmin);
            if (nf != 0xFFFFFFFFu) fmin = nf;
          }
        }
        st[b] = ((uint64_t)i << 32) | 1u;
        class_add(ccount, nz, 1, +1);
        fmin = 1;
        used += w;
        const uint32_t g = a.g8[o][i];
        gc.ins[g] += 1;
        gc.insw[g] += w;
      }
    }
    if ((i & 63) == 63 || i + 1 == p1) {
      if (i >= j.begin || (i | 63) >= j.begin) bits[(i >> 6) - j.word0] = word;
      word = 0;
    }
  }
  ls.used = used;
  ls.fmin = fmin;
  ls.head1 = head[1];
  return ok;
}

struct LfuLds {
  // per access of the chunk (local position)
  int16_t lp[kRChunk];        // previous touch in the chunk; pointer-jumped to the chain root
  uint16_t occ[kRChunk];      // earlier touches of the same block inside the chunk
  int16_t lmiss[kRChunk];     // latest miss of the block at or before this touch
  uint16_t nxloc[kRChunk];    // next touch in the chunk or kInf16
  uint8_t pw[kRChunk];        // weight
  uint8_t hit[kRChunk];
  uint8_t capm[kRChunk];      // miss because the block was evicted earlier in the chunk
  uint8_t mskip[kRChunk];     // the entry inserted here is promoted before its eviction
  uint8_t mcons[kRChunk];     // the entry inserted here is evicted inside the chunk
  uint16_t mpos[kRChunk];     // misses in order: local position
  uint32_t mneed[kRChunk];    // ...and the weight that must have left the cache by then
  // count-1 residents from before the chunk, oldest first
  uint32_t cq[kCand];         // position of their last touch
  uint32_t cb[kCand];         // block
  uint16_t ca[kCand];         // first touch inside the chunk or kInf16
  uint8_t cw[kCand];
  uint8_t cskip[kCand];
  uint8_t ccons[kCand];
  uint64_t red[kRNT / 64 + 1];
  uint32_t red32[kRNT / 64 + 1];
};

constexpr int kCPT = (kCand + kRChunk) / kRNT;  // queue entries per thread

// Exclusive suffix minimum over the threads of the block (threads above t).
template <int NT>
__device__ __forceinline__ uint32_t block_suffix_min_excl(uint32_t v, uint32_t* sh) {
  constexpr int NW = NT / 64;
  const uint32_t lane = lane_id();
  const int w = threadIdx.x / 64;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_down(x, d, 64);
    if (lane + d < 64) x = min(x, y);
  }
  const uint32_t above = __shfl_down(x, 1, 64);
  if (lane == 0) sh[w] = x;
  __syncthreads();
  uint32_t r = (lane < 63) ? above : 0xFFFFFFFFu;
  for (int ww = w + 1; ww < NW; ++ww) r = min(r, sh[ww]);
  __syncthreads();
  return r;
}

// One chunk [c0, c1) without the serial walk.
//
// While no count>=2 block has to go, LFU victims come from count 1, oldest
// last touch first: first the count-1 residents from before the chunk (in
// position order), then the blocks inserted inside the chunk (in insertion
// order).  An entry leaves that queue without eviction when its block is
// touched (promoted) at or before the moment the eviction pointer reaches it.
// Misses are the first touches of blocks absent at the chunk start plus the
// first touch after an eviction inside the chunk.  Misses, evictions and
// promotions depend on each other; they are iterated to a fixed point, and
// the result is accepted only if it is self-consistent: every eviction finds
// a queue entry inserted before it, and the old entries are exhausted before
// any new one is taken.  Returns false, with no block state changed, when
// that fails; the caller then retries with a shorter chunk.
__device__ bool lfu_fast(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ st,
                         uint32_t* ccount, uint64_t* nz, uint32_t nw, LfuShared& ls,
                         GroupCounters& gc, LfuLds& S, uint64_t* __restrict__ bits,
                         uint64_t c0, uint64_t c1) {
  const uint32_t tid = threadIdx.x;
  const uint32_t o = j.order;
  const uint32_t L = (uint32_t)(c1 - c0);
  __shared__ uint32_t s_nc, s_h, s_lastp, s_lastm;
  __shared__ uint64_t s_vw, s_victw;
  uint32_t bb[kRIt], ww[kRIt], gg[kRIt], f0[kRIt];
  bool v[kRIt], cm[kRIt], res0[kRIt];
#pragma unroll
  for (int e = 0; e < kRIt; ++e) {
    const uint32_t loc = tid * kRIt + e;
    const uint64_t p = c0 + loc;
    v[e] = loc < L && p >= j.begin;
    bb[e] = v[e] ? a.bid[o][p] : 0u;
    ww[e] = v[e] ? a.w8[o][p] : 0u;
    gg[e] = v[e] ? a.g8[o][p] : 0u;
    const uint32_t k = v[e] ? a.key[o][p] : 0u;
    const int lp = (k != 0 && (uint64_t)(k - 1) >= c0) ? (int)((uint64_t)(k - 1) - c0) : -1;
    const uint32_t nx = v[e] ? a.nxt[o][p] : kNone;
    const bool again = nx != kNone && (uint64_t)nx < c1;
    const uint64_t s = v[e] ? st[bb[e]] : 0ull;
    f0[e] = (uint32_t)s;
    res0[e] = f0[e] != 0;
    cm[e] = v[e] && lp < 0 && !res0[e];
    S.lp[loc] = (int16_t)lp;
    S.occ[loc] = lp >= 0 ? 1 : 0;
    S.nxloc[loc] = again ? (uint16_t)((uint64_t)nx - c0) : kInf16;
    S.pw[loc] = (uint8_t)ww[e];
    S.capm[loc] = 0;
    S.mskip[loc] = again ? 1 : 0;
    S.mcons[loc] = 0;
  }
  uint64_t x = 0;
#pragma unroll
  for (int e = 0; e < kRIt; ++e) x += cm[e] ? ww[e] : 0u;
  uint64_t itot0;
  block_excl_scan<kRNT>(x, S.red, &itot0);
  const uint64_t used0 = ls.used;
  const uint64_t ev0 = (used0 + itot0 > j.cap) ? used0 + itot0 - j.cap : 0ull;
  if (tid == 0) {
    s_nc = 0;
    s_vw = 0;
    s_h = ls.head1;
    s_lastp = 0;
    s_lastm = 0;
    s_victw = 0;
  }
  __syncthreads();
  uint32_t nc0 = 0;
  bool reached = false;
  if (ev0 > 0) {
    // old count-1 residents from head1 on, until the untouched ones alone
    // cover the first-touch demand (a capacity miss adds as much demand as
    // it adds victims), the chunk start is reached, or the buffer is full
    for (;;) {
      const uint32_t h = s_h;
      const uint64_t vw = s_vw;
      const uint32_t n0 = s_nc;
      if (vw >= ev0 || (uint64_t)h >= c0 || n0 + kRNT > kCand) break;
      const uint64_t q = (uint64_t)h + tid;
      bool live = false, touched = false;
      uint32_t bq = 0, aq = kInf16;
      if (q < c0) {
        bq = a.bid[o][q];
        const uint64_t sq = st[bq];
        live = (uint32_t)sq == 1u && (sq >> 32) == q;
        if (live) {
          const uint32_t nx = a.nxt[o][q];
          touched = nx != kNone && (uint64_t)nx < c1;
          aq = touched ? (uint32_t)((uint64_t)nx - c0) : kInf16;
        }
      }
      uint32_t cnt_live;
      const uint32_t pos = block_excl_scan<kRNT>(live ? 1u : 0u, S.red32, &cnt_live);
      const uint32_t wq = live ? (uint32_t)a.blk_w[bq] : 0u;
      if (live) {
        S.cq[n0 + pos] = (uint32_t)q;
        S.cb[n0 + pos] = bq;
        S.cw[n0 + pos] = (uint8_t)wq;
        S.ca[n0 + pos] = (uint16_t)aq;
        S.cskip[n0 + pos] = touched ? 1 : 0;
        S.ccons[n0 + pos] = 0;
      }
      uint64_t vsum;
      block_excl_scan<kRNT>((uint64_t)((live && !touched) ? wq : 0u), S.red, &vsum);
      if (tid == 0) {
        s_nc = n0 + cnt_live;
        s_vw = vw + vsum;
        s_h = (uint32_t)min<uint64_t>((uint64_t)h + kRNT, c0);
      }
      __syncthreads();
    }
    nc0 = s_nc;
    reached = (uint64_t)s_h >= c0;
    // entries before the first live one are dead for good: skip them from now on
    if (tid == 0) ls.head1 = nc0 ? S.cq[0] : s_h;
  }
  // ---- fixed point over (misses, promotions, evictions)
  uint64_t itot = itot0;
  bool converged = ev0 == 0;
  for (int it = 0; !converged && it < 24; ++it) {
    bool mi[kRIt];
    uint64_t xw = 0;
    uint32_t xm = 0;
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      mi[e] = cm[e] || (v[e] && S.capm[tid * kRIt + e]);
      xw += mi[e] ? ww[e] : 0u;
      xm += mi[e] ? 1u : 0u;
    }
    uint64_t wpre = block_excl_scan<kRNT>(xw, S.red, &itot);
    uint32_t nm;
    uint32_t mpre = block_excl_scan<kRNT>(xm, S.red32, &nm);
    const uint64_t evtot = (used0 + itot > j.cap) ? used0 + itot - j.cap : 0ull;
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      if (mi[e]) {
        wpre += ww[e];
        const int64_t need = (int64_t)(used0 + wpre) - (int64_t)j.cap;
        S.mpos[mpre] = (uint16_t)(tid * kRIt + e);
        S.mneed[mpre] = need > 0 ? (uint32_t)need : 0u;
        ++mpre;
      }
    }
    __syncthreads();
    // the eviction queue: nc0 old entries, then the nm insertions of the chunk
    const uint32_t nq = nc0 + nm;
    uint32_t qw[kCPT];
    uint32_t xs = 0;
#pragma unroll
    for (int e = 0; e < kCPT; ++e) {
      const uint32_t k = tid * kCPT + e;
      qw[e] = 0;
      if (k < nc0) qw[e] = S.cskip[k] ? 0u : S.cw[k];
      else if (k < nq) {
        const uint32_t m = S.mpos[k - nc0];
        qw[e] = S.mskip[m] ? 0u : S.pw[m];
      }
      xs += qw[e];
    }
    uint32_t elig;
    uint32_t run = block_excl_scan<kRNT>(xs, S.red32, &elig);
    bool bad = (uint64_t)elig < evtot;
    uint32_t evk[kCPT];
#pragma unroll
    for (int e = 0; e < kCPT; ++e) {
      const uint32_t k = tid * kCPT + e;
      evk[e] = kInf16;
      if (k < nq && qw[e] && (uint64_t)run < evtot) {
        uint32_t lo = 0, hi = nm;
        while (lo < hi) {
          const uint32_t mid = (lo + hi) >> 1;
          if (S.mneed[mid] > run) hi = mid; else lo = mid + 1;
        }
        evk[e] = (lo < nm) ? S.mpos[lo] : kInf16;
        if (k >= nc0) {
          // a new entry can only go after it was inserted, and only once
          // every old one is gone
          if (evk[e] <= S.mpos[k - nc0] || !reached) bad = true;
        }
      }
      run += qw[e];
    }
    if (__syncthreads_or(bad)) return false;
    // the pointer reaches entry k when the first consumed entry at or after k goes
    uint32_t suf[kCPT];
    uint32_t mn = kInf16;
#pragma unroll
    for (int e = kCPT - 1; e >= 0; --e) {
      mn = min(mn, evk[e]);
      suf[e] = mn;
    }
    const uint32_t tmin = block_suffix_min_excl<kRNT>(mn, S.red32);
    // capacity misses are rebuilt from scratch: remember the old ones, clear
    bool oldcap[kRIt];
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t loc = tid * kRIt + e;
      oldcap[e] = S.capm[loc] != 0;
      S.capm[loc] = 0;
    }
    __syncthreads();
    bool changed = false;
#pragma unroll
    for (int e = 0; e < kCPT; ++e) {
      const uint32_t k = tid * kCPT + e;
      if (k >= nq) continue;
      const uint32_t ptime = min(suf[e], tmin);
      const bool cons = evk[e] != kInf16;
      const uint32_t ak = (k < nc0) ? (uint32_t)S.ca[k] : (uint32_t)S.nxloc[S.mpos[k - nc0]];
      const bool nskip = ak != kInf16 && (ptime == kInf16 || ak <= ptime);
      const bool ncap = ak != kInf16 && !nskip && ptime != kInf16;
      if (k < nc0) {
        changed |= (nskip != (S.cskip[k] != 0)) || (cons != (S.ccons[k] != 0));
        S.cskip[k] = nskip ? 1 : 0;
        S.ccons[k] = cons ? 1 : 0;
      } else {
        const uint32_t m = S.mpos[k - nc0];
        changed |= (nskip != (S.mskip[m] != 0)) || (cons != (S.mcons[m] != 0));
        S.mskip[m] = nskip ? 1 : 0;
        S.mcons[m] = cons ? 1 : 0;
      }
      if (ncap) S.capm[ak] = 1;  // each touch position is the next touch of one entry
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t loc = tid * kRIt + e;
      changed |= oldcap[e] != (S.capm[loc] != 0);
      // entries that stopped being misses lose their queue flags
      if (v[e] && !mi[e] && S.mcons[loc]) {
        S.mcons[loc] = 0;
        changed = true;
      }
    }
    if (!__syncthreads_or(changed)) converged = true;
  }
  if (!converged) return false;
  // ---- consistent: apply.  Pointer jumping gives each touch the number of
  // earlier touches of its block in the chunk and the latest miss among them.
#pragma unroll
  for (int e = 0; e < kRIt; ++e) {
    const uint32_t loc = tid * kRIt + e;
    const bool miss = cm[e] || (v[e] && S.capm[loc]);
    S.lmiss[loc] = miss ? (int16_t)loc : (int16_t)-1;
  }
  __syncthreads();
  for (uint32_t r = 0; (1u << r) < L; ++r) {
    int16_t np[kRIt], nl[kRIt];
    uint16_t no[kRIt];
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t loc = tid * kRIt + e;
      const int16_t p = S.lp[loc];
      no[e] = S.occ[loc];
      np[e] = p;
      nl[e] = S.lmiss[loc];
      if (p >= 0) {
        no[e] = (uint16_t)(S.occ[loc] + S.occ[p]);
        np[e] = S.lp[p] >= 0 ? S.lp[p] : p;
        if (nl[e] < 0) nl[e] = S.lmiss[p];
      }
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t loc = tid * kRIt + e;
      S.lp[loc] = np[e];
      S.occ[loc] = no[e];
      S.lmiss[loc] = nl[e];
    }
    __syncthreads();
  }
  // old entries evicted without being touched again
  uint64_t vw = 0;
  for (uint32_t k = tid; k < nc0; k += kRNT) {
    if (!S.ccons[k]) continue;
    const uint32_t b = S.cb[k];
    const uint32_t g = a.blk_g[b];
    atomicAdd(&gc.ev[g], 1ull);
    atomicAdd(&gc.evw[g], (unsigned long long)S.cw[k]);
    vw += S.cw[k];
    atomicMax(&s_lastp, k + 1);
    if (S.ca[k] == kInf16) {
      st[b] = 0;
      atomicSub(&ccount[1], 1u);
    }
  }
#pragma unroll
  for (int e = 0; e < kRIt; ++e) {
    const uint32_t loc = tid * kRIt + e;
    const bool miss = cm[e] || (v[e] && S.capm[loc]);
    S.hit[loc] = (v[e] && !miss) ? 1 : 0;
    if (!v[e]) continue;
    if (miss) {
      atomicAdd(&gc.ins[gg[e]], 1ull);
      atomicAdd(&gc.insw[gg[e]], (unsigned long long)ww[e]);
      if (S.mcons[loc]) {  // inserted here, evicted later in the chunk
        atomicAdd(&gc.ev[gg[e]], 1ull);
        atomicAdd(&gc.evw[gg[e]], (unsigned long long)ww[e]);
        vw += ww[e];
        atomicMax(&s_lastm, loc + 1);
      }
    }
  }
  if (vw) atomicAdd((unsigned long long*)&s_victw, (unsigned long long)vw);
  // final state of every touched block, at its last touch
  uint32_t fnew[kRIt];
  bool fin[kRIt];
#pragma unroll
  for (int e = 0; e < kRIt; ++e) {
    const uint32_t loc = tid * kRIt + e;
    fnew[e] = 0;
    fin[e] = v[e] && S.nxloc[loc] == kInf16;
    if (!fin[e]) continue;
    const int16_t m = S.lmiss[loc];
    if (m >= 0) {
      fnew[e] = S.mcons[m] ? 0u : (uint32_t)(S.occ[loc] - S.occ[m]) + 1u;
    } else {
      fnew[e] = f0[e] + (uint32_t)S.occ[loc] + 1u;
    }
    st[bb[e]] = fnew[e] ? (((uint64_t)(c0 + loc) << 32) | fnew[e]) : 0ull;
    if (res0[e]) atomicSub(&ccount[f0[e]], 1u);
    if (fnew[e]) atomicAdd(&ccount[fnew[e]], 1u);
  }
  __syncthreads();
  // nonempty-class bits from the final counts of every class touched above
#pragma unroll
  for (int e = 0; e < kRIt; ++e) {
    if (!fin[e]) continue;
#pragma unroll
    for (int z = 0; z < 2; ++z) {
      const uint32_t f = z == 0 ? (res0[e] ? f0[e] : 0u) : fnew[e];
      if (f == 0) continue;
      const uint64_t bit = 1ull << (f & 63);
      if (ld_acq(&ccount[f]) > 0) atomicOr((unsigned long long*)&nz[f >> 6], bit);
      else atomicAnd((unsigned long long*)&nz[f >> 6], ~bit);
    }
  }
  if (tid == 0) {
    if (ld_acq(&ccount[1]) > 0) atomicOr((unsigned long long*)&nz[0], 2ull);
    else atomicAnd((unsigned long long*)&nz[0], ~2ull);
  }
  __syncthreads();
  store_bits(S.hit, c0, L, j, bits);
  if (tid == 0) {
    ls.used = used0 + itot - s_victw;
    if (s_lastm) ls.head1 = (uint32_t)(c0 + s_lastm);           // last new entry taken + 1
    else if (s_lastp) ls.head1 = S.cq[s_lastp - 1] + 1;          // last old entry taken + 1
    const uint32_t nf = next_class(nz, nw, 1);
    if (nf != 0xFFFFFFFFu) ls.fmin = nf;
  }
  __syncthreads();
  return true;
}

__device__ void lfu_chunked(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ st,
                            uint32_t* __restrict__ cls, uint64_t* __restrict__ bits,
                            unsigned long long* cnt) {
  __shared__ LfuLds S;
  __shared__ LfuShared ls;
  __shared__ GroupCounters gc;
  __shared__ bool s_ok;
  const uint32_t tid = threadIdx.x;
  uint32_t* head = cls + j.class_off;
  uint32_t* ccount = head + a.n_class;
  uint64_t* nz = reinterpret_cast<uint64_t*>(ccount + a.n_class);
  const uint32_t nw = (a.n_class + 63) / 64;
  if (tid < KV_MAX_GROUPS) gc.ins[tid] = gc.insw[tid] = gc.ev[tid] = gc.evw[tid] = 0;
  if (tid == 0) {
    ls.used = 0;
    ls.fmin = 1;
    ls.head1 = (uint32_t)j.begin;
    s_ok = true;
  }
  __syncthreads();
  uint64_t pos = j.begin & ~63ull;
  uint32_t len = j.chunk;
  while (pos < j.end) {
    const uint32_t l = (uint32_t)min<uint64_t>(len, j.end - pos);
    if (lfu_fast(j, a, st, ccount, nz, nw, ls, gc, S, bits, pos, pos + l)) {
      pos += l;
      len = min<uint32_t>(len * 2, j.chunk);
    } else if (l > kMinFast) {
      len = max<uint32_t>(kMinFast, (l / 2) & ~63u);
    } else {
      __syncthreads();
      if (tid == 0) s_ok = lfu_serial_range(j, a, st, head, ccount, nz, nw, ls, gc, bits, pos,
                                            pos + l);
      RSTAT(blockIdx.x, kStSerialAcc, l);
      __syncthreads();
      if (!s_ok) break;
      pos += l;
    }
  }
  __syncthreads();
  write_counters(gc, a.n_groups, cnt);
  if (tid == 0 && !s_ok) cnt[0] = ~0ull;  // poison: surfaced as an impossible count
}

__global__ __launch_bounds__(kRNT) void k_replay(const JobDev* __restrict__ jobs, JobArgs a,
                                                 uint64_t* __restrict__ state,
                                                 uint32_t* __restrict__ cls,
                                                 uint64_t* __restrict__ bits,
                                                 unsigned long long* __restrict__ jcnt) {
  const JobDev j = jobs[blockIdx.x];
  if (j.closed) return;
  unsigned long long* cnt = jcnt + (uint64_t)blockIdx.x * a.n_groups * 4;
  if (j.kind == kJobFifoChunk)
    fifo_chunked(j, a, state + j.state_off, bits + j.bits_off, cnt);
  else if (j.kind == kJobFifoSerial)
    fifo_serial(j, a, state + j.state_off, bits + j.bits_off, cnt);
  else
    lfu_chunked(j, a, state + j.state_off, cls, bits + j.bits_off, cnt);
}

// Per order: re-access bits (key != 0), weight bit-planes, group masks.
__global__ __launch_bounds__(256) void k_order_bits(const uint32_t* __restrict__ key,
                                                    const uint8_t* __restrict__ w8,
                                                    const uint8_t* __restrict__ g8, uint64_t n,
                                                    uint64_t* __restrict__ reuse,
                                                    uint64_t* __restrict__ planes,
                                                    uint64_t* __restrict__ gmask,
                                                    uint32_t n_groups, uint64_t nwords) {
  const uint64_t wi = (uint64_t)blockIdx.x * 4 + threadIdx.x / 64;
  if (wi >= nwords) return;
  const uint64_t i = wi * 64 + lane_id();
  const bool in = i < n;
  const uint64_t r = __ballot(in && key[i] != 0);
  const uint32_t w = in ? w8[i] : 0u;
  const uint32_t g = in ? g8[i] : 0xFFu;
  uint64_t pl[8];
#pragma unroll
  for (int b = 0; b < 8; ++b) pl[b] = __ballot((w >> b) & 1u);
  uint64_t gm[KV_MAX_GROUPS];
#pragma unroll
  for (int gg = 0; gg < KV_MAX_GROUPS; ++gg) gm[gg] = __ballot(g == (uint32_t)gg);
  if (lane_id() == 0) {
    reuse[wi] = r;
#pragma unroll
    for (int b = 0; b < 8; ++b) planes[(uint64_t)b * nwords + wi] = pl[b];
    for (uint32_t gg = 0; gg < n_groups; ++gg) gmask[(uint64_t)gg * nwords + wi] = gm[gg];
  }
}

struct RecDev {
  uint32_t cfg, group;
  int32_t job[3];        // -1 = absent tier
  uint32_t order;
  uint64_t begin, end;   // positions in the order
  uint32_t filter;       // 1: count only accesses of `group`
  uint32_t pad;
};

struct CombineArgs {
  const JobDev* jobs;
  const uint64_t* bits;
  const unsigned long long* jcnt;
  const uint64_t* reuse[2];
  const uint64_t* planes[2];
  const uint64_t* gmask;  // shared order only
  uint64_t nwords;
  uint32_t n_groups;
  uint32_t uniform_w;     // 0 = mixed weights
  uint32_t plane_mask;    // weight bits present
};

__device__ __forceinline__ uint64_t job_word(const CombineArgs& a, int32_t jid, uint32_t order,
                                             uint64_t wi) {
  if (jid < 0) return 0ull;
  const JobDev& j = a.jobs[jid];
  if (j.closed) return a.reuse[order][wi];
  return a.bits[j.bits_off + (wi - j.word0)];
}

__device__ __forceinline__ uint64_t wpop(const CombineArgs& a, uint32_t order, uint64_t wi,
                                         uint64_t m) {
  if (a.uniform_w) return (uint64_t)__popcll(m) * a.uniform_w;
  uint64_t s = 0;
  for (int b = 0; b < 8; ++b)
    if (a.plane_mask & (1u << b))
      s += (uint64_t)__popcll(m & a.planes[order][(uint64_t)b * a.nwords + wi]) << b;
  return s;
}

__global__ __launch_bounds__(256) void k_combine(const RecDev* __restrict__ recs, CombineArgs a,
                                                 uint64_t* __restrict__ counts) {
  const RecDev r = recs[blockIdx.x];
  __shared__ unsigned long long sh[8][4];
  // c[0..3] = |mask|, |U0|, |U1|, |U2|; c[4..7] weighted
  unsigned long long c[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (r.end > r.begin) {
    const uint64_t wlo = r.begin >> 6, whi = (r.end - 1) >> 6;
    for (uint64_t wi = wlo + threadIdx.x; wi <= whi; wi += 256) {
      uint64_t m = ~0ull;
      if (wi == wlo) m &= ~0ull << (r.begin & 63);
      if (wi == whi && (r.end & 63)) m &= (1ull << (r.end & 63)) - 1;
      if (r.filter) m &= a.gmask[(uint64_t)r.group * a.nwords + wi];
      const uint64_t p0 = job_word(a, r.job[0], r.order, wi);
      const uint64_t p1 = job_word(a, r.job[1], r.order, wi);
      const uint64_t p2 = job_word(a, r.job[2], r.order, wi);
      const uint64_t u0 = p0 & m, u1 = (p0 | p1) & m, u2 = (p0 | p1 | p2) & m;
      c[0] += __popcll(m);
      c[1] += __popcll(u0);
      c[2] += __popcll(u1);
      c[3] += __popcll(u2);
      c[4] += wpop(a, r.order, wi, m);
      c[5] += wpop(a, r.order, wi, u0);
      c[6] += wpop(a, r.order, wi, u1);
      c[7] += wpop(a, r.order, wi, u2);
    }
  }
  for (int f = 0; f < 8; ++f) c[f] = wave_sum(c[f]);
  if (lane_id() == 0)
    for (int f = 0; f < 8; ++f) sh[f][threadIdx.x / 64] = c[f];
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long tot[8];
    for (int f = 0; f < 8; ++f) tot[f] = sh[f][0] + sh[f][1] + sh[f][2] + sh[f][3];
    uint64_t* out = counts + ((uint64_t)r.cfg * a.n_groups + r.group) * 24;
    for (int k = 0; k < 3; ++k) {
      uint64_t* rec = out + k * 8;
      if (r.job[k] < 0) {
        for (int f = 0; f < 8; ++f) rec[f] = 0;
        continue;
      }
      const unsigned long long* jc = a.jcnt + ((uint64_t)r.job[k] * a.n_groups + r.group) * 4;
      rec[KV_F_HIT] = tot[1 + k] - (k ? tot[k] : 0ull);
      rec[KV_F_HIT_W] = tot[5 + k] - (k ? tot[4 + k] : 0ull);
      rec[KV_F_MISS] = tot[0] - tot[1 + k];
      rec[KV_F_MISS_W] = tot[4] - tot[5 + k];
      rec[KV_F_INS] = jc[0];
      rec[KV_F_INS_W] = jc[1];
      rec[KV_F_EVICT] = jc[2];
      rec[KV_F_EVICT_W] = jc[3];
    }
  }
}

}  // namespace

kv_status replay_run(Trace& t, const std::vector<ReplayJob>& jobs, const kv_config* cfg_host,
                     const kv_config* cfg_dev, uint32_t n_cfg, uint64_t* counts,
                     hipStream_t s) {
  (void)cfg_dev;
  kv_status st;
  const uint32_t G = t.n_groups;
  const uint64_t n = t.n;
  const uint64_t nwords = (n + 63) / 64;
  const uint32_t n_class = (uint32_t)std::min<uint64_t>(t.st.max_multiplicity + 2, 0xFFFFFFF0ull);
  const uint32_t class_words = 2 * n_class + 2 * ((n_class + 63) / 64);  // u32 words per LFU job
  // layout of job state, class arrays and bitmaps
  std::vector<JobDev> jd(jobs.size());
  uint64_t state_words = 0, class_total = 0, bit_words = 0;
  for (size_t i = 0; i < jobs.size(); ++i) {
    const ReplayJob& r = jobs[i];
    JobDev& j = jd[i];
    j.order = r.order;
    j.group = r.group;
    j.policy = r.policy;
    j.closed = r.closed;
    j.cap = r.cap;
    j.begin = r.begin;
    j.end = r.end;
    j.word0 = r.begin >> 6;
    if (r.policy == KV_POLICY_FIFO) {
      const uint64_t lc = std::min<uint64_t>(kRChunk, (r.cap / std::max<uint32_t>(t.st.w_max, 1)) & ~63ull);
      j.kind = lc >= 64 ? kJobFifoChunk : kJobFifoSerial;
      j.chunk = (uint32_t)std::max<uint64_t>(lc, 64);
    } else {
      j.kind = kJobLfu;
      j.chunk = kRChunk;
    }
    if (!r.closed && r.end > r.begin) {
      j.state_off = state_words;
      state_words += t.u;
      if (r.policy == KV_POLICY_LFU) {
        j.class_off = class_total;
        class_total += class_words;
      }
      j.bits_off = bit_words;
      bit_words += ((r.end - 1) >> 6) - j.word0 + 1;
    } else {
      j.closed = 1;  // an empty segment behaves like a closed job
    }
  }
  // job counters, closed jobs preset: every distinct block inserted once
  std::vector<unsigned long long> jc(jobs.size() * G * 4, 0ull);
  for (size_t i = 0; i < jobs.size(); ++i) {
    if (!jd[i].closed) continue;
    for (uint32_t g = 0; g < G; ++g) {
      const bool mine = jd[i].group == KV_MAX_GROUPS || jd[i].group == g;
      if (!mine || jd[i].end <= jd[i].begin) continue;
      jc[(i * G + g) * 4 + 0] = t.st.u_g[g];
      jc[(i * G + g) * 4 + 1] = t.st.u_w_g[g];
    }
  }
  // records: (config, group) pairs with a replayed policy
  std::vector<RecDev> recs;
  std::map<std::tuple<uint32_t, uint32_t, uint32_t, uint64_t>, int32_t> idx;
  for (size_t i = 0; i < jobs.size(); ++i)
    idx[std::make_tuple(jobs[i].order, jobs[i].group, jobs[i].policy, jobs[i].cap)] = (int32_t)i;
  for (uint32_t c = 0; c < n_cfg; ++c) {
    const kv_config& C = cfg_host[c];
    const bool part_order = C.partitioned && G > 1;
    const uint32_t ng = C.partitioned ? G : 1;
    for (uint32_t g = 0; g < ng; ++g) {
      const uint32_t pol = C.partitioned ? C.policy[g] : C.policy[0];
      if (pol == KV_POLICY_LRU) continue;
      const uint32_t ord = part_order ? 1u : 0u;
      const uint32_t grp = part_order ? g : (uint32_t)KV_MAX_GROUPS;
      // a shared cache reports every group; a partitioned one only its own
      const uint32_t gfirst = C.partitioned ? g : 0, glast = C.partitioned ? g : G - 1;
      for (uint32_t gg = gfirst; gg <= glast; ++gg) {
        RecDev r{};
        r.cfg = c;
        r.group = gg;
        r.order = ord;
        for (int k = 0; k < 3; ++k) {
          const uint64_t x = C.partitioned ? C.cap_group[k][g] : C.cap[k];
          r.job[k] = x ? idx.at(std::make_tuple(ord, grp, pol, x)) : -1;
        }
        if (part_order) {
          r.begin = t.part.seg[g];
          r.end = t.part.seg[g + 1];
          r.filter = 0;
        } else {
          r.begin = 0;
          r.end = n;
          r.filter = G > 1 ? 1u : 0u;
        }
        recs.push_back(r);
      }
    }
  }
  DevBuf& bj = t.ws[11];
  DevBuf& bstate = t.ws[12];
  DevBuf& bcls = t.ws[13];
  DevBuf& bbits = t.ws[14];
  DevBuf& bjc = t.ws[15];
  DevBuf& brec = t.ws[16];
  DevBuf& bord = t.ws[17];
  if ((st = bj.reserve(jd.size() * sizeof(JobDev))) != KV_OK) return st;
  if ((st = bstate.reserve(std::max<uint64_t>(state_words, 1) * 8)) != KV_OK) return st;
  if ((st = bcls.reserve(std::max<uint64_t>(class_total, 2) * 4)) != KV_OK) return st;
  if ((st = bbits.reserve(std::max<uint64_t>(bit_words, 1) * 8)) != KV_OK) return st;
  if ((st = bjc.reserve(std::max<size_t>(jc.size(), 1) * 8)) != KV_OK) return st;
  if ((st = brec.reserve(std::max<size_t>(recs.size(), 1) * sizeof(RecDev))) != KV_OK) return st;
  const bool have_part = t.part.built;
  // per order: reuse bits, 8 weight planes, group masks
  const uint64_t per_order = nwords * (1 + 8 + KV_MAX_GROUPS);
  if ((st = bord.reserve(per_order * 2 * 8)) != KV_OK) return st;
  uint64_t* ob = bord.as<uint64_t>();
  uint64_t* reuse[2] = {ob, ob + per_order};
  uint64_t* planes[2] = {ob + nwords, ob + per_order + nwords};
  uint64_t* gmask[2] = {ob + 9 * nwords, ob + per_order + 9 * nwords};
  std::optional<StageTimer> tm;
  tm.emplace(kStReplayInit, s);
  for (int o = 0; o < 2; ++o) {
    const Order& od = o ? t.part : t.shared;
    if (o == 1 && !have_part) continue;
    hipLaunchKernelGGL(k_order_bits, dim3(div_up(nwords, 4)), dim3(256), 0, s,
                       od.key.as<uint32_t>(), od.w.as<uint8_t>(), od.g.as<uint8_t>(), n,
                       reuse[o], planes[o], gmask[o], G, nwords);
    KV_HIP(hipGetLastError());
  }
  // the job tables are staged in the trace so they outlive the async copies
  t.job_stage.resize(jd.size() * sizeof(JobDev));
  std::memcpy(t.job_stage.data(), jd.data(), t.job_stage.size());
  t.jc_stage.assign(jc.begin(), jc.end());
  t.rec_stage.resize(recs.size() * sizeof(RecDev));
  std::memcpy(t.rec_stage.data(), recs.data(), t.rec_stage.size());
  KV_HIP(hipMemcpyAsync(bj.p, t.job_stage.data(), t.job_stage.size(), hipMemcpyHostToDevice, s));
  if (!jc.empty())
    KV_HIP(hipMemcpyAsync(bjc.p, t.jc_stage.data(), jc.size() * 8, hipMemcpyHostToDevice, s));
  if (!recs.empty())
    KV_HIP(hipMemcpyAsync(brec.p, t.rec_stage.data(), t.rec_stage.size(), hipMemcpyHostToDevice,
                          s));
  JobArgs ja{};
  ja.bid[0] = t.shared.bid.as<uint32_t>();
  ja.key[0] = t.shared.key.as<uint32_t>();
  ja.nxt[0] = t.shared.nxt.as<uint32_t>();
  ja.key[1] = have_part ? t.part.key.as<uint32_t>() : ja.key[0];
  ja.nxt[1] = have_part ? t.part.nxt.as<uint32_t>() : ja.nxt[0];
  ja.w8[0] = t.shared.w.as<uint8_t>();
  ja.g8[0] = t.shared.g.as<uint8_t>();
  ja.bid[1] = have_part ? t.part.bid.as<uint32_t>() : ja.bid[0];
  ja.w8[1] = have_part ? t.part.w.as<uint8_t>() : ja.w8[0];
  ja.g8[1] = have_part ? t.part.g.as<uint8_t>() : ja.g8[0];
  ja.blk_w = t.blk_w.as<uint8_t>();
  ja.blk_g = t.blk_g.as<uint8_t>();
  ja.u = t.u;
  ja.n_groups = G;
  ja.n_class = n_class;
  const uint32_t nj = (uint32_t)jd.size();
  if (nj) {
    hipLaunchKernelGGL(k_replay_init, dim3(64, nj), dim3(256), 0, s, bj.as<JobDev>(),
                       bstate.as<uint64_t>(), bcls.as<uint32_t>(), ja);
    KV_HIP(hipGetLastError());
    tm.reset();
    tm.emplace(kStReplay, s);
    hipLaunchKernelGGL(k_replay, dim3(nj), dim3(kRNT), 0, s, bj.as<JobDev>(), ja,
                       bstate.as<uint64_t>(), bcls.as<uint32_t>(), bbits.as<uint64_t>(),
                       bjc.as<unsigned long long>());
    KV_HIP(hipGetLastError());
  }
#ifdef KV_REPLAY_STATS
  {
    KV_HIP(hipStreamSynchronize(s));
    unsigned long long hs[256][kStats];
    KV_HIP(hipMemcpyFromSymbol(hs, HIP_SYMBOL(g_rstats), sizeof(hs)));
    for (uint32_t q = 0; q < nj && q < 256; ++q) {
      if (jd[q].closed || jd[q].kind != kJobLfu) continue;
      fprintf(stderr, "[replay-stats] job %u cap %llu: fast %llu (acc %llu) failpool %llu "
              "failelig %llu failconv %llu serial_acc %llu iters %llu scanned %llu\n", q,
              (unsigned long long)jd[q].cap, hs[q][kStFastOk], hs[q][kStFastAcc],
              hs[q][kStFailPool], hs[q][kStFailElig], hs[q][kStFailConv], hs[q][kStSerialAcc],
              hs[q][kStIters], hs[q][kStScanned]);
    }
  }
#endif
  tm.reset();
  if (!recs.empty()) {
    tm.emplace(kStCombine, s);
    CombineArgs ca{};
    ca.jobs = bj.as<JobDev>();
    ca.bits = bbits.as<uint64_t>();
    ca.jcnt = bjc.as<unsigned long long>();
    ca.reuse[0] = reuse[0];
    ca.reuse[1] = have_part ? reuse[1] : reuse[0];
    ca.planes[0] = planes[0];
    ca.planes[1] = have_part ? planes[1] : planes[0];
    ca.gmask = gmask[0];
    ca.nwords = nwords;
    ca.n_groups = G;
    ca.uniform_w = (t.st.w_min == t.st.w_max) ? t.st.w_max : 0u;
    uint32_t pm = 0;
    for (uint32_t w = t.st.w_min; w <= t.st.w_max; ++w) pm |= w;
    ca.plane_mask = pm;
    hipLaunchKernelGGL(k_combine, dim3((uint32_t)recs.size()), dim3(256), 0, s,
                       brec.as<RecDev>(), ca, counts);
    KV_HIP(hipGetLastError());
  }
  return KV_OK;
}

}  // namespace kv
