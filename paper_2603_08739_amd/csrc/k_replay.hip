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
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
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
  uint64_t n;           // accesses per order; arrays hold 16 readable bytes past n
  uint32_t n_groups;
  uint32_t n_class;     // LFU class heads per job (kLdsClass)
  uint32_t job_lo, job_hi;  // the jobs of this launch (a wave); others return at once
  uint32_t fail_job;    // test hook: this job reports a failed state check (kNone: none)
  uint32_t* err;        // {code, job}: code 1 = an LFU job failed its state check
};

constexpr int kRNT = 1024;                 // threads of a replay workgroup
constexpr int kRNW = kRNT / 64;            // its wavefronts
constexpr int kRIt = 4;                    // accesses per thread per chunk
constexpr uint32_t kRChunk = kRNT * kRIt;  // longest chunk
constexpr uint32_t kCand = 4096;           // LFU eviction candidates per chunk
constexpr int kCScan = 2;                  // candidate positions per thread and pass
constexpr uint32_t kMinFast = 256;         // shorter LFU chunks go serial
constexpr uint32_t kHeadLds = 64;          // class heads held in LDS during a serial walk
constexpr uint16_t kInf16 = 0xFFFF;
constexpr int kLfuNT = 1024;               // threads of an LFU replay workgroup
constexpr uint32_t kLChunk = 4096;         // longest LFU chunk
constexpr uint32_t kLdsClass = 1024;       // LFU count classes (held in LDS)
constexpr uint32_t kTopClass = kLdsClass - 1;  // the class of every count >= kTopClass
constexpr uint32_t kLdsClassWords = kLdsClass / 64;
static_assert(kRIt == 4, "hit words are assembled from four ballots");

// Optional per-job replay statistics (diagnostics build only).

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
  if (blockIdx.y < a.job_lo || blockIdx.y >= a.job_hi) return;
  const JobDev j = jobs[blockIdx.y];
  if (j.closed) return;
  // FIFO: u32 insertion totals per block (two per word, all-ones = never
  // inserted).  LFU: u32 counts per position, each written before it is read.
  if (j.policy == KV_POLICY_FIFO) {
    const uint64_t words = (a.u + 1) / 2;
    uint64_t* st = state + j.state_off;
    for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < words;
         b += (uint64_t)gridDim.x * blockDim.x)
      st[b] = kNoIns;
  }
  if (j.policy == KV_POLICY_LFU) {
    // head[n_class] u32
    uint32_t* head = cls + j.class_off;
    for (uint32_t f = blockIdx.x * blockDim.x + threadIdx.x; f < a.n_class;
         f += gridDim.x * blockDim.x)
      head[f] = (uint32_t)j.begin;
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

// The kRIt consecutive accesses [p0, p0 + 4) of a thread; p0 is a multiple of
// 4, so when all four are valid one 16-byte (or 4-byte) load fetches them.
__device__ __forceinline__ void load4_u32(const uint32_t* __restrict__ a, uint64_t p0, bool all,
                                          const bool v[kRIt], uint32_t out[kRIt]) {
  if (all) {
    const uint4 x = *reinterpret_cast<const uint4*>(a + p0);
    out[0] = x.x;
    out[1] = x.y;
    out[2] = x.z;
    out[3] = x.w;
  } else {
#pragma unroll
    for (int e = 0; e < kRIt; ++e) out[e] = v[e] ? a[p0 + e] : 0u;
  }
}

__device__ __forceinline__ void load4_u8(const uint8_t* __restrict__ a, uint64_t p0, bool all,
                                         const bool v[kRIt], uint32_t out[kRIt]) {
  if (all) {
    const uint32_t x = *reinterpret_cast<const uint32_t*>(a + p0);
#pragma unroll
    for (int e = 0; e < kRIt; ++e) out[e] = (x >> (8 * e)) & 0xFFu;
  } else {
#pragma unroll
    for (int e = 0; e < kRIt; ++e) out[e] = v[e] ? (uint32_t)a[p0 + e] : 0u;
  }
}

// Hit words of a chunk starting at c0 (a multiple of 64).  Thread t holds
// positions 4t..4t+3, so the 16 lanes of each quarter wavefront hold one
// 64-position word: bit 4m+e of word q is item e of lane 16q+m.
__device__ __forceinline__ void store_hits(const bool hit[kRIt], uint64_t c0, uint32_t L,
                                           const JobDev& j, uint64_t* __restrict__ bits) {
  uint64_t bal[kRIt];
#pragma unroll
  for (int e = 0; e < kRIt; ++e) bal[e] = __ballot(hit[e]);
  const uint32_t q = lane_id();
  if (q < 4) {
    uint64_t word = 0;
#pragma unroll
    for (int e = 0; e < kRIt; ++e) word |= spread4(bal[e] >> (16 * q)) << e;
    const uint32_t wloc = (uint32_t)wave_id() * 4 + q;
    const uint64_t base = c0 + (uint64_t)wloc * 64;
    if (wloc * 64 < L && base < j.end && base + 64 > j.begin) bits[(base >> 6) - j.word0] = word;
  }
}

// IT consecutive accesses [p0, p0 + IT) of a thread (p0 a multiple of IT):
// vector loads when all are valid.
// Per-item flags of a thread, one bit per item in a vector register (an
// array of bools holds one scalar lane mask per item, and scalar registers
// run short).
struct ItemBits {
  uint32_t w = 0;
  __device__ __forceinline__ bool operator[](int e) const { return (w >> e) & 1u; }
  __device__ __forceinline__ void set(int e, bool b) { w |= (b ? 1u : 0u) << e; }
};

// IT consecutive elements from position p0 (a multiple of 4), branch-free:
// the read position is clamped to n & ~3 (the arrays' slack covers the
// vector read there; a clamped read only serves invalid items), and items
// with v[e] false read as 0.
template <int IT>
__device__ __forceinline__ void loadn_u32(const uint32_t* __restrict__ a, uint64_t p0, uint64_t n,
                                          const ItemBits& v, uint32_t* out) {
#pragma unroll
  for (int q = 0; q < IT / 4; ++q) {
    const uint64_t pq = min<uint64_t>(p0 + 4 * q, n & ~3ull);
    const uint4 x = *reinterpret_cast<const uint4*>(a + pq);
    out[4 * q] = v[4 * q] ? x.x : 0u;
    out[4 * q + 1] = v[4 * q + 1] ? x.y : 0u;
    out[4 * q + 2] = v[4 * q + 2] ? x.z : 0u;
    out[4 * q + 3] = v[4 * q + 3] ? x.w : 0u;
  }
}

template <int IT>
__device__ __forceinline__ void loadn_u8(const uint8_t* __restrict__ a, uint64_t p0, uint64_t n,
                                         const ItemBits& v, uint32_t* out) {
#pragma unroll
  for (int q = 0; q < IT / 4; ++q) {
    const uint64_t pq = min<uint64_t>(p0 + 4 * q, n & ~3ull);
    const uint32_t x = *reinterpret_cast<const uint32_t*>(a + pq);
#pragma unroll
    for (int e = 0; e < 4; ++e) out[4 * q + e] = v[4 * q + e] ? (x >> (8 * e)) & 0xFFu : 0u;
  }
}

// Hit words of a chunk starting at c0 (a multiple of 64) when thread t holds
// positions IT*t .. IT*t+IT-1: the 64/IT lanes of word q are lanes
// q*64/IT.., and bit m*IT+e of the word is item e of its lane m.
template <int IT>
__device__ __forceinline__ void store_hits_n(const bool* hit, uint64_t c0, uint32_t L,
                                             const JobDev& j, uint64_t* __restrict__ bits) {
  constexpr int LPW = 64 / IT;  // lanes per word
  uint64_t bal[IT];
#pragma unroll
  for (int e = 0; e < IT; ++e) bal[e] = __ballot(hit[e]);
  // the lane index, recomputed here (a value kept from the kernel's start
  // can end up spilled, and its reload would wait for every memory access
  // in flight)
  uint32_t q;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(q));
  if (q < (uint32_t)IT) {
    uint64_t word = 0;
    if constexpr (IT == 4) {
      // bit m of item e's 16-bit slice goes to bit 4m + e: spread eight
      // bits at a time to every fourth bit
      auto spread8 = [](uint32_t x) {
        x &= 0xFFu;
        x = (x | (x << 12)) & 0x000F000Fu;
        x = (x | (x << 6)) & 0x03030303u;
        x = (x | (x << 3)) & 0x11111111u;
        return x;
      };
      uint32_t lo = 0, hi = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t part = (uint32_t)(bal[e] >> (16 * q));
        lo |= spread8(part) << e;
        hi |= spread8(part >> 8) << e;
      }
      word = ((uint64_t)hi << 32) | lo;
    } else {
#pragma unroll
      for (int e = 0; e < IT; ++e) {
        const uint64_t part = bal[e] >> (LPW * q);
#pragma unroll
        for (int m = 0; m < LPW; ++m) word |= ((part >> m) & 1ull) << (m * IT + e);
      }
    }
    const uint32_t wloc = (uint32_t)wave_id() * IT + q;
    const uint64_t base = c0 + (uint64_t)wloc * 64;
    if (wloc * 64 < L && base < j.end && base + 64 > j.begin) bits[(base >> 6) - j.word0] = word;
  }
}

// Adds per-thread (count, weight) partials of one group: one LDS atomic per
// wavefront.
__device__ __forceinline__ void add_uniform(unsigned long long* dc, unsigned long long* dw,
                                            uint32_t c, uint32_t w) {
  const uint32_t sc = wave_sum(c), sw = wave_sum(w);
  if (lane_id() == 0 && sc) {
    atomicAdd(dc, (unsigned long long)sc);
    atomicAdd(dw, (unsigned long long)sw);
  }
}

struct FifoLds {
  uint8_t ex[kRChunk];
  uint32_t red[2 * kRNW];
  uint32_t anyflag[2];
  unsigned long long fin[KV_MAX_GROUPS], finw[KV_MAX_GROUPS];
};

// Inputs of one chunk for one thread (its kRIt consecutive accesses).
struct ChunkIn {
  uint32_t b[kRIt];  // dense block id
  uint32_t k[kRIt];  // previous occurrence + 1, 0 = none
  uint32_t w;        // weights, one byte per access
  uint32_t g;        // groups, one byte per access
};

__device__ __forceinline__ void chunk_valid(const JobDev& j, uint64_t c0, uint32_t L,
                                            bool v[kRIt]) {
  const uint32_t l0 = threadIdx.x * kRIt;
  const uint64_t p0 = c0 + l0;
  const uint64_t c1 = min(c0 + L, j.end);
#pragma unroll
  for (int e = 0; e < kRIt; ++e) v[e] = l0 + e < L && p0 + e >= j.begin && p0 + e < c1;
}

__device__ __forceinline__ uint32_t pack4_u8(const uint32_t x[kRIt]) {
  return x[0] | (x[1] << 8) | (x[2] << 16) | (x[3] << 24);
}

// Issues the loads of a chunk's inputs without branches, so that the
// compiler can leave them in flight while earlier loads are consumed: the
// position is clamped to n (the arrays have readable slack past n) and
// invalid items are zeroed.
__device__ __forceinline__ void issue_inputs(const JobDev& j, const JobArgs& a, uint64_t c0,
                                             uint32_t L, ChunkIn& in) {
  const uint32_t o = j.order;
  const uint64_t p0 = min(c0 + threadIdx.x * kRIt, a.n & ~3ull);  // valid p0 are multiples of 4 below n
  bool v[kRIt];
  chunk_valid(j, c0, L, v);
  const uint4 b = *reinterpret_cast<const uint4*>(a.bid[o] + p0);
  const uint4 k = *reinterpret_cast<const uint4*>(a.key[o] + p0);
  const uint32_t w = *reinterpret_cast<const uint32_t*>(a.w8[o] + p0);
  const uint32_t g = *reinterpret_cast<const uint32_t*>(a.g8[o] + p0);
  in.b[0] = v[0] ? b.x : 0u;
  in.b[1] = v[1] ? b.y : 0u;
  in.b[2] = v[2] ? b.z : 0u;
  in.b[3] = v[3] ? b.w : 0u;
  in.k[0] = v[0] ? k.x : 0u;
  in.k[1] = v[1] ? k.y : 0u;
  in.k[2] = v[2] ? k.z : 0u;
  in.k[3] = v[3] ? k.w : 0u;
  const uint32_t m = (v[0] ? 0xFFu : 0u) | (v[1] ? 0xFF00u : 0u) | (v[2] ? 0xFF0000u : 0u) |
                     (v[3] ? 0xFF000000u : 0u);
  in.w = w & m;
  in.g = g & m;
}

// ---------------------------------------------------------------------------
// FIFO by chunks.  With C >= chunk * w_max a block inserted inside a chunk
// cannot leave the queue before the chunk ends, so each block misses at most
// once per chunk: at its first access whose insertion total W(i) exceeds
// S[b] + C.  W depends on the misses before i, and more misses only raise W,
// so iterating "misses -> W -> misses" from "no misses" rises monotonically
// to the exact answer.
//
// S[b] < 2^32 (weights sum below 2^32); kNoIns32 marks a block never inserted.
// The chunk loop is software-pipelined: the inputs of chunk k+2 are loaded
// while chunk k is resolved, and so are the states of chunk k+1's blocks,
// which brings their lines into the caches; once chunk k's insertions are
// stored, the exact states of chunk k+1 are read again from there.  Dense
// block ids follow first occurrence, so the lines are few and shared.
// ---------------------------------------------------------------------------
constexpr uint32_t kNoIns32 = 0xFFFFFFFFu;

__device__ __forceinline__ void fifo_chunked(const JobDev& j, const JobArgs& a,
                                             uint32_t* __restrict__ S,
                                             uint64_t* __restrict__ bits, GroupCounters& gc,
                                             FifoLds& F, bool g1, uint32_t g0) {
  const uint32_t tid = threadIdx.x;
  const uint32_t L = j.chunk;
  const uint32_t l0 = tid * kRIt;
  const uint64_t cstart = j.begin & ~63ull;
  ChunkIn A, B, C;
  uint32_t sa[kRIt], sb[kRIt];
  issue_inputs(j, a, cstart, L, A);
  issue_inputs(j, a, cstart + L, L, B);
  {
    bool v[kRIt];
    chunk_valid(j, cstart, L, v);
#pragma unroll
    for (int e = 0; e < kRIt; ++e) sa[e] = v[e] ? S[A.b[e]] : kNoIns32;
  }
  if (tid < 2) F.anyflag[tid] = 0;
  __syncthreads();
  BlockAny block_any{F.anyflag, 0};
  uint32_t W0 = 0;
  for (uint64_t c0 = cstart; c0 < j.end; c0 += L) {
    bool v[kRIt], vb[kRIt], miss[kRIt];
    chunk_valid(j, c0, L, v);
    chunk_valid(j, c0 + L, L, vb);
    issue_inputs(j, a, c0 + 2 * (uint64_t)L, L, C);
    // touch the next chunk's states early (block 0 stands in for invalid
    // items) so that the exact re-read after this chunk finds them cached
    uint32_t warm[kRIt];
#pragma unroll
    for (int e = 0; e < kRIt; ++e) warm[e] = S[vb[e] ? B.b[e] : 0u];
    int lp[kRIt];
    uint32_t ww[kRIt], wi[kRIt];
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      const uint32_t k = A.k[e];
      lp[e] = (k != 0 && (uint64_t)(k - 1) >= c0) ? (int)((uint64_t)(k - 1) - c0) : -1;
      ww[e] = (A.w >> (8 * e)) & 0xFFu;
      miss[e] = false;
    }
    uint32_t tot = 0;
    for (uint32_t it = 0; it < L + 2; ++it) {
      uint32_t x = 0;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) x += miss[e] ? ww[e] : 0u;
      const uint32_t pre = block_excl_scan_u32<kRNT>(x, F.red, tot);
      uint32_t run = W0 + pre;
      uint32_t exw = 0;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) {
        wi[e] = run;
        const bool ex = v[e] && (sa[e] == kNoIns32 || (uint64_t)(run - sa[e]) > j.cap);
        exw |= (ex ? 1u : 0u) << (8 * e);
        run += miss[e] ? ww[e] : 0u;
      }
      *reinterpret_cast<uint32_t*>(&F.ex[l0]) = exw;
      __syncthreads();
      bool changed = false;
#pragma unroll
      for (int e = 0; e < kRIt; ++e) {
        const bool ex = (exw >> (8 * e)) & 1u;
        const bool nm = ex && (lp[e] < 0 || F.ex[lp[e]] == 0);
        changed |= nm != miss[e];
        miss[e] = nm;
      }
      const bool again = block_any(changed);
      if (!again) break;
    }
    // tot and wi belong to the final miss set
    bool hit[kRIt];
    uint32_t ci = 0, cw = 0;
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      hit[e] = v[e] && !miss[e];
      if (v[e] && miss[e]) {
        S[A.b[e]] = wi[e];
        if (g1) {
          ++ci;
          cw += ww[e];
        } else {
          const uint32_t g = (A.g >> (8 * e)) & 0xFFu;
          atomicAdd(&gc.ins[g], 1ull);
          atomicAdd(&gc.insw[g], (unsigned long long)ww[e]);
        }
      }
    }
    if (g1) add_uniform(&gc.ins[g0], &gc.insw[g0], ci, cw);
    W0 += tot;
    store_hits(hit, c0, L, j, bits);
    __syncthreads();
    // the next chunk's states after this chunk's insertions (the early
    // loads are kept alive, not used, so that they are issued)
#pragma unroll
    for (int e = 0; e < kRIt; ++e) {
      asm volatile("" ::"v"(warm[e]));
      sb[e] = S[vb[e] ? B.b[e] : 0u];
    }
    A = B;
    B = C;
#pragma unroll
    for (int e = 0; e < kRIt; ++e) sa[e] = sb[e];
  }
  // evictions = insertions - blocks still queued at the end.  The pass over
  // every block's state is bound by load latency: each thread keeps kEndU
  // loads in flight, and with one group the queued blocks add up in
  // registers (LDS atomics on one address are taken one lane at a time).
  if (tid < KV_MAX_GROUPS) F.fin[tid] = F.finw[tid] = 0;
  __syncthreads();
  constexpr int kEndU = 8;
  unsigned long long fc = 0, fw = 0;
  for (uint64_t b0 = tid; b0 < a.u; b0 += (uint64_t)kRNT * kEndU) {
    uint32_t s[kEndU], bw[kEndU], bg[kEndU];
#pragma unroll
    for (int q = 0; q < kEndU; ++q) {
      const uint64_t b = b0 + (uint64_t)q * kRNT;
      const bool in = b < a.u;
      s[q] = in ? S[b] : kNoIns32;
      bw[q] = in ? a.blk_w[b] : 0u;
      bg[q] = in ? a.blk_g[b] : 0u;
    }
#pragma unroll
    for (int q = 0; q < kEndU; ++q) {
      if (s[q] == kNoIns32 || (uint64_t)(W0 - s[q]) > j.cap) continue;
      if (g1) {
        ++fc;
        fw += bw[q];
      } else {
        atomicAdd(&F.fin[bg[q]], 1ull);
        atomicAdd(&F.finw[bg[q]], (unsigned long long)bw[q]);
      }
    }
  }
  if (g1) {
    fc = wave_sum(fc);
    fw = wave_sum(fw);
    if (lane_id() == 0 && fc) {
      atomicAdd(&F.fin[g0], fc);
      atomicAdd(&F.finw[g0], fw);
    }
  }
  __syncthreads();
  if (tid < KV_MAX_GROUPS) {
    gc.ev[tid] = gc.ins[tid] - F.fin[tid];
    gc.evw[tid] = gc.insw[tid] - F.finw[tid];
  }
}

// FIFO for capacities below 64 blocks: lanes of wave 0 gather a batch of 64
// accesses, one lane resolves them in trace order.
__device__ __forceinline__ void fifo_serial(const JobDev& j, const JobArgs& a,
                                            uint32_t* __restrict__ S, uint64_t* __restrict__ bits,
                                            GroupCounters& gc) {
  __shared__ uint32_t sb[64], sw[64], sg[64];
  __shared__ int sdup[64];
  __shared__ uint32_t ss[64], snew[64];
  const uint32_t lane = threadIdx.x;
  const uint32_t o = j.order;
  uint32_t wcur = 0;
  for (uint64_t base = j.begin & ~63ull; base < j.end; base += 64) {
    const uint64_t i = base + lane;
    const bool in = lane < 64 && i >= j.begin && i < j.end;
    if (lane < 64) {
      const uint32_t b = in ? a.bid[o][i] : 0u;
      sb[lane] = b;
      sw[lane] = in ? a.w8[o][i] : 0u;
      sg[lane] = in ? a.g8[o][i] : 0u;
      ss[lane] = in ? S[b] : 0u;
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
        const uint32_t s = sdup[l] >= 0 ? snew[sdup[l]] : ss[l];
        const bool hit = s != kNoIns32 && (uint64_t)(wcur - s) <= j.cap;
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
  __shared__ uint32_t swfin;
  __shared__ unsigned long long sfin[KV_MAX_GROUPS], sfinw[KV_MAX_GROUPS];
  if (lane == 0) swfin = wcur;
  if (lane < KV_MAX_GROUPS) sfin[lane] = sfinw[lane] = 0;
  __syncthreads();
  const uint32_t wf = swfin;
  for (uint64_t b = lane; b < a.u; b += kRNT) {
    const uint32_t s = S[b];
    if (s != kNoIns32 && (uint64_t)(wf - s) <= j.cap) {
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
}

// ---------------------------------------------------------------------------
// LFU.  The state is kept per trace position, not per block: cnt[p] is the
// block's in-cache count after its access at p (0: evicted), read through
// the next access's link to p.  Stores are therefore confined to the chunk
// being replayed.  Members of count class f in victim order are the
// positions of their latest accesses, so class f is a queue over positions
// scanned by a head pointer head[f].  Class 1 loses members oldest first, so
// a count-1 block whose latest access lies before head[1] has been evicted:
// those evictions need no store at all.  Member counts and a nonempty-class
// bitmap, in LDS (the workgroup owns its job for the whole replay), locate
// the lowest nonempty class.  Counts from kTopClass up share the top class:
// only when it is the lowest nonempty one (every resident block was touched
// over a thousand times while cached) is its victim needed, and then a scan
// of the job's positions finds the least (count, latest access).
// ---------------------------------------------------------------------------
struct LfuLds {
  // Small fields and the per-access fields of the hot loops come first, so
  // that they lie within reach of the LDS instructions' 16-bit offsets.
  uint32_t red[2][2 * kRNW];  // block scans, alternating (no trailing barrier)
  uint32_t sfx[2 * kRNW];
  uint32_t anyflag[2];
  uint32_t tot8[8];           // chunk totals: ev | n1 << 16, evicted weight, last old, last new
  uint64_t cnz[kLdsClassWords];
  uint64_t used;              // cached weight
  uint32_t fmin, head1;       // lowest nonempty class; no live count-1 member before head1
  uint32_t nc, h;             // candidate scan: entries found, next position
  uint64_t vw;                // candidate scan: untouched weight found
  int ok;
  // per access of the chunk (local position).  Members of one union serve
  // the fixed point and the apply step respectively, never both at once.
  union {
    struct {                  // fixed point
      uint8_t pw[kLChunk];    // weight
      uint8_t capm[kLChunk];  // stamp of the iteration that found a capacity miss here
      uint8_t mskip[kLChunk]; // the entry inserted here is promoted before its eviction
    };
    uint16_t occ[kLChunk];    // apply: earlier touches of the same block inside the chunk
  };
  uint8_t mcons[kLChunk];     // the entry inserted here is evicted inside the chunk
  // next touch relative to the chunk start: below L inside the chunk, up to
  // 2 * kLChunk in the next full chunk, else kInf16
  uint16_t nxloc[kLChunk];
  int16_t lp[kLChunk];        // previous touch in the chunk; pointer-jumped to the chain root
  union {
    uint16_t mpos[kLChunk];   // fixed point: local position of the m-th miss
    int16_t lmiss[kLChunk];   // apply: latest miss of the block at or before this touch
  };
  // fixed point: the weight that must have left the cache by the m-th miss;
  // apply: a block's count at the chunk start, at its first touch
  uint32_t mneed[kLChunk];
  uint32_t ccnt[kLdsClass];   // members of class f < kLdsClass
  union {
    struct {                  // count-1 residents from before the chunk, oldest first
      uint8_t cw[kCand];
      uint8_t cskip[kCand];
      uint8_t ccons[kCand];
      uint16_t ca[kCand];     // first touch inside the chunk or kInf16
      uint32_t cq[kCand];     // position of their last touch
    };
    struct {                  // serial walk over at most kMinFast accesses
      uint32_t skey[kMinFast];   // link
      uint32_t snx[kMinFast];    // next access
      uint32_t s0[kMinFast];     // count stored at a link before the walk
      uint32_t scnt[kMinFast];   // count stored here by the walk
      uint8_t sw[kMinFast];      // weight
      uint8_t sg[kMinFast];      // group
      uint32_t shead[kHeadLds];  // heads of the classes below kHeadLds
    };
  };
  // the next full chunk, per access: its block link and the stored count
  // at that link (each thread reads and writes only its own accesses)
  alignas(16) uint32_t pkey[kLChunk];
  alignas(16) uint32_t pcnt[kLChunk];
  // apply: the pointer jumping's second copies of lp, occ and lmiss (rounds
  // read one copy and write the other, so one barrier ends a round)
  int16_t lp2[kLChunk];
  uint16_t occ2[kLChunk];
  int16_t lmiss2[kLChunk];
  uint8_t cmf[kLChunk];       // a block's first touch in the chunk misses (no count at the start)
};

// A thread's IT consecutive words of an LDS array (16-byte aligned), moved
// four at a time.
template <int IT>
__device__ __forceinline__ void lds_get(const uint32_t* p, uint32_t* v) {
#pragma unroll
  for (int q = 0; q < IT / 4; ++q) {
    const uint4 x = reinterpret_cast<const uint4*>(p)[q];
    v[4 * q] = x.x;
    v[4 * q + 1] = x.y;
    v[4 * q + 2] = x.z;
    v[4 * q + 3] = x.w;
  }
}
template <int IT>
__device__ __forceinline__ void lds_put(uint32_t* p, const uint32_t* v) {
#pragma unroll
  for (int q = 0; q < IT / 4; ++q)
    reinterpret_cast<uint4*>(p)[q] = make_uint4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
}

// Nonempty-class bits from the class counts (whole block).
template <int NT>
__device__ __forceinline__ void class_bits_rebuild(LfuLds& S) {
  // each wavefront takes whole 64-class words (kLdsClass is a multiple of 64)
  for (uint32_t wd = (uint32_t)wave_id(); wd < kLdsClassWords; wd += NT / 64) {
    const uint64_t bal = __ballot(S.ccnt[wd * 64 + lane_id()] != 0u);
    if (lane_id() == 0) S.cnz[wd] = bal;
  }
}

// In-cache count of a block whose latest access is q with stored count c.
__device__ __forceinline__ uint32_t lfu_live_count(uint32_t c, uint64_t q, uint64_t head1) {
  return (c >= 2u || (c == 1u && q >= head1)) ? c : 0u;
}

struct Classes {
  uint32_t* lcnt;   // LDS member counts per class
  uint64_t* lnz;    // LDS nonempty-class bitmap words
};

// The class of a block of in-cache count f.
__device__ __forceinline__ uint32_t class_of(uint32_t f) { return min(f, kTopClass); }

// Lowest nonempty class >= f.
__device__ __forceinline__ uint32_t next_class(const Classes& c, uint32_t f) {
  for (uint32_t wi = f >> 6; wi < kLdsClassWords; ++wi) {
    uint64_t m = c.lnz[wi];
    if (wi == (f >> 6)) m &= ~0ull << (f & 63);
    if (m) return (wi << 6) + (uint32_t)__ffsll((long long)m) - 1u;
  }
  return 0xFFFFFFFFu;
}

__device__ __forceinline__ uint32_t class_count(const Classes& c, uint32_t f) {
  return c.lcnt[f];
}

// Serial update by one thread (the others wait at a barrier).
__device__ __forceinline__ void class_add1(const Classes& c, uint32_t f, int d) {
  const uint64_t bit = 1ull << (f & 63);
  if (d > 0) {
    if (c.lcnt[f]++ == 0u) c.lnz[f >> 6] |= bit;
  } else {
    if (--c.lcnt[f] == 0u) c.lnz[f >> 6] &= ~bit;
  }
}

// Concurrent count update; bitmap words are rebuilt afterwards.
__device__ __forceinline__ void class_add_par(const Classes& c, uint32_t f, int d) {
  if (d > 0) atomicAdd(&c.lcnt[f], 1u); else atomicSub(&c.lcnt[f], 1u);
}

// The serial walk's inputs for [p0, p1) (at most kMinFast accesses), staged
// in LDS by the whole block: per access its link, next access, weight and
// group, and for a link before p0 the count stored there; the heads of the
// classes below kHeadLds.
template <int NT>
__device__ __forceinline__ void lfu_serial_stage(const JobDev& j, const JobArgs& a,
                                                 const uint32_t* __restrict__ cnt,
                                                 const uint32_t* head, uint32_t n_class,
                                                 LfuLds& S, uint32_t p0, uint32_t p1) {
  const uint32_t o = j.order, b0 = (uint32_t)j.begin;
  for (uint32_t x = threadIdx.x; x < p1 - p0; x += NT) {
    const uint32_t i = p0 + x;
    uint32_t k = 0, nx = kNone, w = 0, g = 0, c = 0;
    if (i >= b0) {
      k = a.key[o][i];
      nx = a.nxt[o][i];
      w = a.w8[o][i];
      g = a.g8[o][i];
      if (k != 0 && k - 1 < p0) c = cnt[k - 1 - b0];
    }
    S.skey[x] = k;
    S.snx[x] = nx;
    S.sw[x] = (uint8_t)w;
    S.sg[x] = (uint8_t)g;
    S.s0[x] = c;
    S.scnt[x] = 0;
  }
  if (threadIdx.x < kHeadLds && threadIdx.x < n_class) S.shead[threadIdx.x] = head[threadIdx.x];
}

// Exact replay of the staged [p0, p1) by the 64 lanes of one wavefront.
// Every lane holds the same state and applies the same updates (stores of
// equal values to one address); only the victim search spreads candidate
// positions over the lanes.  Returns false if the state is found
// inconsistent.
__device__ __forceinline__ bool lfu_serial_wave(const JobDev& j, const JobArgs& a,
                                                uint32_t* __restrict__ cnt, uint32_t* head,
                                                uint32_t n_class, const Classes& cl, LfuLds& S,
                                                GroupCounters& gc, uint64_t* __restrict__ bits,
                                                uint32_t p0, uint32_t p1, uint64_t& used_io,
                                                uint32_t& head1_io) {
  const uint32_t o = j.order;
  const uint32_t b0 = (uint32_t)j.begin;
  const uint32_t lane = lane_id();
  uint32_t head1 = head1_io;
  uint64_t used = used_io;
  uint32_t fmin = S.fmin;
  uint64_t word = 0;
  bool ok = true;
  for (uint32_t i = p0; i < p1 && ok; ++i) {
    const uint32_t x = i - p0;
    if (i >= b0) {
      const uint32_t w = S.sw[x];
      const uint32_t k = S.skey[x];
      uint32_t f = 0;
      if (k != 0) f = lfu_live_count(k - 1 >= p0 ? S.scnt[k - 1 - p0] : S.s0[x], k - 1, head1);
      if (f) {
        word |= 1ull << (i & 63);
        const uint32_t f1 = f + 1;
        const uint32_t cf = class_of(f), cf1 = class_of(f1);
        if (cf != cf1) {
          class_add1(cl, cf, -1);
          class_add1(cl, cf1, +1);
          if (cf == fmin && class_count(cl, cf) == 0) fmin = cf1;
        }
        S.scnt[x] = f1;
        cnt[i - b0] = f1;
      } else {
        while (used + w > j.cap) {
          // the victim: the oldest live member of class fmin (it lies
          // before position i; the bound only guards against corrupted
          // state), or in the top class the least (count, latest access)
          uint32_t q = i, nq = kNone, vw = 0, vg = 0;
          if (fmin < kTopClass) {
            const uint32_t h0 = fmin == 1 ? head1 : (fmin < kHeadLds ? S.shead[fmin] : head[fmin]);
            for (uint32_t base = h0; base < i; base += 64) {
              const uint32_t r = base + lane;
              uint32_t c = 0, nr = kNone, wr = 0, gr = 0;
              if (r < i) {
                if (r >= p0) {
                  c = S.scnt[r - p0];
                  nr = S.snx[r - p0];
                  wr = S.sw[r - p0];
                  gr = S.sg[r - p0];
                } else {
                  c = cnt[r - b0];
                  nr = a.nxt[o][r];
                  wr = a.w8[o][r];
                  gr = a.g8[o][r];
                }
              }
              const uint64_t m = __ballot(r < i && c == fmin && (nr == kNone || nr >= i));
              if (m) {
                const int l = __ffsll((long long)m) - 1;
                q = base + (uint32_t)l;
                nq = (uint32_t)__builtin_amdgcn_readlane((int)nr, l);
                vw = (uint32_t)__builtin_amdgcn_readlane((int)wr, l);
                vg = (uint32_t)__builtin_amdgcn_readlane((int)gr, l);
                break;
              }
            }
          } else {
            uint64_t best = ~0ull;  // count << 32 | position
            for (uint32_t r = b0 + lane; r < i; r += 64) {
              const uint32_t c = r >= p0 ? S.scnt[r - p0] : cnt[r - b0];
              if (c < kTopClass) continue;
              const uint32_t nr = r >= p0 ? S.snx[r - p0] : a.nxt[o][r];
              if (nr != kNone && nr < i) continue;
              best = min(best, ((uint64_t)c << 32) | r);
            }
#pragma unroll
            for (int d = 32; d >= 1; d >>= 1) best = min(best, (uint64_t)__shfl_xor(best, d, 64));
            if (best != ~0ull) {
              q = (uint32_t)best;
              nq = q >= p0 ? S.snx[q - p0] : a.nxt[o][q];
              vw = q >= p0 ? S.sw[q - p0] : a.w8[o][q];
              vg = q >= p0 ? S.sg[q - p0] : a.g8[o][q];
            }
          }
          if (q >= i) {
            ok = false;
            break;
          }
          if (fmin == 1) head1 = q + 1;
          else if (fmin < kHeadLds) S.shead[fmin] = q + 1;
          else if (fmin < kTopClass) head[fmin] = q + 1;
          cnt[q - b0] = 0;
          // the access that links to q reads the eviction
          if (q >= p0) S.scnt[q - p0] = 0;
          else if (nq != kNone && nq < p1) S.s0[nq - p0] = 0;
          used -= vw;
          gc.ev[vg] += 1;
          gc.evw[vg] += vw;
          class_add1(cl, fmin, -1);
          if (class_count(cl, fmin) == 0) {
            const uint32_t nf = next_class(cl, fmin);
            if (nf != 0xFFFFFFFFu) fmin = nf;
          }
        }
        S.scnt[x] = 1;
        cnt[i - b0] = 1;
        class_add1(cl, 1, +1);
        fmin = 1;
        used += w;
        const uint32_t g = S.sg[x];
        gc.ins[g] += 1;
        gc.insw[g] += w;
      }
    }
    if ((i & 63) == 63 || i + 1 == p1) {
      if (i >= b0 || (i | 63) >= b0) bits[(i >> 6) - j.word0] = word;
      word = 0;
    }
  }
  if (lane >= 2 && lane < kHeadLds && lane < n_class) head[lane] = S.shead[lane];
  S.fmin = fmin;
  used_io = used;
  head1_io = head1;
  return ok;
}

constexpr int kWin = 8;                           // demands searched in registers

// Exclusive suffix minimum over the threads of the block (threads above t)
// of values below 2^31, and whether any thread raised `flag`; one barrier.
// `sh` (NT / 64 words) may be written again only after another barrier.
template <int NT>
__device__ __forceinline__ void block_suffix_min_flag(uint32_t v, bool flag, uint32_t* sh,
                                                      uint32_t& smin, bool& any) {
  constexpr int NW = NT / 64;
  constexpr int kInf = 0x7FFFFFFF;
  const uint32_t lane = lane_id();
  const int w = wave_id();
  // inclusive suffix minimum within rows of 16 lanes (row_shl: from lane + n)
  int x = (int)v;
  x = min(x, __builtin_amdgcn_update_dpp(kInf, x, 0x101, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(kInf, x, 0x102, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(kInf, x, 0x104, 0xf, 0xf, false));
  x = min(x, __builtin_amdgcn_update_dpp(kInf, x, 0x108, 0xf, 0xf, false));
  // ... then across rows, from the row heads
  const int r1 = __builtin_amdgcn_readlane(x, 16), r2 = __builtin_amdgcn_readlane(x, 32),
            r3 = __builtin_amdgcn_readlane(x, 48);
  const int row = (int)(lane >> 4);
  x = min(x, row < 3 ? r3 : kInf);
  x = min(x, row < 2 ? r2 : kInf);
  x = min(x, row < 1 ? r1 : kInf);
  const int wmin = __builtin_amdgcn_readlane(x, 0);
  // exclusive: the next lane's inclusive value (wave_shl:1; lane 63 gets none)
  int r = __builtin_amdgcn_update_dpp(kInf, x, 0x130, 0xf, 0xf, false);
  const bool wflag = __ballot(flag) != 0ull;
  if (lane == 0) sh[w] = (uint32_t)wmin | (wflag ? 0x80000000u : 0u);
  __syncthreads();
  // the waves' minima and flags, one per lane of the first row: a suffix
  // minimum across the row, read at wave w + 1
  static_assert(NW <= 16, "one row of lanes holds the wave minima");
  const uint32_t y = lane < (uint32_t)NW ? sh[lane] : (uint32_t)kInf;
  any = __ballot((y >> 31) != 0u) != 0ull;
  int z = (int)(y & 0x7FFFFFFFu);
  z = min(z, __builtin_amdgcn_update_dpp(kInf, z, 0x101, 0xf, 0xf, false));
  z = min(z, __builtin_amdgcn_update_dpp(kInf, z, 0x102, 0xf, 0xf, false));
  z = min(z, __builtin_amdgcn_update_dpp(kInf, z, 0x104, 0xf, 0xf, false));
  z = min(z, __builtin_amdgcn_update_dpp(kInf, z, 0x108, 0xf, 0xf, false));
  if (w + 1 < NW) r = min(r, __builtin_amdgcn_readlane(z, w + 1));
  smin = (uint32_t)r;
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
//
// The count-1 residents from before the chunk are found without reading the
// block states: every count-1 member at or after head1 is a block inserted
// by a miss at that position and not touched since, and every such block is
// still a member (count-1 members only leave by a touch or, oldest first, by
// eviction, which moves head1 past them).
// G1: every access of the job belongs to group g0 (counters add up per
// wavefront); otherwise each access's group is read.
// The next full chunk's weights and next-access links and the block links
// of the chunk after it, loaded at the end of a full chunk (after its last
// awaited load, so that no wait of its own covers them) and kept in
// registers until the next chunk reads them.
template <int IT>
struct LfuAhead {
  uint32_t w[IT / 4];   // four weights per word
  uint4 nx[IT / 4];
  uint4 key[IT / 4];
};

template <int NT, bool G1>
__device__ __forceinline__ bool lfu_fast(const JobDev& j, const JobArgs& a,
                                         uint32_t* __restrict__ cnt, const Classes& cl,
                                         GroupCounters& gc, LfuLds& S,
                                         uint64_t* __restrict__ bits, uint32_t c0, uint32_t c1,
                                         uint32_t g0, BlockAny& block_any, bool have_pref,
                                         uint64_t& used_io, uint32_t& head1_io,
                                         LfuAhead<kLChunk / NT>& ahead) {
  constexpr bool g1 = G1;
  constexpr int IT = kLChunk / NT;               // accesses per thread
  // queue entries per thread: the queue rarely holds more than about a
  // chunk's worth (NT * CPT); a longer one fails the chunk, which is then
  // retried shorter
  constexpr int CPT = kLChunk / NT + 1;
  static_assert(IT % 4 == 0 && IT <= 64, "accesses are loaded four at a time");
  const uint32_t tid = threadIdx.x;
  const uint32_t o = j.order;
  // positions fit in 32 bits (n <= 2^29), as do the capacities of replayed
  // jobs (below the trace's distinct weight, itself below 2^32)
  const uint32_t jb = (uint32_t)j.begin, je = (uint32_t)j.end, jw0 = (uint32_t)j.word0;
  const uint32_t L = c1 - c0;
  const uint32_t l0 = tid * IT;
  const uint32_t p0 = c0 + l0;
  ItemBits v;
#pragma unroll
  for (int e = 0; e < IT; ++e) v.set(e, l0 + e < L && p0 + e >= jb);
  uint32_t ww[IT], gg[IT], kk[IT], nx[IT], f0[IT];
  bool cm[IT], res0[IT];
  if (have_pref) {
    lds_get<IT>(S.pkey + l0, kk);
#pragma unroll
    for (int q = 0; q < IT / 4; ++q) {
      const uint32_t xn[4] = {ahead.nx[q].x, ahead.nx[q].y, ahead.nx[q].z, ahead.nx[q].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ww[4 * q + e] = v[4 * q + e] ? (ahead.w[q] >> (8 * e)) & 0xFFu : 0u;
        nx[4 * q + e] = v[4 * q + e] ? xn[e] : 0u;
      }
    }
  } else {
    loadn_u32<IT>(a.key[o], p0, a.n, v, kk);
    loadn_u8<IT>(a.w8[o], p0, a.n, v, ww);
    loadn_u32<IT>(a.nxt[o], p0, a.n, v, nx);
  }
  {
    // the next full chunk's block links.  The read position is clamped to
    // the arrays' readable slack; whatever lies outside the job (or past n,
    // where the slack holds no links) becomes 0, no earlier access.
    const uint32_t pnext = c0 + kLChunk + l0;
    const uint32_t pn = min<uint32_t>(pnext, (uint32_t)a.n & ~3u);
    uint32_t nk[IT];
#pragma unroll
    for (int q = 0; q < IT / 4; ++q) {
      const uint4 x = have_pref ? ahead.key[q]
                                : *reinterpret_cast<const uint4*>(a.key[o] + pn + 4 * q);
      const uint32_t xv[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t pe = pnext + 4 * q + r;
        nk[4 * q + r] = (pn == pnext && pe >= jb && pe < je) ? xv[r] : 0u;
      }
    }
    lds_put<IT>(S.pkey + l0, nk);
  }
#pragma unroll
  for (int e = 0; e < IT; ++e) gg[e] = g0;
  if constexpr (!G1) loadn_u8<IT>(a.g8[o], p0, a.n, v, gg);
  uint32_t h = head1_io;
  // the candidate scan's first step, loaded ahead (whether it runs is known
  // only after the first block scan).  The links and weights never change;
  // a hit word is taken from here only for positions at least a full chunk
  // back, whose words were stored before a barrier every wave has passed
  // (the previous chunk stores its own after its last one).
  uint64_t sc_word[kCScan];
  uint32_t sc_nx[kCScan], sc_w[kCScan];
  {
    const uint32_t hend = min(min<uint32_t>(h + NT * kCScan, h + kCand), c0);
#pragma unroll
    for (int e = 0; e < kCScan; ++e) {
      const uint32_t q = h + tid * kCScan + e;
      sc_word[e] = 0;
      sc_nx[e] = kNone;
      sc_w[e] = 0;
      if (q < hend) {
        if (q + kLChunk < c0) sc_word[e] = bits[(q >> 6) - jw0];
        sc_nx[e] = a.nxt[o][q];
        sc_w[e] = a.w8[o][q];
      }
    }
  }
  // stored counts at the latest earlier accesses (prefetched by the
  // previous chunk when it covered the whole chunk before this one); only a
  // block's first access in the chunk needs one
  uint32_t s0[IT];
  if (have_pref) {
    lds_get<IT>(S.pcnt + l0, s0);
  } else {
#pragma unroll
    for (int e = 0; e < IT; ++e) {
      const bool old_prev = v[e] && kk[e] != 0 && kk[e] - 1 < c0;
      s0[e] = cnt[old_prev ? kk[e] - 1 - jb : 0];
      if (!old_prev) s0[e] = 0;
    }
  }
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t loc = l0 + e;
    const int lp = (kk[e] != 0 && kk[e] - 1 >= c0) ? (int)(kk[e] - 1 - c0) : -1;
    const bool again = v[e] && nx[e] != kNone && nx[e] < c1;
    S.lp[loc] = (int16_t)lp;
    // the block's count at the chunk start (first accesses only)
    f0[e] = (v[e] && kk[e] != 0 && lp < 0) ? lfu_live_count(s0[e], kk[e] - 1, h) : 0u;
    res0[e] = f0[e] != 0;
    cm[e] = v[e] && lp < 0 && !res0[e];
    S.nxloc[loc] = (v[e] && nx[e] != kNone && nx[e] - c0 < 2 * kLChunk) ? (uint16_t)(nx[e] - c0)
                                                                        : kInf16;
    S.pw[loc] = (uint8_t)ww[e];
    S.capm[loc] = 0;
    S.cmf[loc] = cm[e] ? 1 : 0;
    S.mskip[loc] = again ? 1 : 0;
    S.mcons[loc] = 0;
  }
  // the first-touch misses: the fixed point's first miss list
  uint32_t x = 0, xc = 0;
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    x += cm[e] ? ww[e] : 0u;
    xc += cm[e] ? 1u : 0u;
  }
  uint32_t itot0, nm0, wpre0, mpre0;
  // block scans alternate between two LDS buffers and skip their trailing
  // barrier (every call has a barrier, so a buffer is reused only after
  // all threads have left the call before)
  uint32_t rg = 0;
  block_excl_scan2_u32<NT, false>(x, xc, S.red[rg++ & 1], wpre0, mpre0, itot0, nm0);
  // past the chunk's first barrier every thread has left the previous
  // chunk, which read the totals last
  if (tid < 8) S.tot8[tid] = 0;
  const uint64_t used0 = used_io;
  // evictions the chunk needs never exceed its insertions (used0 <= cap)
  const uint32_t ev0 = (used0 + itot0 > j.cap) ? (uint32_t)(used0 + itot0 - j.cap) : 0u;
  // used0 - cap, clamped so that adding a chunk's miss weight stays in 32 bits
  const int32_t room = (int32_t)max<int64_t>((int64_t)used0 - (int64_t)j.cap, -(1ll << 30));
  if (ev0 > 0) {
#pragma unroll
    for (int e = 0; e < IT; ++e) {
      if (cm[e]) {
        wpre0 += ww[e];
        const int32_t need = room + (int32_t)wpre0;
        S.mpos[mpre0] = (uint16_t)(l0 + e);
        S.mneed[mpre0] = need > 0 ? (uint32_t)need : 0u;
        ++mpre0;
      }
    }
  }
  uint32_t nc0 = 0;
  bool reached = false;
  if (ev0 > 0) {
    // count-1 residents from head1 on, until the untouched ones alone cover
    // the first-touch demand (a capacity miss adds as much demand as it adds
    // victims), the chunk start is reached, or the buffer is full
    uint32_t n0 = 0;
    uint64_t vw = 0;
    for (bool first = true;; first = false) {
      if (vw >= ev0 || h >= c0 || n0 >= kCand) break;
      // each position lists at most one entry: near the end of the buffer
      // the step shrinks to the room left
      const uint32_t hend = min(min<uint32_t>(h + NT * kCScan, h + (kCand - n0)), c0);
      bool live[kCScan], touched[kCScan];
      uint32_t wq[kCScan], aq[kCScan];
#pragma unroll
      for (int e = 0; e < kCScan; ++e) {
        const uint32_t q = h + tid * kCScan + e;
        live[e] = false;
        touched[e] = false;
        aq[e] = kInf16;
        wq[e] = 0;
        if (q < hend) {
          const uint64_t word = (first && q + kLChunk < c0) ? sc_word[e] : bits[(q >> 6) - jw0];
          const uint32_t nxq = first ? sc_nx[e] : a.nxt[o][q];
          wq[e] = first ? sc_w[e] : a.w8[o][q];
          live[e] = !((word >> (q & 63)) & 1ull) && (nxq == kNone || nxq >= c0);
          touched[e] = live[e] && nxq != kNone && nxq < c1;
          aq[e] = touched[e] ? nxq - c0 : kInf16;
        }
      }
      uint32_t cl_ = 0, cw_ = 0;
#pragma unroll
      for (int e = 0; e < kCScan; ++e) {
        cl_ += live[e] ? 1u : 0u;
        cw_ += (live[e] && !touched[e]) ? wq[e] : 0u;
      }
      uint32_t pos, dummy, cnt_live, vsum;
      block_excl_scan2_u32<NT, false>(cl_, cw_, S.red[rg++ & 1], pos, dummy, cnt_live, vsum);
#pragma unroll
      for (int e = 0; e < kCScan; ++e) {
        if (!live[e]) continue;
        const uint32_t k = n0 + pos++;
        S.cq[k] = h + tid * kCScan + e;
        S.cw[k] = (uint8_t)wq[e];
        S.ca[k] = (uint16_t)aq[e];
        S.cskip[k] = touched[e] ? 1 : 0;
        S.ccons[k] = 0;
      }
      n0 += cnt_live;
      vw += vsum;
      h = hend;
    }
    __syncthreads();
    nc0 = n0;
    reached = h >= c0;
    // positions before the first live entry hold no count-1 member any more
    h = nc0 ? S.cq[0] : h;
  } else {
    h = head1_io;
  }
  // ---- fixed point over (misses, promotions, evictions)
  uint32_t itot = itot0;   // weight of the chunk's misses (insertions)
  uint32_t nmiss = nm0;     // and their number
  bool converged = ev0 == 0;
  bool capnow[IT];  // capacity misses of the latest iteration
  uint32_t ns_last = 0;  // the latest iteration's stamp in capm (0: none ran)
#pragma unroll
  for (int e = 0; e < IT; ++e) capnow[e] = false;
  for (int it = 0; !converged && it < 24; ++it) {
    bool mi[IT], oldcap[IT];
    uint32_t nm = nm0;
#pragma unroll
    for (int e = 0; e < IT; ++e) {
      oldcap[e] = false;
      mi[e] = cm[e];
    }
    if (it > 0) {  // the first miss list is the first touches, listed above
      uint32_t xw = 0, xm = 0;
#pragma unroll
      for (int e = 0; e < IT; ++e) {
        oldcap[e] = capnow[e];
        mi[e] = cm[e] || oldcap[e];
        xw += mi[e] ? ww[e] : 0u;
        xm += mi[e] ? 1u : 0u;
      }
      uint32_t wpre, mpre;
      block_excl_scan2_u32<NT, false>(xw, xm, S.red[rg++ & 1], wpre, mpre, itot, nm);
#pragma unroll
      for (int e = 0; e < IT; ++e) {
        if (mi[e]) {
          wpre += ww[e];
          const int32_t need = room + (int32_t)wpre;
          S.mpos[mpre] = (uint16_t)(l0 + e);
          S.mneed[mpre] = need > 0 ? (uint32_t)need : 0u;
          ++mpre;
        }
      }
      __syncthreads();
    }
    nmiss = nm;
    const uint32_t evtot = (used0 + itot > j.cap) ? (uint32_t)(used0 + itot - j.cap) : 0u;
    // the eviction queue: nc0 old entries, then the nm insertions of the
    // chunk; thread t holds entries t*qpt .. t*qpt+qpt-1
    const uint32_t nq = nc0 + nm;
    const uint32_t qpt = (nq + NT - 1) / NT;
    if (qpt > (uint32_t)CPT) {
      return false;
    }
    uint32_t qw[CPT];
    uint32_t xs = 0;
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      const uint32_t k = (uint32_t)e < qpt ? tid * qpt + e : nq;
      qw[e] = 0;
      if (k < nc0) qw[e] = S.cskip[k] ? 0u : S.cw[k];
      else if (k < nq) {
        const uint32_t m = S.mpos[k - nc0];
        qw[e] = S.mskip[m] ? 0u : S.pw[m];
      }
      xs += qw[e];
    }
    uint32_t elig;
    uint32_t run = block_excl_scan_u32<NT, false>(xs, S.red[rg++ & 1], elig);
    bool bad = elig < evtot;
    // entry k is consumed by the first miss whose demand exceeds the
    // eligible weight queued before k.  Demands and prefixes both rise, so
    // a thread's answers lie between the answers for its first and last
    // prefixes; a window of kWin demands usually holds them all.
    uint32_t evk[CPT];
    {
      const uint32_t r_lo = run;
      uint32_t r_hi = run;
      {
        uint32_t rr = run;
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          const uint32_t k = (uint32_t)e < qpt ? tid * qpt + e : nq;
          if (k < nq && qw[e] && rr < evtot) r_hi = rr;
          rr += qw[e];
        }
      }
      const bool active = r_lo < evtot && tid * qpt < nq;
      uint32_t lo = active ? upper_bound(S.mneed, 0u, nm, r_lo) : 0u;
      uint32_t win[kWin];
#pragma unroll
      for (int t = 0; t < kWin; ++t) win[t] = lo + t < nm ? S.mneed[lo + t] : 0xFFFFFFFFu;
      // the window holds every answer when its last demand exceeds r_hi (or
      // it reaches past the last miss)
      const bool inwin = lo + kWin >= nm || win[kWin - 1] > r_hi;
#pragma unroll
      for (int e = 0; e < CPT; ++e) {
        const uint32_t k = (uint32_t)e < qpt ? tid * qpt + e : nq;
        evk[e] = kInf16;
        if (k < nq && qw[e] && run < evtot) {
          uint32_t idx;
          if (inwin) {
            idx = lo;
#pragma unroll
            for (int t = 0; t < kWin; ++t) idx += win[t] <= run ? 1u : 0u;
          } else {
            idx = upper_bound(S.mneed, lo, nm, run);
            lo = idx;
          }
          evk[e] = (idx < nm) ? S.mpos[idx] : kInf16;
          if (k >= nc0) {
            // a new entry can only go after it was inserted, and only once
            // every old one is gone
            if (evk[e] <= S.mpos[k - nc0] || !reached) bad = true;
          }
        }
        run += qw[e];
      }
    }
    // the pointer reaches entry k when the first consumed entry at or after k goes
    uint32_t suf[CPT];
    uint32_t mn = kInf16;
#pragma unroll
    for (int e = CPT - 1; e >= 0; --e) {
      mn = min(mn, evk[e]);
      suf[e] = mn;
    }
    uint32_t tmin;
    bool anybad;
    block_suffix_min_flag<NT>(mn, bad, S.sfx, tmin, anybad);
    // A shortfall of count-1 victims found here may be an artefact of the
    // skip flags, which start out assuming that every entry touched in the
    // chunk is touched before its turn: the update below can make such an
    // entry eligible.  A chunk fails only if a shortfall outlives the last
    // change.
    // the inputs of an iteration are the skip flags and the capacity
    // misses; the consumption flags are its outputs
    const uint8_t ns = (uint8_t)(it + 1);
    ns_last = ns;
    bool changed = false;
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      const uint32_t k = (uint32_t)e < qpt ? tid * qpt + e : nq;
      if (k >= nq) continue;
      const uint32_t ptime = min(suf[e], tmin);
      const bool cons = evk[e] != kInf16;
      uint32_t ak = (k < nc0) ? (uint32_t)S.ca[k] : (uint32_t)S.nxloc[S.mpos[k - nc0]];
      if (ak >= L) ak = kInf16;  // next touch beyond the chunk
      const bool nskip = ak != kInf16 && (ptime == kInf16 || ak <= ptime);
      const bool ncap = ak != kInf16 && !nskip && ptime != kInf16;
      if (k < nc0) {
        changed |= nskip != (S.cskip[k] != 0);
        S.cskip[k] = nskip ? 1 : 0;
        S.ccons[k] = cons ? 1 : 0;
      } else {
        const uint32_t m = S.mpos[k - nc0];
        changed |= nskip != (S.mskip[m] != 0);
        S.mskip[m] = nskip ? 1 : 0;
        S.mcons[m] = cons ? 1 : 0;
      }
      if (ncap) S.capm[ak] = ns;  // each touch position is the next touch of one entry
    }
    __syncthreads();
#pragma unroll
    for (int e = 0; e < IT; ++e) {
      const uint32_t loc = l0 + e;
      capnow[e] = v[e] && S.capm[loc] == ns;
      changed |= oldcap[e] != capnow[e];
      // entries that stopped being misses lose their queue flags (their
      // miss status changed with the capacity misses, counted above)
      if (v[e] && !mi[e] && S.mcons[loc]) S.mcons[loc] = 0;
    }
    if (!block_any(changed)) {
      if (anybad) {
        return false;
      }
      converged = true;
    }
  }
  if (!converged) {
    return false;
  }
  // ---- consistent: apply.  First the next chunk's stored counts at links
  // before this chunk (final already; a link inside it reads this chunk's
  // final counts once they are known).
  uint32_t nold[IT], nk[IT];
  lds_get<IT>(S.pkey + l0, nk);
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t k = nk[e];
    const bool old = k != 0 && k - 1 < c0;
    nold[e] = cnt[old ? k - 1 - jb : 0];
    if (!old) nold[e] = 0;
  }
  // Pointer jumping gives each touch the number of earlier touches of its
  // block in the chunk and the latest miss among them.
  bool miss[IT];
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    miss[e] = cm[e] || capnow[e];
    S.mneed[l0 + e] = f0[e];  // a block's count at the chunk start, read via its first access
  }
  // Rounds read copy A of (lp, occ, lmiss) and write copy B; the final
  // values end up in B.  Round 0 needs no copy A: a touch's initial occ is
  // 1 if it has an earlier touch in the chunk, and its initial lmiss is
  // itself if it misses (a first-touch miss, or a capacity miss of the
  // fixed point's last iteration), from fields every thread sees already.
  // (Copy A's occ and lmiss share storage with the fixed point's pw, capm,
  // mskip and mpos: round 0 still reads capm, and copy A is first written
  // in round 1, after the barrier that ends round 0.)
  int16_t *lpA = S.lp, *lpB = S.lp2, *lmA = S.lmiss, *lmB = S.lmiss2;
  uint16_t *ocA = S.occ, *ocB = S.occ2;
  bool moved0 = false;
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t loc = l0 + e;
    const int16_t p = S.lp[loc];
    uint16_t no = p >= 0 ? 1 : 0;
    int16_t np = p, nl = miss[e] ? (int16_t)loc : (int16_t)-1;
    if (p >= 0) {
      const int16_t pp = S.lp[p];
      if (pp >= 0) {
        no = (uint16_t)(no + 1);
        np = pp;
        moved0 = true;
      }
      if (nl < 0 && (S.cmf[p] || (ns_last != 0 && S.capm[p] == ns_last))) nl = p;
    }
    lpB[loc] = np;
    ocB[loc] = no;
    lmB[loc] = nl;
  }
  if (block_any(moved0)) {
    for (;;) {
      int16_t* t16 = lpA;
      lpA = lpB;
      lpB = t16;
      t16 = lmA;
      lmA = lmB;
      lmB = t16;
      uint16_t* tu = ocA;
      ocA = ocB;
      ocB = tu;
      int16_t np[IT], nl[IT];
      uint16_t no[IT];
      bool moved = false;
#pragma unroll
      for (int e = 0; e < IT; ++e) {
        const uint32_t loc = l0 + e;
        const int16_t p = lpA[loc];
        no[e] = ocA[loc];
        np[e] = p;
        nl[e] = lmA[loc];
        if (p >= 0) {
          const int16_t pp = lpA[p];
          if (pp >= 0) {
            no[e] = (uint16_t)(no[e] + ocA[p]);
            np[e] = pp;
            moved = true;
          }
          if (nl[e] < 0) nl[e] = lmA[p];
        }
      }
#pragma unroll
      for (int e = 0; e < IT; ++e) {
        const uint32_t loc = l0 + e;
        lpB[loc] = np[e];
        ocB[loc] = no[e];
        lmB[loc] = nl[e];
      }
      if (!block_any(moved)) break;
    }
  }
  // per-thread partials: evictions (and, 16 bits up, old count-1 entries
  // leaving class 1), evicted weight, last entries taken.  Insertions are
  // the misses, counted by the fixed point.
  uint32_t p_evn = 0, p_vw = 0, p_lastp = 0, p_laste = 0;
  // old entries evicted (loads issued unconditionally, several in flight)
  for (uint32_t k = tid; k < nc0; k += NT) {
    const bool cons = S.ccons[k] != 0;
    const uint32_t w = S.cw[k];
    const bool untouched = S.ca[k] == kInf16;
    if (!cons) continue;
    if (g1) {
      ++p_evn;
    } else {
      const uint32_t g = a.g8[o][S.cq[k]];
      atomicAdd(&gc.ev[g], 1ull);
      atomicAdd(&gc.evw[g], (unsigned long long)w);
    }
    p_vw += w;
    p_lastp = max(p_lastp, k + 1);
    // not touched again in the chunk: leaves class 1 for good (head1 passes
    // it: no store)
    if (untouched) p_evn += 1u << 16;
  }
  // per-access chunk data, loaded for all items at once
  uint32_t mc[IT], nxl[IT], lm[IT], oc[IT];
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t loc = l0 + e;
    mc[e] = S.mcons[loc];
    nxl[e] = S.nxloc[loc];
    lm[e] = (uint32_t)(int32_t)lmB[loc];
    oc[e] = ocB[loc];
  }
  uint32_t mocc[IT], mcm[IT], rf0[IT];
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t m = (int32_t)lm[e] >= 0 ? lm[e] : 0u;
    mocc[e] = ocB[m];
    mcm[e] = S.mcons[m];
    const int16_t r = lpB[l0 + e];  // the block's first access in the chunk
    rf0[e] = r >= 0 ? S.mneed[r] : f0[e];
  }
  bool hit[IT];
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    hit[e] = v[e] && !miss[e];
    if (!(v[e] && miss[e])) continue;
    const bool cons = mc[e] != 0;  // inserted here, evicted later in the chunk
    if (g1) {
      p_evn += cons ? 1u : 0u;
    } else {
      atomicAdd(&gc.ins[gg[e]], 1ull);
      atomicAdd(&gc.insw[gg[e]], (unsigned long long)ww[e]);
      if (cons) {
        atomicAdd(&gc.ev[gg[e]], 1ull);
        atomicAdd(&gc.evw[gg[e]], (unsigned long long)ww[e]);
      }
    }
    if (cons) {
      p_vw += ww[e];
      p_laste = e + 1;  // items run in position order: the last one wins
    }
  }
  const uint32_t p_lastm = p_laste ? l0 + p_laste : 0u;
  // final state of every touched block, at its last touch.  Moves into and
  // out of classes 1 and 2 (the crowded ones) add up per wavefront by
  // ballot; the others go one by one.
  uint32_t fnew[IT];
  bool fin[IT];
  int d12[2] = {0, 0};
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    fnew[e] = 0;
    fin[e] = v[e] && nxl[e] >= L;
    if (fin[e]) {
      if ((int32_t)lm[e] >= 0) {
        fnew[e] = mcm[e] ? 0u : oc[e] - mocc[e] + 1u;
      } else {
        fnew[e] = rf0[e] + oc[e] + 1u;
      }
      // the block's next access opens the next full chunk's prefetch slot
      if (L == kLChunk && nxl[e] != kInf16) S.pcnt[nxl[e] - kLChunk] = fnew[e];
    }
    const uint32_t fo = fin[e] ? rf0[e] : 0u, fn = fnew[e];
#pragma unroll
    for (int c = 0; c < 2; ++c)
      d12[c] += __popcll(__ballot(fn == (uint32_t)(c + 1))) -
                __popcll(__ballot(fo == (uint32_t)(c + 1)));
    const uint32_t co = class_of(fo), cn = class_of(fn);
    if (co != cn) {
      if (fo > 2) class_add_par(cl, co, -1);
      if (fn > 2) class_add_par(cl, cn, +1);
    }
  }
  // the counts at the chunk's positions: the final ones at last touches, 0
  // at the others (never read: a later access links to a later touch).
  // Stored unconditionally (items outside the job go to the slot past its
  // end), so that waits for the earlier gather need not cover them.
#pragma unroll
  for (int e = 0; e < IT; ++e) cnt[v[e] ? c0 + l0 + e - jb : je - jb] = fin[e] ? fnew[e] : 0u;
  if (lane_id() == 0) {
    if (d12[0]) atomicAdd(&S.ccnt[1], (uint32_t)d12[0]);
    if (d12[1]) atomicAdd(&S.ccnt[2], (uint32_t)d12[1]);
  }
  {
    const uint32_t r[4] = {wave_add_dpp(p_evn), wave_add_dpp(p_vw), wave_max_dpp(p_lastp),
                           wave_max_dpp(p_lastm)};
    if (lane_id() == 0) {
      if (r[0]) atomicAdd(&S.tot8[0], r[0]);
      if (r[1]) atomicAdd(&S.tot8[1], r[1]);
      if (r[2]) atomicMax(&S.tot8[2], r[2]);
      if (r[3]) atomicMax(&S.tot8[3], r[3]);
      if (r[0] >> 16) atomicSub(&S.ccnt[1], r[0] >> 16);
    }
  }
  __syncthreads();
  // the next chunk's stored counts at links before this chunk (a link
  // inside it was filled in by its last touch above; only a link before the
  // next chunk is ever read)
#pragma unroll
  for (int e = 0; e < IT; ++e) {
    const uint32_t k = nk[e];
    if (!(k != 0 && k - 1 >= c0 && k - 1 < c0 + kLChunk)) S.pcnt[l0 + e] = nold[e];
  }
  if (L == kLChunk) {
    // read positions clamped as for the links above: a clamped group lies
    // wholly past n, where the next chunks mask every item
    const uint32_t nmax = (uint32_t)a.n & ~3u;
    const uint32_t pn1 = min<uint32_t>(c0 + kLChunk + l0, nmax);
    const uint32_t pn2 = min<uint32_t>(c0 + 2 * kLChunk + l0, nmax);
#pragma unroll
    for (int q = 0; q < IT / 4; ++q) {
      ahead.w[q] = *reinterpret_cast<const uint32_t*>(a.w8[o] + pn1 + 4 * q);
      ahead.nx[q] = *reinterpret_cast<const uint4*>(a.nxt[o] + pn1 + 4 * q);
      ahead.key[q] = *reinterpret_cast<const uint4*>(a.key[o] + pn2 + 4 * q);
    }
  }
  // the nonempty-class bitmap is rebuilt only when class 1 is empty (the
  // serial walk rebuilds it before it starts)
  const bool c1empty = S.ccnt[1] == 0u;
  if (c1empty) class_bits_rebuild<NT>(S);
  store_hits_n<IT>(hit, c0, L, j, bits);
  // every thread takes the chunk totals: the cached weight and the count-1
  // queue head go on in registers, with no barrier to end the chunk (the
  // next chunk's writes touch nothing read here)
  const uint32_t t_ev = S.tot8[0] & 0xFFFFu, t_vw = S.tot8[1], t_lastp = S.tot8[2],
                 t_lastm = S.tot8[3];
  if (g1 && tid == 0) {
    gc.ins[g0] += nmiss;
    gc.insw[g0] += itot;
    gc.ev[g0] += t_ev;
    gc.evw[g0] += t_vw;
  }
  used_io = used0 + itot - t_vw;
  if (t_lastm) head1_io = c0 + t_lastm;                 // last new entry taken + 1
  else if (t_lastp) head1_io = S.cq[t_lastp - 1] + 1;   // last old entry taken + 1
  else head1_io = h;
  if (c1empty) {
    // the lowest nonempty class, for the serial walk (class 1 otherwise)
    __syncthreads();
    if (tid == 0) {
      const uint32_t nf = next_class(cl, 1);
      if (nf != 0xFFFFFFFFu) S.fmin = nf;
    }
  } else if (tid == 0) {
    S.fmin = 1;
  }
  return true;
}

template <int NT, bool G1>
__device__ __forceinline__ void lfu_chunked(const JobDev& j, const JobArgs& a,
                                            uint32_t* __restrict__ cnt, uint32_t* __restrict__ cls,
                                            uint64_t* __restrict__ bits, GroupCounters& gc,
                                            LfuLds& S, uint32_t g0) {
  const uint32_t tid = threadIdx.x;
  uint32_t* head = cls + j.class_off;
  Classes cl;
  cl.lcnt = S.ccnt;
  cl.lnz = S.cnz;
  for (uint32_t f = tid; f < kLdsClass; f += NT) S.ccnt[f] = 0;
  if (tid < kLdsClassWords) S.cnz[tid] = 0;
  if (tid < 2) S.anyflag[tid] = 0;
  BlockAny block_any{S.anyflag, 0};
  if (tid == 0) {
    S.fmin = 1;
    S.ok = 1;
  }
  __syncthreads();
  uint64_t pos = j.begin & ~63ull;
  uint32_t len = j.chunk;
  uint64_t ppos = ~0ull;  // the chunk whose links and counts are prefetched in LDS
  uint64_t used = 0;                    // cached weight
  uint32_t head1 = (uint32_t)j.begin;   // no live count-1 member before head1
  LfuAhead<kLChunk / NT> ahead;
  while (pos < j.end) {
    const uint32_t l = (uint32_t)min<uint64_t>(len, j.end - pos);
    if (lfu_fast<NT, G1>(j, a, cnt, cl, gc, S, bits, (uint32_t)pos, (uint32_t)(pos + l), g0,
                         block_any, ppos == pos, used, head1, ahead)) {
      ppos = (l == kLChunk) ? pos + l : ~0ull;
      pos += l;
      len = min<uint32_t>(len * 2, j.chunk);
    } else if (l > kMinFast) {
      len = max<uint32_t>(kMinFast, (l / 2) & ~63u);
      ppos = ~0ull;  // the failed attempt replaced the prefetched links
    } else {
      __syncthreads();
      class_bits_rebuild<NT>(S);
      lfu_serial_stage<NT>(j, a, cnt, head, a.n_class, S, (uint32_t)pos, (uint32_t)(pos + l));
      __syncthreads();
      if (wave_id() == 0) {
        const bool ok = lfu_serial_wave(j, a, cnt, head, a.n_class, cl, S, gc, bits,
                                        (uint32_t)pos, (uint32_t)(pos + l), used, head1);
        if (lane_id() == 0) {
          S.ok = ok ? 1 : 0;
          S.used = used;
          S.head1 = head1;
        }
      }
      __syncthreads();
      used = S.used;
      head1 = S.head1;
      if (!S.ok) break;
      pos += l;
      ppos = ~0ull;
    }
  }
  __syncthreads();
}


// Whether every access of a job belongs to one group (a partitioned job, or
// a trace with one group).
__host__ __device__ __forceinline__ bool lfu_one_group(const JobDev& j, uint32_t n_groups) {
  return n_groups == 1 || j.group != KV_MAX_GROUPS;
}

// The job's access order moved to slot 0, so that every pointer is known
// without indexing (kept in registers).
__device__ __forceinline__ JobArgs job_args(const JobArgs& a_in, JobDev& j) {
  JobArgs a = a_in;
  if (j.order) {
    a.bid[0] = a_in.bid[1];
    a.key[0] = a_in.key[1];
    a.nxt[0] = a_in.nxt[1];
    a.w8[0] = a_in.w8[1];
    a.g8[0] = a_in.g8[1];
  }
  j.order = 0;
  return a;
}

// FIFO jobs (LFU jobs are left to k_replay_lfu).
__global__ __launch_bounds__(kRNT) void k_replay(const JobDev* __restrict__ jobs, JobArgs a_in,
                                                 uint64_t* __restrict__ state,
                                                 uint64_t* __restrict__ bits,
                                                 unsigned long long* __restrict__ jcnt) {
  __shared__ FifoLds lds;
  __shared__ GroupCounters gc;
  if (blockIdx.x < a_in.job_lo || blockIdx.x >= a_in.job_hi) return;
  JobDev j = jobs[blockIdx.x];
  if (j.closed || j.kind == kJobLfu) return;
  const JobArgs a = job_args(a_in, j);
  const uint32_t tid = threadIdx.x;
  if (tid < KV_MAX_GROUPS) gc.ins[tid] = gc.insw[tid] = gc.ev[tid] = gc.evw[tid] = 0;
  __syncthreads();
  // one group for every access of the job: counters add up per wavefront
  const bool g1 = a.n_groups == 1 || j.group != KV_MAX_GROUPS;
  const uint32_t g0 = j.group == KV_MAX_GROUPS ? 0u : j.group;
  unsigned long long* cnt = jcnt + (uint64_t)blockIdx.x * a.n_groups * 4;
  if (j.kind == kJobFifoChunk)
    fifo_chunked(j, a, reinterpret_cast<uint32_t*>(state + j.state_off), bits + j.bits_off, gc,
                 lds, g1, g0);
  else
    fifo_serial(j, a, reinterpret_cast<uint32_t*>(state + j.state_off), bits + j.bits_off, gc);
  __syncthreads();
  write_counters(gc, a.n_groups, cnt);
}

// LFU jobs, NT threads per job; G1: the jobs whose accesses all belong to
// one group (the others are left to the G1 = false instance).
template <int NT, bool G1>
__global__ __launch_bounds__(NT) void k_replay_lfu(const JobDev* __restrict__ jobs, JobArgs a_in,
                                                   uint64_t* __restrict__ state,
                                                   uint32_t* __restrict__ cls,
                                                   uint64_t* __restrict__ bits,
                                                   unsigned long long* __restrict__ jcnt) {
  __shared__ LfuLds lds;
  __shared__ GroupCounters gc;
  if (blockIdx.x < a_in.job_lo || blockIdx.x >= a_in.job_hi) return;
  JobDev j = jobs[blockIdx.x];
  if (j.closed || j.kind != kJobLfu) return;
  if (lfu_one_group(j, a_in.n_groups) != G1) return;
  const JobArgs a = job_args(a_in, j);
  const uint32_t tid = threadIdx.x;
  if (tid < KV_MAX_GROUPS) gc.ins[tid] = gc.insw[tid] = gc.ev[tid] = gc.evw[tid] = 0;
  __syncthreads();
  const uint32_t g0 = j.group == KV_MAX_GROUPS ? 0u : j.group;
  unsigned long long* cnt = jcnt + (uint64_t)blockIdx.x * a.n_groups * 4;
  lfu_chunked<NT, G1>(j, a, reinterpret_cast<uint32_t*>(state + j.state_off), cls,
                      bits + j.bits_off, gc, lds, g0);
  const bool ok = lds.ok != 0 && blockIdx.x != a.fail_job;
  __syncthreads();
  write_counters(gc, a.n_groups, cnt);
  // a failed state check is recorded for the host (the first failing job wins)
  if (tid == 0 && !ok && atomicCAS(&a.err[0], 0u, 1u) == 0u) atomicExch(&a.err[1], blockIdx.x);
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
  int16_t src[3];        // tiled combine: staged hit-bit source per tier, -1 = none
  uint16_t pad;
  uint64_t m_cnt, m_w;   // accesses (and weight) the record counts over
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


// Records combined tile by tile.  A block owns a range of words (64 accesses
// each) and every record of the launch (one per thread); each batch of kCbB
// words of every hit-bit source (job bitmaps, re-access bits), group mask
// and (mixed weights only) weight plane is staged once in LDS and read by
// all records, so the sources cross HBM once instead of once per record.
// The next batch is loaded while the current one is counted.  Two constant
// rows (all zeros, all ones) stand in for an absent tier and for the mask
// of a record that counts every group, so a batch inside a record's range
// is counted without a branch or a mask.
constexpr int kCbB = 32;          // words per batch
constexpr int kCbSrc = 128;       // hit-bit sources at most
constexpr int kCbNT = 1024;       // records per launch
constexpr int kCbZero = 0, kCbOnes = 1, kCbRow0 = 2;   // constant rows, first staged row
constexpr int kCbRows = kCbRow0 + kCbSrc + KV_MAX_GROUPS + 16;  // + sources, masks, 2 x 8 planes
constexpr int kCbLd = ((kCbRows - kCbRow0) * kCbB + kCbNT - 1) / kCbNT;  // staged words per thread

struct CbSrc {
  const uint64_t* p;   // word w at p[w - wlo]
  uint64_t wlo, whi;   // readable words [wlo, whi]
};

struct CombineTileArgs {
  const RecDev* recs;
  uint32_t n_recs, rec0;
  const CbSrc* src;
  uint32_t n_src;
  const uint64_t* planes[2];
  uint32_t plane_mask;   // weight bits present
  uint32_t uniform_w;    // 0 = mixed weights
  const uint64_t* gmask; // shared order
  uint32_t n_gm;         // group masks staged (0: no filtered record)
  uint64_t nwords, wpb;  // words in all, words per block
  unsigned long long* part;  // [n_recs][6]: hits of u0, u1, u2, then their weights
};

// Staged row `row` (counted from the first staged row): the sources, the
// group masks, then (mixed weights) the 2 x 8 weight planes.
__device__ __forceinline__ uint64_t cb_load(const CombineTileArgs& a, const CbSrc* src,
                                            uint32_t row, uint64_t w) {
  if (w >= a.nwords) return 0ull;
  if (row < a.n_src) {
    const CbSrc c = src[row];
    return (w >= c.wlo && w <= c.whi) ? c.p[w - c.wlo] : 0ull;
  }
  row -= a.n_src;
  if (row < a.n_gm) return a.gmask[(uint64_t)row * a.nwords + w];
  row -= a.n_gm;
  const uint32_t o = row >> 3, b = row & 7;
  if (!a.planes[o] || !((a.plane_mask >> b) & 1u)) return 0ull;
  return a.planes[o][(uint64_t)b * a.nwords + w];
}

// One word's three union counts (and, with weight planes, their weights)
// under mask m.  rows = the staged batch, s* = the rows of the record's
// tiers, p = its order's first weight plane, pm = the weight bits present.
template <bool kPlanes>
__device__ __forceinline__ void cb_count(const uint64_t (*rows)[kCbB + 1], int b, uint64_t m,
                                         uint32_t s0, uint32_t s1, uint32_t s2, uint32_t p,
                                         uint32_t pm, uint32_t* c, uint32_t* cw) {
  const uint64_t p0 = rows[s0][b], p1 = rows[s1][b], p2 = rows[s2][b];
  const uint64_t u0 = p0 & m, u1 = (p0 | p1) & m, u2 = (p0 | p1 | p2) & m;
  c[0] += __popcll(u0);
  c[1] += __popcll(u1);
  c[2] += __popcll(u2);
  if (kPlanes) {
#pragma unroll
    for (int pb = 0; pb < 8; ++pb) {
      if (!((pm >> pb) & 1u)) continue;
      const uint64_t pl = rows[p + pb][b];
      cw[0] += (uint32_t)__popcll(u0 & pl) << pb;
      cw[1] += (uint32_t)__popcll(u1 & pl) << pb;
      cw[2] += (uint32_t)__popcll(u2 & pl) << pb;
    }
  }
}

// A batch of the record's words: the interior ones (every access inside the
// record's range) without range checks, the others one by one.
template <bool kPlanes>
__device__ __forceinline__ void cb_batch(const uint64_t (*rows)[kCbB + 1], uint64_t wb,
                                         uint64_t w1, const RecDev& r, uint32_t rm, uint32_t s0,
                                         uint32_t s1, uint32_t s2, uint32_t p, uint32_t pm,
                                         uint32_t* c, uint32_t* cw) {
  const uint64_t rwlo = r.begin >> 6, rwhi = (r.end - 1) >> 6;
  const uint64_t fwlo = (r.begin + 63) >> 6, fwhi = r.end >> 6;
  if (wb >= fwlo && wb + kCbB <= fwhi && wb + kCbB <= w1) {
#pragma unroll(kPlanes ? 2 : 8)
    for (int b = 0; b < kCbB; ++b) cb_count<kPlanes>(rows, b, rows[rm][b], s0, s1, s2, p, pm, c, cw);
  } else {
    for (int b = 0; b < kCbB; ++b) {
      const uint64_t w = wb + b;
      if (w < rwlo || w > rwhi || w >= w1) continue;
      uint64_t m = rows[rm][b];
      if (w == rwlo) m &= ~0ull << (r.begin & 63);
      if (w == rwhi && (r.end & 63)) m &= (1ull << (r.end & 63)) - 1;
      cb_count<kPlanes>(rows, b, m, s0, s1, s2, p, pm, c, cw);
    }
  }
}

__global__ __launch_bounds__(kCbNT) void k_combine_tile(const CombineTileArgs a) {
  // rows padded by one word: records read different rows at the same word
  __shared__ uint64_t sw[2][kCbRows][kCbB + 1];
  __shared__ CbSrc ssrc[kCbSrc];
  const uint32_t tid = threadIdx.x;
  if (tid < a.n_src) ssrc[tid] = a.src[tid];
  if (tid < 2 * (kCbB + 1)) {
    const uint32_t bf = tid / (kCbB + 1), b = tid % (kCbB + 1);
    sw[bf][kCbZero][b] = 0ull;
    sw[bf][kCbOnes][b] = ~0ull;
  }
  __syncthreads();
  const bool weighted = a.uniform_w == 0;
  const uint32_t n_items = (a.n_src + a.n_gm + (weighted ? 16u : 0u)) * kCbB;
  const uint32_t ri = a.rec0 + tid;
  const bool have = ri < a.n_recs;
  RecDev r{};
  if (have) r = a.recs[ri];
  const bool live = have && r.end > r.begin;
  const uint64_t rwlo = r.begin >> 6, rwhi = live ? (r.end - 1) >> 6 : 0;
  const uint32_t s0 = r.src[0] >= 0 ? kCbRow0 + r.src[0] : kCbZero;
  const uint32_t s1 = r.src[1] >= 0 ? kCbRow0 + r.src[1] : kCbZero;
  const uint32_t s2 = r.src[2] >= 0 ? kCbRow0 + r.src[2] : kCbZero;
  const uint32_t rm = r.filter ? kCbRow0 + a.n_src + r.group : kCbOnes;
  const uint32_t rp = kCbRow0 + a.n_src + a.n_gm + 8 * r.order;
  const uint64_t w0 = (uint64_t)blockIdx.x * a.wpb;
  const uint64_t w1 = min<uint64_t>(a.nwords, w0 + a.wpb);
  unsigned long long acc[6] = {0, 0, 0, 0, 0, 0};
  uint64_t nxt[kCbLd];
  auto fetch = [&](uint64_t wb) {
#pragma unroll
    for (int q = 0; q < kCbLd; ++q) {
      const uint32_t item = tid + q * kCbNT;
      nxt[q] = item < n_items ? cb_load(a, ssrc, item / kCbB, wb + item % kCbB) : 0ull;
    }
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int q = 0; q < kCbLd; ++q) {
      const uint32_t item = tid + q * kCbNT;
      if (item < n_items) sw[buf][kCbRow0 + item / kCbB][item % kCbB] = nxt[q];
    }
  };
  if (w0 < w1) {
    fetch(w0);
    put(0);
  }
  __syncthreads();
  int cur = 0;
  for (uint64_t wb = w0; wb < w1; wb += kCbB) {
    if (wb + kCbB < w1) fetch(wb + kCbB);
    if (live && wb <= rwhi && wb + kCbB > rwlo) {
      uint32_t c[3] = {0, 0, 0}, cw[3] = {0, 0, 0};   // at most 64 x 255 x kCbB each
      if (weighted)
        cb_batch<true>(sw[cur], wb, w1, r, rm, s0, s1, s2, rp, a.plane_mask, c, cw);
      else
        cb_batch<false>(sw[cur], wb, w1, r, rm, s0, s1, s2, rp, 0u, c, cw);
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        acc[k] += c[k];
        acc[3 + k] += cw[k];
      }
    }
    if (wb + kCbB < w1) put(cur ^ 1);
    __syncthreads();
    cur ^= 1;
  }
  if (live) {
    if (!weighted)
      for (int k = 0; k < 3; ++k) acc[3 + k] = acc[k] * a.uniform_w;
    unsigned long long* o = a.part + (uint64_t)ri * 6;
#pragma unroll
    for (int f = 0; f < 6; ++f)
      if (acc[f]) atomicAdd(o + f, acc[f]);
  }
}

// Per record: its three tiers' count fields from the summed union counts.
__global__ __launch_bounds__(256) void k_combine_fin(const RecDev* __restrict__ recs,
                                                     uint32_t n_recs,
                                                     const unsigned long long* __restrict__ part,
                                                     const unsigned long long* __restrict__ jcnt,
                                                     uint32_t n_groups, uint64_t* __restrict__ counts) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_recs) return;
  const RecDev r = recs[i];
  const unsigned long long* pc = part + (uint64_t)i * 6;
  const unsigned long long tot[8] = {r.m_cnt, pc[0], pc[1], pc[2], r.m_w, pc[3], pc[4], pc[5]};
  uint64_t* out = counts + ((uint64_t)r.cfg * n_groups + r.group) * 24;
  for (int k = 0; k < 3; ++k) {
    uint64_t* rec = out + k * 8;
    if (r.job[k] < 0) {
      for (int f = 0; f < 8; ++f) rec[f] = 0;
      continue;
    }
    const unsigned long long* jc = jcnt + ((uint64_t)r.job[k] * n_groups + r.group) * 4;
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

}  // namespace

// Two more streams per device (default priority) with a fork event and a
// join event each, created on first use and kept until the process ends.
constexpr int kAux = 3;  // LFU one-group jobs, other LFU jobs, FIFO jobs
struct AuxStream {
  hipStream_t s[kAux] = {};
  hipEvent_t fork = nullptr, join[kAux] = {};
  std::mutex mu;
};

static kv_status aux_stream(AuxStream** out) {
  static std::mutex mu;
  static AuxStream aux[64];
  int dev = 0;
  KV_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(KV_ERR_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> g(mu);
  AuxStream& a = aux[dev];
  if (!a.s[0]) {
    for (int i = 0; i < kAux; ++i) {
      KV_HIP(hipStreamCreateWithFlags(&a.s[i], hipStreamNonBlocking));
      KV_HIP(hipEventCreateWithFlags(&a.join[i], hipEventDisableTiming));
    }
    KV_HIP(hipEventCreateWithFlags(&a.fork, hipEventDisableTiming));
  }
  *out = &a;
  return KV_OK;
}

// Test hooks, read at every call: KVCFG_TEST_REPLAY_BUDGET caps the replay
// state of one wave (bytes), so that a small batch needs several waves;
// KVCFG_TEST_FAIL_JOB makes that replay job report a failed state check
// (its kernel still runs to completion), so that the error path is seen.
static uint64_t replay_test_budget() {
  const char* e = std::getenv("KVCFG_TEST_REPLAY_BUDGET");
  return e ? std::strtoull(e, nullptr, 10) : 0ull;
}

static uint32_t replay_test_fail_job() {
  const char* e = std::getenv("KVCFG_TEST_FAIL_JOB");
  return e ? (uint32_t)std::strtoul(e, nullptr, 10) : kNone;
}

kv_status replay_run(Trace& t, const std::vector<ReplayJob>& jobs, const kv_config* cfg_host,
                     const kv_config* cfg_dev, uint32_t n_cfg, uint64_t* counts,
                     hipStream_t s, const std::function<kv_status()>& meanwhile) {
  (void)cfg_dev;
  kv_status st;
  const uint32_t G = t.n_groups;
  const uint64_t n = t.n;
  const uint64_t nwords = (n + 63) / 64;
  const uint32_t n_class = kLdsClass;
  const uint32_t class_words = n_class;  // u32 words per LFU job: class heads
  // layout of job state, class arrays and bitmaps
  std::vector<JobDev> jd(jobs.size());
  std::vector<uint64_t> jw(jobs.size(), 0);  // replay-state words of each job
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
      j.chunk = kLChunk;
    }
    if (!r.closed && r.end > r.begin) {
      // FIFO: one u32 per block; LFU: one count per position and a spare slot
      jw[i] = (r.policy == KV_POLICY_FIFO) ? (t.u + 1) / 2 : (r.end - r.begin + 2) / 2;
      state_words += jw[i];
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
  // Waves: the replay state of every job at once, or, when that does not fit
  // the device (or the test budget), consecutive groups of jobs that share
  // one state buffer and run one group after another.
  std::vector<uint32_t> wave_lo;  // first job of each wave
  uint64_t wave_words = 0;        // state words of the largest wave
  auto plan_waves = [&](uint64_t budget_words) {
    wave_lo.assign(1, 0);
    wave_words = 0;
    uint64_t cur = 0;
    for (size_t i = 0; i < jd.size(); ++i) {
      if (cur && cur + jw[i] > budget_words) {
        wave_lo.push_back((uint32_t)i);
        cur = 0;
      }
      jd[i].state_off = cur;
      cur += jw[i];
      wave_words = std::max(wave_words, cur);
    }
  };
  uint64_t max_job = 0;
  for (uint64_t x : jw) max_job = std::max(max_job, x);
  uint64_t budget = std::max<uint64_t>(state_words, 1);
  if (const uint64_t tb = replay_test_budget()) budget = std::max<uint64_t>(tb / 8, 1);
  DevBuf& bstate = t.ws[12];
  for (;;) {
    plan_waves(std::max(budget, max_job));
    if ((st = bstate.reserve(std::max<uint64_t>(wave_words, 1) * 8)) == KV_OK) break;
    if (st != KV_ERR_NOMEM || budget <= max_job) return st;
    budget = budget / 2;  // retry with smaller waves
  }
  const uint32_t n_waves = (uint32_t)wave_lo.size();
  wave_lo.push_back((uint32_t)jd.size());
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
      if (pol == KV_POLICY_LRU || pol == KV_POLICY_LEAF) continue;
      if (C.mode == KV_MODE_EXCLUSIVE_DEMOTE) continue;  // replayed access by access
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
        // what the record counts over: its group's accesses, or all of them
        const bool whole = !part_order && G == 1;
        r.m_cnt = whole ? n : t.st.n_g[gg];
        r.m_w = whole ? t.st.n_w : t.st.n_w_g[gg];
        recs.push_back(r);
      }
    }
  }
  // FIFO records first: they are combined on the FIFO jobs' stream as soon
  // as those are done, the others once every job is
  auto rec_fifo = [&](const RecDev& r) {
    for (int k = 0; k < 3; ++k)
      if (r.job[k] >= 0) return jd[r.job[k]].policy == KV_POLICY_FIFO;
    return true;
  };
  std::stable_partition(recs.begin(), recs.end(), rec_fifo);
  uint32_t nf = 0;
  while (nf < recs.size() && rec_fifo(recs[nf])) ++nf;
  // hit-bit sources of the tiled combine, per record class (FIFO / other):
  // one per replayed job, one per order for jobs whose cache holds
  // everything (a hit is a re-access)
  std::vector<int32_t> src_of[2] = {std::vector<int32_t>(jd.size() + 2, -1),
                                    std::vector<int32_t>(jd.size() + 2, -1)};
  uint32_t n_src[2] = {0, 0};
  for (size_t i = 0; i < recs.size(); ++i) {
    RecDev& r = recs[i];
    const int cls = i < nf ? 0 : 1;
    for (int k = 0; k < 3; ++k) {
      r.src[k] = -1;
      if (r.job[k] < 0) continue;
      const size_t key = jd[r.job[k]].closed ? jd.size() + r.order : (size_t)r.job[k];
      if (src_of[cls][key] < 0) src_of[cls][key] = (int32_t)n_src[cls]++;
      r.src[k] = (int16_t)std::min<int32_t>(src_of[cls][key], 0x7FFF);
    }
  }
  const bool tiled = n_src[0] <= (uint32_t)kCbSrc && n_src[1] <= (uint32_t)kCbSrc;
  DevBuf& bj = t.ws[11];
  DevBuf& bcls = t.ws[13];
  DevBuf& bbits = t.ws[14];
  DevBuf& bjc = t.ws[15];
  DevBuf& brec = t.ws[16];
  DevBuf& bord = t.ws[17];
  if ((st = bj.reserve(jd.size() * sizeof(JobDev))) != KV_OK) return st;
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
  ja.n = t.n;
  ja.n_groups = G;
  ja.n_class = n_class;
  ja.err = t.err.as<uint32_t>();
  ja.fail_job = replay_test_fail_job();
  const uint32_t nj = (uint32_t)jd.size();
  auto wave_args = [&](uint32_t w) {
    JobArgs x = ja;
    x.job_lo = wave_lo[w];
    x.job_hi = wave_lo[w + 1];
    return x;
  };
  if (nj) {
    hipLaunchKernelGGL(k_replay_init, dim3(64, nj), dim3(256), 0, s, bj.as<JobDev>(),
                       bstate.as<uint64_t>(), bcls.as<uint32_t>(), wave_args(0));
    KV_HIP(hipGetLastError());
  }
  tm.reset();
  // the combine's inputs, staged before the streams fork (the FIFO records
  // are combined on the FIFO stream)
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
  const uint32_t nrec = (uint32_t)recs.size();
  CombineTileArgs ta{};
  DevBuf& bsrc = t.ws[18];
  DevBuf& bpart = t.ws[19];
  if (tiled && nrec) {
    std::vector<CbSrc> srcs(n_src[0] + n_src[1]);
    for (int cls = 0; cls < 2; ++cls) {
      for (size_t key = 0; key < src_of[cls].size(); ++key) {
        const int32_t sl = src_of[cls][key];
        if (sl < 0) continue;
        CbSrc c{};
        if (key >= jd.size()) {
          c.p = ca.reuse[key - jd.size()];
          c.wlo = 0;
          c.whi = nwords - 1;
        } else {
          const JobDev& q = jd[key];
          c.p = bbits.as<uint64_t>() + q.bits_off;
          c.wlo = q.word0;
          c.whi = (q.end - 1) >> 6;
        }
        srcs[(cls ? n_src[0] : 0) + sl] = c;
      }
    }
    if ((st = bsrc.reserve(std::max<size_t>(srcs.size(), 1) * sizeof(CbSrc))) != KV_OK) return st;
    if ((st = bpart.reserve((size_t)nrec * 6 * 8)) != KV_OK) return st;
    t.src_stage.resize(srcs.size() * sizeof(CbSrc));
    std::memcpy(t.src_stage.data(), srcs.data(), t.src_stage.size());
    if (!srcs.empty())
      KV_HIP(hipMemcpyAsync(bsrc.p, t.src_stage.data(), t.src_stage.size(),
                            hipMemcpyHostToDevice, s));
    if ((st = fill_u64(bpart.as<uint64_t>(), 0, (uint64_t)nrec * 6, s)) != KV_OK) return st;
    bool any_filter = false;
    for (const RecDev& r : recs) any_filter |= r.filter != 0;
    ta.recs = brec.as<RecDev>();
    ta.planes[0] = planes[0];
    ta.planes[1] = have_part ? planes[1] : nullptr;
    ta.plane_mask = pm;
    ta.uniform_w = ca.uniform_w;
    ta.gmask = gmask[0];
    ta.n_gm = any_filter ? G : 0u;
    ta.nwords = nwords;
    ta.part = bpart.as<unsigned long long>();
    int ncu = 0;
    KV_HIP(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, t.device));
    const uint64_t nb0 = std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)std::max(ncu, 1),
                                                                  div_up(nwords, kCbB)));
    ta.wpb = (uint64_t)div_up(div_up(nwords, nb0), kCbB) * kCbB;
  }
  // records [r0, r1) of one class, tile by tile
  auto combine_range = [&](uint32_t r0, uint32_t r1, hipStream_t sk) -> kv_status {
    if (r0 >= r1) return KV_OK;
    CombineTileArgs x = ta;
    const int cls = r0 < nf ? 0 : 1;
    x.src = bsrc.as<CbSrc>() + (cls ? n_src[0] : 0);
    x.n_src = n_src[cls];
    x.n_recs = r1;
    const uint32_t nb = div_up(nwords, x.wpb);
    for (uint32_t q = r0; q < r1; q += kCbNT) {
      x.rec0 = q;
      hipLaunchKernelGGL(k_combine_tile, dim3(nb), dim3(kCbNT), 0, sk, x);
      KV_HIP(hipGetLastError());
    }
    return KV_OK;
  };
  // LFU jobs of one group, other LFU jobs, FIFO jobs and the caller's other
  // work (the LRU stack pass) run concurrently: the replay kernels on
  // streams forked from the caller's and joined back into it before the
  // records are combined
  bool any[kAux] = {false, false, false};
  for (const JobDev& q : jd) {
    if (q.closed) continue;
    if (q.kind != kJobLfu) any[2] = true;
    else if (lfu_one_group(q, G)) any[0] = true;
    else any[1] = true;
  }
  // one replay kernel (k: LFU one-group, other LFU, FIFO) over the jobs of x
  auto launch = [&](int k, hipStream_t sk, const JobArgs& x) -> kv_status {
    tm.emplace(k == 2 ? kStReplayFifo : kStReplay, sk);
    if (k == 0)
      hipLaunchKernelGGL((k_replay_lfu<kLfuNT, true>), dim3(nj), dim3(kLfuNT), 0, sk,
                         bj.as<JobDev>(), x, bstate.as<uint64_t>(), bcls.as<uint32_t>(),
                         bbits.as<uint64_t>(), bjc.as<unsigned long long>());
    else if (k == 1)
      hipLaunchKernelGGL((k_replay_lfu<kLfuNT, false>), dim3(nj), dim3(kLfuNT), 0, sk,
                         bj.as<JobDev>(), x, bstate.as<uint64_t>(), bcls.as<uint32_t>(),
                         bbits.as<uint64_t>(), bjc.as<unsigned long long>());
    else
      hipLaunchKernelGGL(k_replay, dim3(nj), dim3(kRNT), 0, sk, bj.as<JobDev>(), x,
                         bstate.as<uint64_t>(), bbits.as<uint64_t>(),
                         bjc.as<unsigned long long>());
    KV_HIP(hipGetLastError());
    tm.reset();
    return KV_OK;
  };
  bool fifo_combined = false;
  if (n_waves == 1) {
    // LFU jobs of one group, other LFU jobs, FIFO jobs and the caller's other
    // work (the LRU stack pass) run concurrently: the replay kernels on
    // streams forked from the caller's and joined back into it before the
    // records are combined
    AuxStream* aux = nullptr;
    std::unique_lock<std::mutex> lk;
    if (any[0] || any[1] || any[2]) {
      if ((st = aux_stream(&aux)) != KV_OK) return st;
      lk = std::unique_lock<std::mutex>(aux->mu);
      KV_HIP(hipEventRecord(aux->fork, s));
    }
    for (int k = 0; k < kAux; ++k) {
      if (!any[k]) continue;
      hipStream_t sk = aux->s[k];
      KV_HIP(hipStreamWaitEvent(sk, aux->fork, 0));
      if ((st = launch(k, sk, wave_args(0))) != KV_OK) return st;
      if (k == 2 && tiled && nf) {
        tm.emplace(kStCombine, sk);
        if ((st = combine_range(0, nf, sk)) != KV_OK) return st;
        tm.reset();
        fifo_combined = true;
      }
      KV_HIP(hipEventRecord(aux->join[k], sk));
    }
    const kv_status st_mid = meanwhile();
    for (int k = 0; k < kAux; ++k)
      if (any[k]) KV_HIP(hipStreamWaitEvent(s, aux->join[k], 0));
    lk = std::unique_lock<std::mutex>();
    if (st_mid != KV_OK) return st_mid;
  } else {
    // waves share the state buffer: the caller's other work, then every
    // wave's kernels, one after another on the caller's stream
    if ((st = meanwhile()) != KV_OK) return st;
    for (uint32_t w = 0; w < n_waves; ++w) {
      const JobArgs x = wave_args(w);
      if (w > 0) {
        hipLaunchKernelGGL(k_replay_init, dim3(64, nj), dim3(256), 0, s, bj.as<JobDev>(),
                           bstate.as<uint64_t>(), bcls.as<uint32_t>(), x);
        KV_HIP(hipGetLastError());
      }
      for (int k = 0; k < kAux; ++k)
        if (any[k] && (st = launch(k, s, x)) != KV_OK) return st;
    }
  }
  tm.reset();
  if (!recs.empty()) {
    tm.emplace(kStCombine, s);
    if (tiled) {
      if (!fifo_combined && (st = combine_range(0, nf, s)) != KV_OK) return st;
      if ((st = combine_range(nf, nrec, s)) != KV_OK) return st;
      hipLaunchKernelGGL(k_combine_fin, dim3(div_up(nrec, 256)), dim3(256), 0, s,
                         brec.as<RecDev>(), nrec, bpart.as<unsigned long long>(),
                         bjc.as<unsigned long long>(), G, counts);
      KV_HIP(hipGetLastError());
    } else {
      hipLaunchKernelGGL(k_combine, dim3(nrec), dim3(256), 0, s, brec.as<RecDev>(), ca, counts);
      KV_HIP(hipGetLastError());
    }
  }
  tm.reset();
  if (any[0] || any[1]) {
    // the LFU jobs' error record, read by the next call on this trace
    t.err_jobs.resize(jd.size());
    for (size_t i = 0; i < jd.size(); ++i)
      t.err_jobs[i] = ReplayJobInfo{jd[i].policy, jd[i].group, jd[i].cap};
    KV_HIP(hipMemcpyAsync(t.err_host, t.err.p, 2 * sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    KV_HIP(hipEventRecord(t.err_ev, s));
    t.err_pending = true;
  }
  return KV_OK;
}

}  // namespace kv
