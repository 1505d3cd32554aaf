// k_stack.hip - one pass that serves every LRU capacity at once.
//
// Under LRU a block is resident in a cache of capacity C exactly when its
// stack distance D_i <= C, where D_i is the weight of the block itself plus
// the weight of the distinct other blocks touched since its previous access
// (Mattson et al., "Evaluation techniques for storage hierarchies", IBM
// Systems Journal 1970; with unit weights D_i counts distinct blocks).  The
// paper's tiers use LRU (Section 2.1) and its simulator models the tier
// hierarchy by replay (Section 3.2); the inclusion property lets one pass
// over the trace answer every tier capacity of every configuration.
//
// With p = prev(i) and key_j = prev(j) + 1 (0 for a first access):
//   D_i = w_i + sum_{p < j < i} w_j [key_j <= p]
// (a block touched in (p, i) is counted at its first touch there, the one
// whose own previous access lies before p).  Positions are cut into 8192-wide
// blocks; with P = block(p), I = block(i):
//   P == I:  D_i = w_i + A(i) - Wloc(p)
//   P <  I:  D_i = w_i + A(i) + E(p) + RQ[I-1][P]
// where, inside one block,
//   A(i)    = sum_{j in block(i), j < i} w_j [key_j < key_i]     (dominance count)
//   Wloc(p) = sum_{j in block(p), j <= p} w_j
//   E(p)    = Cnt_P(p) - Wloc(p) + C(p)
//   Cnt_P(p)= sum_{j in block P} w_j [key_j <= p]
//   C(p)    = sum_{q in block P, q < p} w_q [P < block(next(q)) < block(next(p))]
// and across blocks RQ[X][Y] = sum_{X'=Y+1..X} Q[X'][Y] with
//   Q[X][Y] = sum_{j in block X} w_j [key_j <= Y * 8192]
// stored as a lower triangle.  The two in-block dominance counts come from
// an LDS merge sort that accumulates, for every element of a right-hand run,
// the weight of smaller keys in the left-hand run.
//
// Outputs per (group, bin): the count / weight of accesses whose D falls in
// the bin (bins cut at the batch's capacity values), and the count / weight
// of blocks whose final stack depth (the weight of distinct blocks accessed
// at or after their last access) falls in the bin; cumulative over bins on
// return, so hits(C) is one lookup.
#include <algorithm>
#include <cstdlib>

#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr int kLocNT = 1024;
constexpr int kLocItems = 8;
static_assert(kLocNT * kLocItems == (int)kSdB, "block tile mismatch");
constexpr uint32_t kSentinel = 0xFFFFFFFFu;
constexpr uint32_t kRowChunk = 16384;   // LDS histogram bins per row chunk
constexpr int kRowNT = 1024;            // threads per row of the block matrix
constexpr int kAsmNT = 1024;            // threads per workgroup of the distance binning kernels
constexpr uint32_t kColRows = 64;       // rows per column-scan chunk
constexpr uint32_t kThrLds = 6144;      // thresholds kept in LDS for binning

__host__ __device__ __forceinline__ uint64_t tri_off(uint64_t x) { return x * (x - 1) / 2; }

// ---------------------------------------------------------------------------
// Q rows: Q[X][Y] for Y < X, inclusive prefix over ceil(key / 8192).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kRowNT) void k_sd_rowhist(const uint32_t* __restrict__ key,
                                                    const uint8_t* __restrict__ w8, uint64_t n,
                                                    uint32_t row_chunk, uint32_t* __restrict__ Q) {
  // bin j lives at hp(j), one padding word after every 64: the scan below
  // gives each thread a run of up to kRowChunk / kRowNT bins, which would
  // otherwise put the lanes of a wavefront on a few banks
  __shared__ uint32_t h[kRowChunk + kRowChunk / 64];
  __shared__ uint32_t sh[kRowNT / 64 + 1];
  const auto hp = [](uint32_t j) { return j + (j >> 6); };
  const uint32_t X = blockIdx.x;
  if (X == 0) return;
  const uint64_t base = (uint64_t)X * kSdB;
  const uint32_t nb = (uint32_t)min<uint64_t>(kSdB, n - base);
  const uint64_t row = tri_off(X);
  for (uint32_t c0 = 0; c0 < X; c0 += row_chunk) {
    const uint32_t width = min(row_chunk, X - c0);
    for (uint32_t j = threadIdx.x; j < width; j += kRowNT) h[hp(j)] = 0;
    __syncthreads();
    uint32_t carry = 0;
    for (uint32_t j = threadIdx.x; j < nb; j += kRowNT) {
      const uint32_t c = (key[base + j] + (kSdB - 1)) >> kSdLogB;
      const uint32_t w = w8[base + j];
      if (c < c0) carry += w;
      else if (c < c0 + width) atomicAdd(&h[hp(c - c0)], w);
    }
    carry = block_sum<kRowNT>(carry, sh);
    // inclusive scan of h[0, width) in LDS, each thread a contiguous run
    const uint32_t per = (width + kRowNT - 1) / kRowNT;
    const uint32_t a = min(width, threadIdx.x * per), b = min(width, a + per);
    uint32_t run = 0;
    for (uint32_t j = a; j < b; ++j) run += h[hp(j)];
    uint32_t tot;
    uint32_t pre = block_excl_scan<kRowNT>(run, sh, &tot) + carry;
    for (uint32_t j = a; j < b; ++j) {
      pre += h[hp(j)];
      h[hp(j)] = pre;
    }
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < width; j += kRowNT) Q[row + c0 + j] = h[hp(j)];
    __syncthreads();
  }
}

// Column sums of Q over chunks of kColRows rows (only rows X > Y count).
__global__ __launch_bounds__(256) void k_sd_colsum(const uint32_t* __restrict__ Q, uint32_t G,
                                                   uint32_t* __restrict__ csum) {
  const uint32_t Y = blockIdx.x * 256 + threadIdx.x;
  const uint32_t c = blockIdx.y;
  if (Y >= G) return;
  const uint32_t x0 = max(Y + 1, c * kColRows), x1 = min(G, (c + 1) * kColRows);
  uint32_t s = 0;
  for (uint32_t X = x0; X < x1; ++X) s += Q[tri_off(X) + Y];
  csum[(uint64_t)c * G + Y] = s;
}

__global__ __launch_bounds__(256) void k_sd_colchunks(uint32_t* __restrict__ csum, uint32_t G,
                                                      uint32_t nchunks) {
  const uint32_t Y = blockIdx.x * 256 + threadIdx.x;
  if (Y >= G) return;
  uint32_t run = 0;
  for (uint32_t c = 0; c < nchunks; ++c) {
    const uint32_t v = csum[(uint64_t)c * G + Y];
    csum[(uint64_t)c * G + Y] = run;
    run += v;
  }
}

__global__ __launch_bounds__(256) void k_sd_colapply(uint32_t* __restrict__ Q, uint32_t G,
                                                     const uint32_t* __restrict__ csum) {
  const uint32_t Y = blockIdx.x * 256 + threadIdx.x;
  const uint32_t c = blockIdx.y;
  if (Y >= G) return;
  const uint32_t x0 = max(Y + 1, c * kColRows), x1 = min(G, (c + 1) * kColRows);
  uint32_t run = csum[(uint64_t)c * G + Y];
  for (uint32_t X = x0; X < x1; ++X) {
    run += Q[tri_off(X) + Y];
    Q[tri_off(X) + Y] = run;
  }
}

// ---------------------------------------------------------------------------
// In-block dominance by LDS merge sort.
// ---------------------------------------------------------------------------
// Element i of a block-wide LDS array lives at pd(i): one padding word after
// every 16, so that the 16-element runs of the threads of a wavefront (and
// the merge positions inside them, about 8 apart) fall into different banks.
constexpr uint32_t kSdPad = kSdB + kSdB / 16;
__device__ __forceinline__ uint32_t pd(uint32_t i) { return i + (i >> 4); }

struct SortLds {
  uint32_t v[kSdPad];     // sorted keys of the current runs
  uint32_t pw[kSdPad];    // inclusive prefix weight inside each run
  uint32_t acc[kSdPad];   // accumulated weight of smaller keys at earlier positions
  uint16_t idx[kSdPad];   // local position of the element
};

// First index in S.v[lo, hi) (padded, sorted) with a value > x.
__device__ __forceinline__ uint32_t upper_bound_pd(const uint32_t* a, uint32_t lo, uint32_t hi,
                                                   uint32_t x) {
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (a[pd(mid)] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

template <int N>
__device__ __forceinline__ void cswap(uint32_t (&v)[N], uint32_t (&w)[N], uint32_t (&a)[N],
                                      uint32_t (&x)[N], int i, int l, bool up) {
  const bool sw = (v[i] > v[l]) == up;
  if (sw) {
    uint32_t t;
    t = v[i]; v[i] = v[l]; v[l] = t;
    t = w[i]; w[i] = w[l]; w[l] = t;
    t = a[i]; a[i] = a[l]; a[l] = t;
    t = x[i]; x[i] = x[l]; x[l] = t;
  }
}

// LDS exchange among the lanes of one wavefront: its LDS operations execute
// in issue order, so a compiler fence at wavefront scope suffices.
__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// On return S holds the block's elements sorted by v, each with
// acc = sum over earlier positions j of w_j [v_j < v] (exact whenever v is
// unique in the block, i.e. for every element whose acc is used).
__device__ void block_sort_dominance(SortLds& S, const uint32_t (&vin)[kLocItems],
                                     const uint32_t (&win)[kLocItems]) {
  const uint32_t t = threadIdx.x;
  uint32_t v[kLocItems], w[kLocItems], a[kLocItems], x[kLocItems];
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    v[e] = vin[e];
    w[e] = win[e];
    x[e] = t * kLocItems + e;
    uint32_t s = 0;
#pragma unroll
    for (int f = 0; f < e; ++f) s += (vin[f] < vin[e]) ? win[f] : 0u;
    a[e] = s;
  }
  // bitonic network on the thread's register-resident elements
#pragma unroll
  for (int k = 2; k <= kLocItems; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
#pragma unroll
      for (int i = 0; i < kLocItems; ++i) {
        const int l = i ^ j;
        if (l > i) cswap<kLocItems>(v, w, a, x, i, l, (i & k) == 0);
      }
    }
  }
  uint32_t run = 0;
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    run += w[e];
    const uint32_t s = pd(t * kLocItems + e);
    S.v[s] = v[e];
    S.pw[s] = run;
    S.acc[s] = a[e];
    S.idx[s] = (uint16_t)x[e];
  }
  uint32_t pw[kLocItems];
  for (uint32_t s = kLocItems; s < kSdB; s <<= 1) {
    // a pair of runs of s spans 2s / kLocItems threads: up to 64, one wavefront
    const bool in_wave = 2 * s <= 64u * kLocItems;
    if (in_wave) wave_sync_lds(); else __syncthreads();
    const uint32_t o0 = t * kLocItems;
    const uint32_t pair = o0 & ~(2 * s - 1);
    const uint32_t d0 = o0 - pair;
    const uint32_t Lb = pair, Rb = pair + s;
    uint32_t lo = d0 > s ? d0 - s : 0u, hi = min(d0, s);
    while (lo < hi) {
      const uint32_t mid = (lo + hi) >> 1;
      if (S.v[pd(Lb + mid)] <= S.v[pd(Rb + d0 - mid - 1)]) lo = mid + 1; else hi = mid;
    }
    uint32_t ia = lo, ib = d0 - lo;
#pragma unroll
    for (int e = 0; e < kLocItems; ++e) {
      const uint32_t li = pd(Lb + ia), ri = pd(Rb + ib);
      const bool takeL = (ib >= s) || (ia < s && S.v[li] <= S.v[ri]);
      if (takeL) {
        v[e] = S.v[li];
        a[e] = S.acc[li];
        x[e] = S.idx[li];
        pw[e] = S.pw[li] + (ib ? S.pw[pd(Rb + ib - 1)] : 0u);
        ++ia;
      } else {
        const uint32_t pl = ia ? S.pw[pd(Lb + ia - 1)] : 0u;
        v[e] = S.v[ri];
        a[e] = S.acc[ri] + pl;
        x[e] = S.idx[ri];
        pw[e] = pl + S.pw[ri];
        ++ib;
      }
    }
    if (in_wave) wave_sync_lds(); else __syncthreads();
#pragma unroll
    for (int e = 0; e < kLocItems; ++e) {
      const uint32_t o = pd(o0 + e);
      S.v[o] = v[e];
      S.acc[o] = a[e];
      S.idx[o] = (uint16_t)x[e];
      S.pw[o] = pw[e];
    }
  }
  __syncthreads();
}

// Per position block: A(i) and same-block distances -> partial[i]; E(p) for
// positions whose next access lies in a later block.
__global__ __launch_bounds__(kLocNT, 1) void k_sd_local(const uint32_t* __restrict__ key,
                                                        const uint32_t* __restrict__ nxt,
                                                        const uint8_t* __restrict__ w8,
                                                        uint64_t n, uint32_t G,
                                                        uint32_t* __restrict__ partial,
                                                        uint32_t* __restrict__ E) {
  __shared__ SortLds S;
  __shared__ uint32_t P[kSdPad];   // padded like S
  __shared__ uint32_t sh[kLocNT / 64 + 1];
  const uint32_t X = blockIdx.x;
  const uint64_t base = (uint64_t)X * kSdB;
  const uint32_t nb = (uint32_t)min<uint64_t>(kSdB, n - base);
  const uint32_t t = threadIdx.x;
  for (uint32_t j = t; j < kSdB; j += kLocNT) {
    const bool in = j < nb;
    S.v[pd(j)] = in ? key[base + j] : kSentinel;
    S.acc[pd(j)] = in ? nxt[base + j] : kNone;
    S.pw[pd(j)] = in ? (uint32_t)w8[base + j] : 0u;
  }
  __syncthreads();
  uint32_t k[kLocItems], nx[kLocItems], w[kLocItems];
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t j = pd(t * kLocItems + e);
    k[e] = S.v[j];
    nx[e] = S.acc[j];
    w[e] = S.pw[j];
  }
  __syncthreads();
  // Wloc (inclusive, position order) -> P;  same-block-next prefix -> sn
  uint32_t loc[kLocItems], sn[kLocItems];
  uint32_t run = 0, run2 = 0;
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    run += w[e];
    loc[e] = run;
    sn[e] = run2;
    const bool same = nx[e] != kNone && (nx[e] >> kSdLogB) == X;
    run2 += same ? w[e] : 0u;
  }
  uint32_t tot;
  const uint32_t pre = block_excl_scan<kLocNT>(run, sh, &tot);
  const uint32_t pre2 = block_excl_scan<kLocNT>(run2, sh, &tot);
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    P[pd(t * kLocItems + e)] = loc[e] + pre;
    sn[e] += pre2;
  }
  // ---- sort 1: keys -> A(i)
  block_sort_dominance(S, k, w);
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t s = t * kLocItems + e, sp = pd(s);
    const uint32_t i = S.idx[sp];
    const uint32_t kk = S.v[sp];
    if (i < nb && kk != 0u) {
      const uint32_t wi = S.pw[sp] - (s ? S.pw[pd(s - 1)] : 0u);
      const uint32_t p = kk - 1u;
      uint32_t d = wi + S.acc[sp];
      if ((uint64_t)p >= base) d -= P[pd((uint32_t)(p - base))];
      partial[base + i] = d;
    }
  }
  // Cnt_X(p) - Wloc(p) for positions whose next access is in a later block
  uint32_t ev[kLocItems];
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t lp = t * kLocItems + e;
    ev[e] = 0;
    if (lp < nb && nx[e] != kNone && (nx[e] >> kSdLogB) > X) {
      const uint32_t p = (uint32_t)(base + lp);
      const uint32_t ub = upper_bound_pd(S.v, 0u, kSdB, p);
      ev[e] = (ub ? S.pw[pd(ub - 1)] : 0u) - P[pd(lp)];
    }
  }
  __syncthreads();
  // ---- sort 2: (block of next access, reversed position) -> C(p)
  uint32_t v2[kLocItems];
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t lp = t * kLocItems + e;
    const uint32_t nbk = (nx[e] == kNone) ? G : (nx[e] >> kSdLogB);
    v2[e] = (lp < nb) ? ((nbk << kSdLogB) | (kSdB - 1u - lp)) : kSentinel;
  }
  block_sort_dominance(S, v2, w);
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t s = pd(t * kLocItems + e);
    const uint32_t i = S.idx[s];
    if (i < nb) P[pd(i)] = S.acc[s];
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < kLocItems; ++e) {
    const uint32_t lp = t * kLocItems + e;
    if (lp < nb && nx[e] != kNone && (nx[e] >> kSdLogB) > X)
      E[base + lp] = ev[e] + (P[pd(lp)] - sn[e]);
  }
}

// ---------------------------------------------------------------------------
// Assembly of cross-block distances and binning.
// ---------------------------------------------------------------------------
struct BinArgs {
  const uint32_t* thr;   // thresholds of all groups, concatenated
  const uint32_t* off;   // [n_groups + 1]
  uint32_t n_thr, n_groups;
  uint64_t* hist;        // u64[bins][4]
};

template <bool kLds>
__global__ __launch_bounds__(kAsmNT) void k_sd_assemble(const uint32_t* __restrict__ key,
                                                     const uint8_t* __restrict__ w8,
                                                     const uint8_t* __restrict__ g8, uint64_t n,
                                                     uint32_t G,
                                                     const uint32_t* __restrict__ partial,
                                                     const uint32_t* __restrict__ E,
                                                     const uint32_t* __restrict__ RQ,
                                                     BinArgs ba, uint32_t* __restrict__ dout,
                                                     const uint8_t* __restrict__ real) {
  __shared__ uint32_t sthr[kLds ? kThrLds : 1];
  __shared__ uint32_t scnt[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t sw[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t soff[KV_MAX_GROUPS + 1];
  const uint32_t nbins = ba.n_thr + ba.n_groups;
  if (threadIdx.x <= ba.n_groups) soff[threadIdx.x] = ba.off[threadIdx.x];
  if (kLds) {
    for (uint32_t j = threadIdx.x; j < ba.n_thr; j += kAsmNT) sthr[j] = ba.thr[j];
    for (uint32_t j = threadIdx.x; j < nbins; j += kAsmNT) {
      scnt[j] = 0;
      sw[j] = 0;
    }
  }
  __syncthreads();
  for (uint32_t X = blockIdx.x; X < G; X += gridDim.x) {
    const uint64_t base = (uint64_t)X * kSdB;
    const uint32_t nb = (uint32_t)min<uint64_t>(kSdB, n - base);
    const uint64_t row = X >= 2 ? tri_off(X - 1) : 0;
    for (uint32_t j = threadIdx.x; j < nb; j += kAsmNT) {
      const uint64_t i = base + j;
      if (real && !real[i]) continue;  // a re-touch of the radix-tree order: not binned
      const uint32_t kk = key[i];
      if (kk == 0) {
        if (dout) dout[i] = kNone;  // a first access: no finite distance
        continue;
      }
      const uint32_t p = kk - 1u;
      const uint32_t Pb = p >> kSdLogB;
      uint32_t d = partial[i];
      if (Pb < X) {
        d += E[p];
        if (Pb + 1 < X) d += RQ[row + Pb];
      }
      if (dout) dout[i] = d;
      const uint32_t g = g8[i];
      const uint32_t w = w8[i];
      const uint32_t lo = soff[g], hi = soff[g + 1];
      if (kLds) {
        const uint32_t b = lower_bound(sthr, lo, hi, d) - lo;
        const uint32_t bin = lo + g + b;
        atomicAdd(&scnt[bin], 1u);
        atomicAdd(&sw[bin], w);
      } else {
        const uint32_t b = lower_bound(ba.thr, lo, hi, d) - lo;
        const uint32_t bin = lo + g + b;
        atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 0], 1ull);
        atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 1], (unsigned long long)w);
      }
    }
  }
  if (kLds) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < nbins; j += kAsmNT) {
      if (scnt[j]) {
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 0], (unsigned long long)scnt[j]);
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 1], (unsigned long long)sw[j]);
      }
    }
  }
}

// First position of every request r (rstart[r], r <= n_req; an empty
// request starts where the next one does): request indices are
// non-decreasing over the positions.
__global__ __launch_bounds__(256) void k_sd_rstart(const uint32_t* __restrict__ req, uint64_t n,
                                                   uint32_t n_req, uint32_t* __restrict__ rstart) {
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p <= n;
       p += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t lo = p == 0 ? 0u : req[p - 1] + 1u;  // requests that start here
    const uint32_t hi = p == n ? n_req : req[p];
    for (uint32_t r = lo; r <= hi && r <= n_req; ++r) rstart[r] = (uint32_t)p;
  }
}

// Prefix reuse: a block is reused from a cache of capacity C only if every
// block of its request up to it is (radix-tree caches reuse a request's
// longest cached prefix), i.e. the running maximum of the stack distances
// over the request, D'_i = max(D_j : j <= i in i's request), is at most C.
// One wavefront per request scans its distances 64 at a time and bins D'
// into fields 0 and 1 of `ba.hist`.
template <bool kLds>
__global__ __launch_bounds__(256) void k_sd_prefix(const uint32_t* __restrict__ D,
                                                   const uint32_t* __restrict__ rstart,
                                                   uint32_t n_req, const uint8_t* __restrict__ w8,
                                                   const uint8_t* __restrict__ g8, BinArgs ba) {
  __shared__ uint32_t sthr[kLds ? kThrLds : 1];
  __shared__ uint32_t scnt[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t sw[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t soff[KV_MAX_GROUPS + 1];
  const uint32_t nbins = ba.n_thr + ba.n_groups;
  if (threadIdx.x <= ba.n_groups) soff[threadIdx.x] = ba.off[threadIdx.x];
  if (kLds) {
    for (uint32_t j = threadIdx.x; j < ba.n_thr; j += 256) sthr[j] = ba.thr[j];
    for (uint32_t j = threadIdx.x; j < nbins; j += 256) {
      scnt[j] = 0;
      sw[j] = 0;
    }
  }
  __syncthreads();
  const uint32_t lane = lane_id();
  const uint32_t waves = gridDim.x * 4;
  for (uint32_t r = blockIdx.x * 4 + threadIdx.x / 64; r < n_req; r += waves) {
    const uint32_t b = rstart[r], e = rstart[r + 1];
    uint32_t carry = 0;
    for (uint32_t c = b; c < e; c += 64) {
      const uint32_t i = c + lane;
      uint32_t m = i < e ? D[i] : 0u;
#pragma unroll
      for (int s2 = 1; s2 < 64; s2 <<= 1) {
        const uint32_t o = (uint32_t)__shfl_up((int)m, s2, 64);
        if (lane >= (uint32_t)s2) m = max(m, o);
      }
      m = max(m, carry);
      carry = (uint32_t)__builtin_amdgcn_readlane((int)m, 63);
      if (i >= e || m == kNone) continue;   // past the request, or behind a first access
      const uint32_t g = g8[i];
      const uint32_t w = w8[i];
      const uint32_t lo = soff[g], hi = soff[g + 1];
      if (kLds) {
        const uint32_t bin = lo + g + (lower_bound(sthr, lo, hi, m) - lo);
        atomicAdd(&scnt[bin], 1u);
        atomicAdd(&sw[bin], w);
      } else {
        const uint32_t bin = lo + g + (lower_bound(ba.thr, lo, hi, m) - lo);
        atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 0], 1ull);
        atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 1], (unsigned long long)w);
      }
    }
  }
  if (kLds) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < nbins; j += 256) {
      if (scnt[j]) {
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 0], (unsigned long long)scnt[j]);
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 1], (unsigned long long)sw[j]);
      }
    }
  }
}

// weight of last occurrences, position order (scanned afterwards)
__global__ __launch_bounds__(256) void k_sd_lastw(const uint32_t* __restrict__ nxt,
                                                  const uint8_t* __restrict__ w8, uint64_t n,
                                                  uint32_t* __restrict__ lw) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x)
    lw[i] = nxt[i] == kNone ? (uint32_t)w8[i] : 0u;
}

struct SegArgs {
  uint64_t seg[KV_MAX_GROUPS + 1];
  uint32_t partitioned;
};

// Final stack depth of each block = weight of distinct blocks whose last
// access is at or after its own (inside its segment); bin it.
template <bool kLds>
__global__ __launch_bounds__(kAsmNT) void k_sd_finocc(const uint32_t* __restrict__ nxt,
                                                   const uint8_t* __restrict__ w8,
                                                   const uint8_t* __restrict__ g8, uint64_t n,
                                                   const uint32_t* __restrict__ S,
                                                   SegArgs sa, BinArgs ba) {
  __shared__ uint32_t sthr[kLds ? kThrLds : 1];
  __shared__ uint32_t scnt[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t sw[kLds ? kThrLds + KV_MAX_GROUPS : 1];
  __shared__ uint32_t soff[KV_MAX_GROUPS + 1];
  __shared__ uint32_t send[KV_MAX_GROUPS];
  const uint32_t nbins = ba.n_thr + ba.n_groups;
  if (threadIdx.x <= ba.n_groups) soff[threadIdx.x] = ba.off[threadIdx.x];
  if (threadIdx.x < KV_MAX_GROUPS) {
    const uint64_t e = sa.partitioned ? sa.seg[threadIdx.x + 1] : n;
    const uint64_t b = sa.partitioned ? sa.seg[threadIdx.x] : 0;
    send[threadIdx.x] = (e > b) ? S[e - 1] : 0u;
  }
  if (kLds) {
    for (uint32_t j = threadIdx.x; j < ba.n_thr; j += kAsmNT) sthr[j] = ba.thr[j];
    for (uint32_t j = threadIdx.x; j < nbins; j += kAsmNT) {
      scnt[j] = 0;
      sw[j] = 0;
    }
  }
  __syncthreads();
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    if (nxt[i] != kNone) continue;
    const uint32_t g = g8[i];
    const uint32_t w = w8[i];
    const uint32_t segend = sa.partitioned ? send[g] : send[0];
    const uint32_t depth = segend - (S[i] - w);
    const uint32_t lo = soff[g], hi = soff[g + 1];
    if (kLds) {
      const uint32_t bin = lo + g + (lower_bound(sthr, lo, hi, depth) - lo);
      atomicAdd(&scnt[bin], 1u);
      atomicAdd(&sw[bin], w);
    } else {
      const uint32_t bin = lo + g + (lower_bound(ba.thr, lo, hi, depth) - lo);
      atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 2], 1ull);
      atomicAdd((unsigned long long*)&ba.hist[bin * 4 + 3], (unsigned long long)w);
    }
  }
  if (kLds) {
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < nbins; j += kAsmNT) {
      if (scnt[j]) {
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 2], (unsigned long long)scnt[j]);
        atomicAdd((unsigned long long*)&ba.hist[j * 4 + 3], (unsigned long long)sw[j]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Disk TTL tiers.  A bounded TTL tier (capacity C, TTL t, least recently
// accessed block displaced first) holds a block at access i iff D_i <= C and
// its gap delta_i <= t: the blocks it holds are the top of the LRU stack up
// to C, minus those not accessed for t, and with one TTL the latter are a
// bottom part of the stack (ages grow with depth).  An unbounded one is
// C = infinity.  So per group one joint histogram of (D bin, gap bin) serves
// every (capacity, TTL), and one of (final depth bin, end-age bin) gives the
// blocks held at the last request.
// ---------------------------------------------------------------------------
constexpr uint32_t kJointNT = 1024;
constexpr uint32_t kJThrLds = 2048;     // stack-distance thresholds in LDS
constexpr uint32_t kJTtlLds = 1024;     // TTL values (+ groups) in LDS
constexpr uint32_t kJBinsLds = 4096;    // joint bins in LDS

struct JointLds {
  uint32_t thr[kJThrLds];
  double tthr[kJTtlLds];
  double wd[kJTtlLds];
  uint32_t jc[kJBinsLds], jw[kJBinsLds];
  uint32_t off[KV_MAX_GROUPS + 1], toff[KV_MAX_GROUPS + 1], jbase[KV_MAX_GROUPS + 1];
};

template <bool kLds>
__device__ __forceinline__ void joint_setup(JointLds& L, const BinArgs& ba, const JointArgs& ja) {
  const uint32_t G = ba.n_groups;
  if (threadIdx.x <= G) {
    L.off[threadIdx.x] = ba.off[threadIdx.x];
    L.toff[threadIdx.x] = ja.toff[threadIdx.x];
    L.jbase[threadIdx.x] = ja.jbase[threadIdx.x];
  }
  if (kLds) {
    for (uint32_t j = threadIdx.x; j < ba.n_thr; j += kJointNT) L.thr[j] = ba.thr[j];
    for (uint32_t j = threadIdx.x; j < ja.n_tthr; j += kJointNT) L.tthr[j] = ja.tthr[j];
    for (uint32_t j = threadIdx.x; j < ja.n_tthr + G; j += kJointNT) L.wd[j] = 0.0;
    for (uint32_t j = threadIdx.x; j < ja.n_joint; j += kJointNT) L.jc[j] = L.jw[j] = 0;
  }
  __syncthreads();
}

// bin of (d, x) in group g: d against the capacities, x against the TTLs
template <bool kLds>
__device__ __forceinline__ uint32_t joint_bin(const JointLds& L, const BinArgs& ba,
                                              const JointArgs& ja, uint32_t g, uint32_t d,
                                              bool has_x, double x, uint32_t* tb) {
  const uint32_t lo = L.off[g], hi = L.off[g + 1];
  const uint32_t db = d == kNone ? hi - lo
                                 : (kLds ? lower_bound(L.thr, lo, hi, d) : lower_bound(ba.thr, lo, hi, d)) - lo;
  const uint32_t tlo = L.toff[g], thi = L.toff[g + 1];
  const uint32_t t = !has_x ? thi - tlo
                            : (kLds ? lower_bound(L.tthr, tlo, thi, x) : lower_bound(ja.tthr, tlo, thi, x)) - tlo;
  *tb = tlo + g + t;
  return L.jbase[g] + db * (thi - tlo + 1) + t;
}

template <bool kLds>
__device__ __forceinline__ void joint_flush(JointLds& L, const JointArgs& ja, uint64_t* h,
                                            uint32_t n_groups, bool with_wd) {
  if (!kLds) return;
  __syncthreads();
  for (uint32_t j = threadIdx.x; j < ja.n_joint; j += kJointNT) {
    if (L.jc[j]) {
      atomicAdd((unsigned long long*)&h[2 * (uint64_t)j], (unsigned long long)L.jc[j]);
      atomicAdd((unsigned long long*)&h[2 * (uint64_t)j + 1], (unsigned long long)L.jw[j]);
    }
  }
  if (with_wd)
    for (uint32_t j = threadIdx.x; j < ja.n_tthr + n_groups; j += kJointNT)
      if (L.wd[j] != 0.0) atomicAdd(&ja.wd[j], L.wd[j]);
}

// Accesses by (stack distance, gap to the block's previous access), plus the
// weighted gaps per gap bin (for the storage integral).
template <bool kLds>
__global__ __launch_bounds__(kJointNT) void k_sd_joint(const uint32_t* __restrict__ dist,
                                                       const uint32_t* __restrict__ key,
                                                       const uint32_t* __restrict__ req,
                                                       const double* __restrict__ rt,
                                                       const uint8_t* __restrict__ w8,
                                                       const uint8_t* __restrict__ g8, uint64_t n,
                                                       BinArgs ba, JointArgs ja) {
  __shared__ JointLds L;
  joint_setup<kLds>(L, ba, ja);
  for (uint64_t i = (uint64_t)blockIdx.x * kJointNT + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * kJointNT) {
    const uint32_t k = key[i];
    const uint32_t g = g8[i], w = w8[i];
    const double gap = k ? rt[req[i]] - rt[req[k - 1]] : 0.0;
    uint32_t tb;
    const uint32_t b = joint_bin<kLds>(L, ba, ja, g, dist[i], k != 0, gap, &tb);
    if (kLds) {
      atomicAdd(&L.jc[b], 1u);
      atomicAdd(&L.jw[b], w);
      if (k) atomicAdd(&L.wd[tb], (double)w * gap);
    } else {
      atomicAdd((unsigned long long*)&ja.jh[2 * (uint64_t)b], 1ull);
      atomicAdd((unsigned long long*)&ja.jh[2 * (uint64_t)b + 1], (unsigned long long)w);
      if (k) atomicAdd(&ja.wd[tb], (double)w * gap);
    }
  }
  joint_flush<kLds>(L, ja, ja.jh, ba.n_groups, true);
}

// Blocks by (final stack depth, age at the last request), at their last access.
template <bool kLds>
__global__ __launch_bounds__(kJointNT) void k_sd_finjoint(const uint32_t* __restrict__ nxt,
                                                          const uint32_t* __restrict__ req,
                                                          const double* __restrict__ rt,
                                                          const uint8_t* __restrict__ w8,
                                                          const uint8_t* __restrict__ g8,
                                                          uint64_t n,
                                                          const uint32_t* __restrict__ S,
                                                          BinArgs ba, JointArgs ja) {
  __shared__ JointLds L;
  joint_setup<kLds>(L, ba, ja);
  const uint32_t segend = S[n - 1];
  const double t_end = rt[req[n - 1]];  // the last access's request
  for (uint64_t i = (uint64_t)blockIdx.x * kJointNT + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * kJointNT) {
    if (nxt[i] != kNone) continue;
    const uint32_t g = g8[i], w = w8[i];
    const uint32_t depth = segend - (S[i] - w);
    uint32_t tb;
    const uint32_t b = joint_bin<kLds>(L, ba, ja, g, depth, true, t_end - rt[req[i]], &tb);
    if (kLds) {
      atomicAdd(&L.jc[b], 1u);
      atomicAdd(&L.jw[b], w);
    } else {
      atomicAdd((unsigned long long*)&ja.fh[2 * (uint64_t)b], 1ull);
      atomicAdd((unsigned long long*)&ja.fh[2 * (uint64_t)b + 1], (unsigned long long)w);
    }
  }
  joint_flush<kLds>(L, ja, ja.fh, ba.n_groups, false);
}

// Cumulative over both bin dimensions, one block per group; wd over gap bins.
__global__ __launch_bounds__(256) void k_joint_cum(uint64_t* __restrict__ jh,
                                                   uint64_t* __restrict__ fh,
                                                   double* __restrict__ wd,
                                                   const uint32_t* __restrict__ off,
                                                   const uint32_t* __restrict__ toff,
                                                   const uint32_t* __restrict__ jbase) {
  const uint32_t g = blockIdx.x;
  const uint32_t nd = off[g + 1] - off[g] + 1, nt = toff[g + 1] - toff[g] + 1;
  const uint64_t b0 = jbase[g];
  for (uint32_t q = threadIdx.x; q < 4 * nd; q += blockDim.x) {  // along gap bins
    uint64_t* h = (q & 2) ? fh : jh;
    const uint32_t f = q & 1, d = q >> 2;
    uint64_t run = 0;
    for (uint32_t t = 0; t < nt; ++t) {
      uint64_t& x = h[2 * (b0 + (uint64_t)d * nt + t) + f];
      run += x;
      x = run;
    }
  }
  __syncthreads();
  for (uint32_t q = threadIdx.x; q < 4 * nt; q += blockDim.x) {  // along distance bins
    uint64_t* h = (q & 2) ? fh : jh;
    const uint32_t f = q & 1, t = q >> 2;
    uint64_t run = 0;
    for (uint32_t d = 0; d < nd; ++d) {
      uint64_t& x = h[2 * (b0 + (uint64_t)d * nt + t) + f];
      run += x;
      x = run;
    }
  }
  if (threadIdx.x == 0) {
    double run = 0.0;
    for (uint32_t t = 0; t < nt; ++t) {
      run += wd[toff[g] + g + t];
      wd[toff[g] + g + t] = run;
    }
  }
}

// cumulative over the bins of each group, one thread per (group, field)
__global__ void k_hist_cum(uint64_t* hist, const uint32_t* __restrict__ off, uint32_t n_groups) {
  const uint32_t g = threadIdx.x / 4, f = threadIdx.x % 4;
  if (g >= n_groups) return;
  const uint32_t b0 = off[g] + g, b1 = off[g + 1] + g + 1;
  uint64_t run = 0;
  for (uint32_t b = b0; b < b1; ++b) {
    run += hist[b * 4 + f];
    hist[b * 4 + f] = run;
  }
}

// Test hooks, read at every call: KVCFG_TEST_ROW_CHUNK narrows the LDS
// histogram of a block-matrix row (so that short traces take the
// column-chunk path of long ones); KVCFG_TEST_THR_LDS lowers the number of
// thresholds binned in LDS (so that few thresholds take the global-atomic
// path of very many).  Both only select among paths of the same result.
uint32_t env_limit(const char* name, uint32_t dflt, uint32_t lo) {
  const char* e = std::getenv(name);
  if (!e) return dflt;
  const unsigned long v = std::strtoul(e, nullptr, 10);
  return (uint32_t)std::max<unsigned long>(lo, std::min<unsigned long>(v, dflt));
}

uint32_t grid_of(uint64_t m, uint32_t cap = 32768) {
  uint64_t g = (m + 255) / 256;
  if (g > cap) g = cap;
  return (uint32_t)(g ? g : 1);
}

}  // namespace

kv_status stack_pass(Trace& t, Order& o, bool partitioned, const ThresholdSet& ts,
                     const uint32_t* thr_dev, const uint32_t* off_dev, uint64_t* hist,
                     uint64_t* phist, const JointArgs* ja, const uint8_t* real, hipStream_t s) {
  const uint64_t n = o.n ? o.n : t.n;
  const uint32_t G = div_up(n, kSdB);
  kv_status st;
  const uint64_t tri = G >= 2 ? tri_off(G) : 1;
  const uint32_t nchunks = div_up(G, kColRows);
  DevBuf& b_partial = t.ws[0];
  DevBuf& b_E = t.ws[1];
  DevBuf& b_Q = t.ws[2];
  DevBuf& b_csum = t.ws[3];
  DevBuf& b_scan = t.ws[4];
  if ((st = b_partial.reserve(n * 4)) != KV_OK) return st;
  if ((st = b_E.reserve(n * 4)) != KV_OK) return st;
  if ((st = b_Q.reserve(tri * 4)) != KV_OK) return st;
  if ((st = b_csum.reserve((uint64_t)nchunks * G * 4)) != KV_OK) return st;
  if ((st = b_scan.reserve(std::max<uint64_t>(scan_scratch_elems(n), 1) * 4)) != KV_OK) return st;
  // prefix reuse and disk TTL tiers (trace order only): every access's
  // distance; request starts
  uint32_t* dist = nullptr;
  uint32_t* rstart = nullptr;
  if (phist || ja) {
    if (partitioned) return fail(KV_ERR_UNSUPPORTED, "this mode needs the trace order");
    if ((st = t.ws[25].reserve(n * 4)) != KV_OK) return st;
    dist = t.ws[25].as<uint32_t>();
  }
  if (phist) {
    if ((st = t.ws[26].reserve(((uint64_t)t.st.n_req + 1) * 4)) != KV_OK) return st;
    rstart = t.ws[26].as<uint32_t>();
  }
  const uint32_t* key = o.key.as<uint32_t>();
  const uint32_t* nxt = o.nxt.as<uint32_t>();
  const uint8_t* w8 = o.w.as<uint8_t>();
  const uint8_t* g8 = o.g.as<uint8_t>();
  uint32_t* Q = b_Q.as<uint32_t>();
  if (G >= 2) {
    StageTimer tm(kStStackMatrix, s);
    const uint32_t row_chunk = env_limit("KVCFG_TEST_ROW_CHUNK", kRowChunk, 1);
    hipLaunchKernelGGL(k_sd_rowhist, dim3(G), dim3(kRowNT), 0, s, key, w8, n, row_chunk, Q);
    KV_HIP(hipGetLastError());
    const dim3 cg(div_up(G, 256), nchunks);
    hipLaunchKernelGGL(k_sd_colsum, cg, dim3(256), 0, s, Q, G, b_csum.as<uint32_t>());
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_sd_colchunks, dim3(div_up(G, 256)), dim3(256), 0, s,
                       b_csum.as<uint32_t>(), G, nchunks);
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_sd_colapply, cg, dim3(256), 0, s, Q, G,
                       (const uint32_t*)b_csum.as<uint32_t>());
    KV_HIP(hipGetLastError());
  }
  {
    StageTimer tm(kStStackLocal, s);
    hipLaunchKernelGGL(k_sd_local, dim3(G), dim3(kLocNT), 0, s, key, nxt, w8, n, G,
                       b_partial.as<uint32_t>(), b_E.as<uint32_t>());
    KV_HIP(hipGetLastError());
  }
  BinArgs ba{thr_dev, off_dev, (uint32_t)ts.values.size(), ts.n_groups, hist};
  const uint32_t lds_limit = env_limit("KVCFG_TEST_THR_LDS", kThrLds, 0);
  const bool lds = ts.values.size() + ts.n_groups <= lds_limit;
  const bool jlds = ja && lds_limit > 0 && ts.values.size() <= kJThrLds &&
                    ja->n_tthr + ts.n_groups <= kJTtlLds && ja->n_joint <= kJBinsLds;
  const uint32_t gj = std::min<uint32_t>(div_up(n, kJointNT), 1024);
  // two workgroups per compute unit (their LDS histograms allow two): each
  // flushes its histogram once, so fewer and larger ones flush less
  const uint32_t ga = std::min<uint32_t>(G, 512);
  {
  StageTimer tm(kStStackAssemble, s);
  if (lds)
    hipLaunchKernelGGL(k_sd_assemble<true>, dim3(ga), dim3(kAsmNT), 0, s, key, w8, g8, n, G,
                       (const uint32_t*)b_partial.as<uint32_t>(),
                       (const uint32_t*)b_E.as<uint32_t>(), (const uint32_t*)Q, ba, dist, real);
  else
    hipLaunchKernelGGL(k_sd_assemble<false>, dim3(ga), dim3(kAsmNT), 0, s, key, w8, g8, n, G,
                       (const uint32_t*)b_partial.as<uint32_t>(),
                       (const uint32_t*)b_E.as<uint32_t>(), (const uint32_t*)Q, ba, dist, real);
  KV_HIP(hipGetLastError());
  if (phist) {
    const uint32_t nr = t.st.n_req;
    hipLaunchKernelGGL(k_sd_rstart, dim3(grid_of(n + 1)), dim3(256), 0, s,
                       t.req.as<uint32_t>(), n, nr, rstart);
    KV_HIP(hipGetLastError());
    BinArgs bp{thr_dev, off_dev, (uint32_t)ts.values.size(), ts.n_groups, phist};
    const uint32_t gp = std::min<uint32_t>(div_up(nr, 4), 4096);
    if (lds)
      hipLaunchKernelGGL(k_sd_prefix<true>, dim3(gp), dim3(256), 0, s, (const uint32_t*)dist,
                         (const uint32_t*)rstart, nr, w8, g8, bp);
    else
      hipLaunchKernelGGL(k_sd_prefix<false>, dim3(gp), dim3(256), 0, s, (const uint32_t*)dist,
                         (const uint32_t*)rstart, nr, w8, g8, bp);
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_hist_cum, dim3(1), dim3(4 * KV_MAX_GROUPS), 0, s, phist, off_dev,
                       ts.n_groups);
    KV_HIP(hipGetLastError());
  }
  if (ja) {
    const uint32_t* rq = t.req.as<uint32_t>();
    const double* rt = t.req_time.as<double>();
    if (jlds)
      hipLaunchKernelGGL(k_sd_joint<true>, dim3(gj), dim3(kJointNT), 0, s, (const uint32_t*)dist,
                         key, rq, rt, w8, g8, n, ba, *ja);
    else
      hipLaunchKernelGGL(k_sd_joint<false>, dim3(gj), dim3(kJointNT), 0, s,
                         (const uint32_t*)dist, key, rq, rt, w8, g8, n, ba, *ja);
    KV_HIP(hipGetLastError());
  }
  }
  StageTimer tm(kStStackFinal, s);
  // final occupancy: reuse `partial` for the scanned last-occurrence weights
  uint32_t* S = b_partial.as<uint32_t>();
  hipLaunchKernelGGL(k_sd_lastw, dim3(grid_of(n)), dim3(256), 0, s, nxt, w8, n, S);
  KV_HIP(hipGetLastError());
  if ((st = scan_u32(S, S, n, true, b_scan.as<uint32_t>(), s)) != KV_OK) return st;
  SegArgs sa{};
  for (int g = 0; g <= KV_MAX_GROUPS; ++g) sa.seg[g] = o.seg[g];
  sa.partitioned = partitioned ? 1u : 0u;
  const uint32_t gf = std::min<uint32_t>(div_up(n, kAsmNT), 512);  // two per compute unit, as above
  if (lds)
    hipLaunchKernelGGL(k_sd_finocc<true>, dim3(gf), dim3(kAsmNT), 0, s, nxt, w8, g8, n,
                       (const uint32_t*)S, sa, ba);
  else
    hipLaunchKernelGGL(k_sd_finocc<false>, dim3(gf), dim3(kAsmNT), 0, s, nxt, w8, g8, n,
                       (const uint32_t*)S, sa, ba);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_hist_cum, dim3(1), dim3(4 * KV_MAX_GROUPS), 0, s, hist, off_dev,
                     ts.n_groups);
  KV_HIP(hipGetLastError());
  if (ja) {
    const uint32_t* rq = t.req.as<uint32_t>();
    const double* rt = t.req_time.as<double>();
    if (jlds)
      hipLaunchKernelGGL(k_sd_finjoint<true>, dim3(gj), dim3(kJointNT), 0, s, nxt, rq, rt, w8,
                         g8, n, (const uint32_t*)S, ba, *ja);
    else
      hipLaunchKernelGGL(k_sd_finjoint<false>, dim3(gj), dim3(kJointNT), 0, s, nxt, rq, rt, w8,
                         g8, n, (const uint32_t*)S, ba, *ja);
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_joint_cum, dim3(ts.n_groups), dim3(256), 0, s, ja->jh, ja->fh, ja->wd,
                       off_dev, ja->toff, ja->jbase);
    KV_HIP(hipGetLastError());
  }
  return KV_OK;
}

}  // namespace kv
