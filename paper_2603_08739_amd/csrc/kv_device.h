// kv_device.h - small device-side building blocks for 64-wide wavefronts.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kv {

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// The wave's index in the block, as a wave-uniform (scalar) value: tests on
// it need no per-lane masks.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / 64));
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const uint32_t l = lane_id();
  return (l == 0) ? 0ull : (~0ull >> (64 - l));
}

// Inclusive prefix sum across the 64 lanes of a wavefront.
template <class T>
__device__ __forceinline__ T wave_incl_scan(T v) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    T o = __shfl_up(v, d, 64);
    if ((int)lane_id() >= d) v += o;
  }
  return v;
}

// Inclusive prefix sum of 32-bit values across the 64 lanes with DPP: row
// shifts build the sums inside each row of 16 lanes, two row broadcasts carry
// them across rows.  Lanes outside a DPP source row add 0.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

// Inclusive prefix sum over the first row of 16 lanes (lanes past 15 hold
// partial sums of their own rows, unused here).
__device__ __forceinline__ uint32_t row_incl_scan_u32(uint32_t v) {
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);  // row_shr:8
  return v;
}

// The wave totals `sh[0..NW)` combined for wave w: the sum over waves below
// w and the sum over all, as wave-uniform values.  Lane i reads total i and
// a row scan adds them up, so every thread does one LDS read.
template <int NW>
__device__ __forceinline__ void wave_totals(const uint32_t* sh, int w, uint32_t& below,
                                            uint32_t& all) {
  static_assert(NW <= 16, "one row of lanes holds the wave totals");
  const uint32_t lane = lane_id();
  const uint32_t y = lane < (uint32_t)NW ? sh[lane] : 0u;
  const int incl = (int)row_incl_scan_u32(y);
  all = (uint32_t)__builtin_amdgcn_readlane(incl, NW - 1);
  below = w ? (uint32_t)__builtin_amdgcn_readlane(incl, w - 1) : 0u;
}

// Exclusive prefix sums of two 32-bit values over a block of NT threads.
// `sh` holds 2 * (NT / 64) words of shared memory; two barriers.  With
// Trail = false the second barrier (which lets the next call reuse `sh`) is
// left out: consecutive calls must then alternate between two buffers.
template <int NT, bool Trail = true>
__device__ __forceinline__ void block_excl_scan2_u32(uint32_t a, uint32_t b, uint32_t* sh,
                                                     uint32_t& pa, uint32_t& pb, uint32_t& ta,
                                                     uint32_t& tb) {
  constexpr int NW = NT / 64;
  const int w = wave_id();
  const uint32_t ia = wave_incl_scan_u32(a), ib = wave_incl_scan_u32(b);
  if (lane_id() == 63) {
    sh[w] = ia;
    sh[NW + w] = ib;
  }
  __syncthreads();
  uint32_t sa, sb, xa, xb;
  wave_totals<NW>(sh, w, xa, sa);
  wave_totals<NW>(sh + NW, w, xb, sb);
  if constexpr (Trail) __syncthreads();
  pa = xa + ia - a;
  pb = xb + ib - b;
  ta = sa;
  tb = sb;
}

template <int NT, bool Trail = true>
__device__ __forceinline__ uint32_t block_excl_scan_u32(uint32_t a, uint32_t* sh, uint32_t& ta) {
  constexpr int NW = NT / 64;
  const int w = wave_id();
  const uint32_t ia = wave_incl_scan_u32(a);
  if (lane_id() == 63) sh[w] = ia;
  __syncthreads();
  uint32_t xa, sa;
  wave_totals<NW>(sh, w, xa, sa);
  if constexpr (Trail) __syncthreads();
  ta = sa;
  return xa + ia - a;
}

// Sum and maximum over the 64 lanes via DPP (result in every lane).
__device__ __forceinline__ uint32_t wave_add_dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan_u32(v), 63);
}

__device__ __forceinline__ uint32_t wave_max_dpp(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false));
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Whether any thread of the block passes true: one barrier per call.  Two
// LDS flag words (zero at start) alternate between calls, so a call never
// overwrites the word a slower thread may still read from the call before.
struct BlockAny {
  uint32_t* flag;
  uint32_t gen;
  __device__ __forceinline__ bool operator()(bool p) {
    ++gen;
    const bool any = __ballot(p) != 0ull;
    if (any && lane_id() == 0) flag[gen & 1u] = gen;
    __syncthreads();
    return flag[gen & 1u] == gen;
  }
};

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = max(v, (uint32_t)__shfl_xor(v, d, 64));
  return v;
}

// Bit m of the low 16 bits moves to bit 4m.
__device__ __forceinline__ uint64_t spread4(uint64_t x) {
  x &= 0xFFFFull;
  x = (x | (x << 24)) & 0x000000FF000000FFull;
  x = (x | (x << 12)) & 0x000F000F000F000Full;
  x = (x | (x << 6)) & 0x0303030303030303ull;
  x = (x | (x << 3)) & 0x1111111111111111ull;
  return x;
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// Exclusive prefix sum over a block of NT threads; returns the thread's
// exclusive prefix and writes the block total to *total.  `sh` must hold
// NT/64 + 1 elements of shared memory.
template <int NT, class T>
__device__ __forceinline__ T block_excl_scan(T v, T* sh, T* total) {
  constexpr int NW = NT / 64;
  const int w = wave_id();
  T inc = wave_incl_scan(v);
  if (lane_id() == 63) sh[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = 0;
    for (int i = 0; i < NW; ++i) {
      T x = sh[i];
      sh[i] = run;
      run += x;
    }
    sh[NW] = run;
  }
  __syncthreads();
  T r = sh[w] + inc - v;
  *total = sh[NW];
  __syncthreads();
  return r;
}

template <int NT, class T>
__device__ __forceinline__ T block_sum(T v, T* sh) {
  constexpr int NW = NT / 64;
  const int w = wave_id();
  T s = wave_sum(v);
  if (lane_id() == 0) sh[w] = s;
  __syncthreads();
  T r = 0;
  for (int i = 0; i < NW; ++i) r += sh[i];
  __syncthreads();
  return r;
}

// First index in sorted a[lo, hi) with a[i] >= x.
template <class T, class A>
__device__ __forceinline__ uint32_t lower_bound(const A* a, uint32_t lo, uint32_t hi, T x) {
  while (lo < hi) {
    uint32_t mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// First index in sorted a[lo, hi) with a[i] > x.
template <class T, class A>
__device__ __forceinline__ uint32_t upper_bound(const A* a, uint32_t lo, uint32_t hi, T x) {
  while (lo < hi) {
    uint32_t mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

inline uint32_t div_up(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }

}  // namespace kv
