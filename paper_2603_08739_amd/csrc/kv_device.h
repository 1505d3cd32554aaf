// kv_device.h - small device-side building blocks for 64-wide wavefronts.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kv {

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

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
  const int w = threadIdx.x / 64;
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
  const int w = threadIdx.x / 64;
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
