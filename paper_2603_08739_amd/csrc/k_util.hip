// k_util.hip - device-wide prefix sums and fills.
#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr int kScanNT = 256;
constexpr int kScanItems = 16;
constexpr uint32_t kScanTile = kScanNT * kScanItems;  // 4096

__global__ __launch_bounds__(kScanNT) void k_scan_reduce(const uint32_t* __restrict__ in,
                                                         uint64_t m, uint32_t* __restrict__ sums) {
  __shared__ uint32_t sh[kScanNT / 64 + 1];
  const uint64_t base = (uint64_t)blockIdx.x * kScanTile;
  uint32_t v = 0;
  for (int e = 0; e < kScanItems; ++e) {
    uint64_t i = base + (uint64_t)e * kScanNT + threadIdx.x;
    if (i < m) v += in[i];
  }
  uint32_t s = block_sum<kScanNT>(v, sh);
  if (threadIdx.x == 0) sums[blockIdx.x] = s;
}

// Each thread scans kScanItems consecutive elements; `offs` (may be null)
// holds the exclusive prefix of every tile.
__global__ __launch_bounds__(kScanNT) void k_scan_apply(const uint32_t* in,
                                                        uint32_t* out, uint64_t m,
                                                        const uint32_t* __restrict__ offs,
                                                        int inclusive) {
  __shared__ uint32_t stage[kScanTile];
  __shared__ uint32_t sh[kScanNT / 64 + 1];
  const uint64_t base = (uint64_t)blockIdx.x * kScanTile;
  for (int e = 0; e < kScanItems; ++e) {
    uint32_t j = e * kScanNT + threadIdx.x;
    uint64_t i = base + j;
    stage[j] = (i < m) ? in[i] : 0u;
  }
  __syncthreads();
  uint32_t loc[kScanItems];
  uint32_t run = 0;
  for (int e = 0; e < kScanItems; ++e) {
    uint32_t x = stage[threadIdx.x * kScanItems + e];
    loc[e] = inclusive ? run + x : run;
    run += x;
  }
  uint32_t total;
  uint32_t pre = block_excl_scan<kScanNT>(run, sh, &total);
  const uint32_t off = offs ? offs[blockIdx.x] : 0u;
  for (int e = 0; e < kScanItems; ++e) stage[threadIdx.x * kScanItems + e] = loc[e] + pre + off;
  __syncthreads();
  for (int e = 0; e < kScanItems; ++e) {
    uint32_t j = e * kScanNT + threadIdx.x;
    uint64_t i = base + j;
    if (i < m) out[i] = stage[j];
  }
}

__global__ void k_fill_u32(uint32_t* p, uint32_t v, uint64_t m) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_fill_u64(uint64_t* p, uint64_t v, uint64_t m) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m;
       i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

uint32_t grid_for(uint64_t m, uint32_t nt) {
  uint64_t g = (m + nt - 1) / nt;
  if (g > 65536) g = 65536;
  return (uint32_t)(g ? g : 1);
}

}  // namespace

kv_status fill_u32(uint32_t* p, uint32_t v, uint64_t m, hipStream_t s) {
  if (m == 0) return KV_OK;
  hipLaunchKernelGGL(k_fill_u32, dim3(grid_for(m, 256)), dim3(256), 0, s, p, v, m);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

kv_status fill_u64(uint64_t* p, uint64_t v, uint64_t m, hipStream_t s) {
  if (m == 0) return KV_OK;
  hipLaunchKernelGGL(k_fill_u64, dim3(grid_for(m, 256)), dim3(256), 0, s, p, v, m);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

uint64_t scan_scratch_elems(uint64_t m) {
  uint64_t tiles = (m + kScanTile - 1) / kScanTile;
  if (tiles <= 1) return 0;
  return 2 * tiles + scan_scratch_elems(tiles);
}

kv_status scan_u32(const uint32_t* in, uint32_t* out, uint64_t m, bool inclusive,
                   uint32_t* scratch, hipStream_t s) {
  if (m == 0) return KV_OK;
  const uint64_t tiles = (m + kScanTile - 1) / kScanTile;
  if (tiles == 1) {
    hipLaunchKernelGGL(k_scan_apply, dim3(1), dim3(kScanNT), 0, s, in, out, m,
                       (const uint32_t*)nullptr, inclusive ? 1 : 0);
    KV_HIP(hipGetLastError());
    return KV_OK;
  }
  uint32_t* a = scratch;
  uint32_t* b = a + tiles;
  hipLaunchKernelGGL(k_scan_reduce, dim3((uint32_t)tiles), dim3(kScanNT), 0, s, in, m, a);
  KV_HIP(hipGetLastError());
  kv_status st = scan_u32(a, b, tiles, false, b + tiles, s);
  if (st != KV_OK) return st;
  hipLaunchKernelGGL(k_scan_apply, dim3((uint32_t)tiles), dim3(kScanNT), 0, s, in, out, m,
                     (const uint32_t*)b, inclusive ? 1 : 0);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

}  // namespace kv
