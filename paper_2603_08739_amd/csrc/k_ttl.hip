// k_ttl.hip - TTL retention curves of the disk tier (Section 4.3).
//
// Under a time-to-live t a block stays on disk for t seconds after each of
// its accesses, so an access hits iff the gap delta to its block's previous
// access is at most t, and a block with accesses a_1 < ... < a_m occupies
// storage for sum_j min(t, a_{j+1} - a_j) + t seconds.  Per group, the hits
// H_g(t) and the storage integral C_g(t) for every t of a sorted list follow
// from one histogram of the gaps over the list's bins:
//   bin(delta) = #{k : ttl[k] < delta}, so delta <= ttl[k] <=> bin <= k;
//   H_g(ttl[k])  = sum of the counts of bins 0..k
//   C_g(ttl[k])  = W_g*ttl[k] + sum_{delta <= ttl[k]} w*delta
//                  + ttl[k] * (weight of the gaps above ttl[k]).
// The pass is a stream over the trace with one dependent gather per access
// (the request of the previous access); the histogram lives in LDS.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr int kTtlNT = 1024;       // threads per workgroup
constexpr int kTtlU = 8;           // accesses per thread per step (gathers in flight)
static_assert(kTtlU % 4 == 0, "accesses are read four at a time");
constexpr uint32_t kTtlMax = 1024; // TTL values per call
constexpr uint32_t kTtlBins = 4096;  // groups * (TTL values + 1)

// Gap histogram: per (group, bin) the number of gaps, their summed weight
// and the summed weight * gap, added into the zeroed global arrays.  In LDS
// the count and the weight share one 64-bit word (count << 32 | weight: with
// n <= 2^29 over up to 1024 workgroups a workgroup sees at most 2^19
// accesses of at most 255 granules each, so the weight never carries).
__global__ __launch_bounds__(kTtlNT) void k_ttl_hist(
    const uint32_t* __restrict__ key, const uint32_t* __restrict__ req,
    const double* __restrict__ rt, const uint8_t* __restrict__ w8,
    const uint8_t* __restrict__ g8, uint64_t n, const double* __restrict__ ttl, uint32_t n_ttl,
    uint32_t bins, unsigned long long* __restrict__ cnt, unsigned long long* __restrict__ wsum,
    double* __restrict__ wd) {
  __shared__ unsigned long long hcw[kTtlBins];
  __shared__ double hd[kTtlBins];
  __shared__ double tt[kTtlMax];
  const uint32_t tid = threadIdx.x;
  const uint32_t nb = n_ttl + 1;
  for (uint32_t i = tid; i < bins; i += kTtlNT) {
    hcw[i] = 0;
    hd[i] = 0.0;
  }
  for (uint32_t i = tid; i < n_ttl; i += kTtlNT) tt[i] = ttl[i];
  __syncthreads();
  const uint64_t step = (uint64_t)gridDim.x * kTtlNT * kTtlU;
  for (uint64_t p0 = (uint64_t)blockIdx.x * kTtlNT * kTtlU; p0 < n; p0 += step) {
    // each thread takes kTtlU consecutive accesses, read as vectors (the
    // arrays hold 16 readable bytes past n; accesses past n are dropped)
    uint32_t k[kTtlU], r[kTtlU], rp[kTtlU], w[kTtlU], g[kTtlU];
    const uint64_t pt = p0 + (uint64_t)tid * kTtlU;
#pragma unroll
    for (int q = 0; q < kTtlU / 4; ++q) {
      const uint64_t pq = min<uint64_t>(pt + 4 * q, n & ~3ull);
      const uint4 kv = *reinterpret_cast<const uint4*>(key + pq);
      const uint4 rv = *reinterpret_cast<const uint4*>(req + pq);
      const uint32_t wv = *reinterpret_cast<const uint32_t*>(w8 + pq);
      const uint32_t gv = *reinterpret_cast<const uint32_t*>(g8 + pq);
      const uint32_t ka[4] = {kv.x, kv.y, kv.z, kv.w}, ra[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool in = pq == pt + 4 * q && pt + 4 * q + e < n;
        k[4 * q + e] = in ? ka[e] : 0u;
        r[4 * q + e] = ra[e];
        w[4 * q + e] = (wv >> (8 * e)) & 0xFFu;
        g[4 * q + e] = (gv >> (8 * e)) & 0xFFu;
      }
    }
#pragma unroll
    for (int u = 0; u < kTtlU; ++u) rp[u] = k[u] ? req[k[u] - 1] : 0u;
#pragma unroll
    for (int u = 0; u < kTtlU; ++u) {
      if (!k[u]) continue;  // no earlier access: no gap
      const double delta = rt[r[u]] - rt[rp[u]];
      const uint32_t b = lower_bound(tt, 0u, n_ttl, delta);
      const uint32_t idx = g[u] * nb + b;
      atomicAdd(&hcw[idx], (1ull << 32) | w[u]);
      atomicAdd(&hd[idx], (double)w[u] * delta);
    }
  }
  __syncthreads();
  for (uint32_t i = tid; i < bins; i += kTtlNT) {
    const unsigned long long x = hcw[i];
    if (!x) continue;
    atomicAdd(&cnt[i], x >> 32);
    atomicAdd(&wsum[i], x & 0xFFFFFFFFull);
    atomicAdd(&wd[i], hd[i]);
  }
}

struct GroupWeights {
  unsigned long long w[KV_MAX_GROUPS];  // distinct weight per group
};

// Cumulative curves, one thread per group (bins in ascending order).
__global__ void k_ttl_fin(const unsigned long long* __restrict__ cnt,
                          const unsigned long long* __restrict__ wsum,
                          const double* __restrict__ wd, const double* __restrict__ ttl,
                          uint32_t n_ttl, uint32_t n_groups, GroupWeights W,
                          uint64_t* __restrict__ hits, uint64_t* __restrict__ hitw,
                          double* __restrict__ store) {
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  const uint32_t nb = n_ttl + 1;
  const unsigned long long* c = cnt + (uint64_t)g * nb;
  const unsigned long long* ws = wsum + (uint64_t)g * nb;
  const double* d = wd + (uint64_t)g * nb;
  unsigned long long P = 0;  // weight of every gap of the group
  for (uint32_t b = 0; b < nb; ++b) P += ws[b];
  unsigned long long hc = 0, hw = 0;
  double s = 0.0;
  const double Wg = (double)W.w[g];
  for (uint32_t k = 0; k < n_ttl; ++k) {
    hc += c[k];
    hw += ws[k];
    s += d[k];
    const double t = ttl[k];
    hits[(uint64_t)g * n_ttl + k] = hc;
    hitw[(uint64_t)g * n_ttl + k] = hw;
    store[(uint64_t)g * n_ttl + k] = Wg * t + s + t * (double)(P - hw);
  }
}

}  // namespace

// The no-allocation variant's device memory: the TTL values, then the three
// gap histograms (count, weight, weight * gap) of at most kTtlBins bins.
// Each device holds its own copy for the life of the process; host code
// reaches it only through the address hipGetSymbolAddress returns.
constexpr size_t kScratchTtlBytes = (size_t)kTtlMax * sizeof(double);
constexpr size_t kScratchBytes = kScratchTtlBytes + (size_t)kTtlBins * 3 * sizeof(uint64_t);
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
kv_status scratch_ptr(uint8_t** out) {
  static std::mutex mu;
  static void* per_dev[64] = {};
  int d = 0;
  KV_HIP(hipGetDevice(&d));
  if (d < 0 || d >= 64) return fail(KV_ERR_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(mu);
  if (!per_dev[d]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      (void)hipGetLastError();
      return fail(KV_ERR_DEVICE, std::string("kv_ttl_curves_noalloc: no address for the "
                                             "scratch array: ") + hipGetErrorString(e));
    }
    per_dev[d] = p;
  }
  *out = static_cast<uint8_t*>(per_dev[d]);
  return KV_OK;
}
}  // namespace

kv_status ttl_curves_noalloc(Trace& t, const double* ttl_host, uint32_t n_ttl, uint64_t* hits,
                             uint64_t* hitw, double* store, hipStream_t s) {
  if (n_ttl > kTtlMax || (uint64_t)t.n_groups * (n_ttl + 1) > kTtlBins)
    return fail(KV_ERR_UNSUPPORTED,
                "kv_ttl_curves_noalloc: n_groups * (n_ttl + 1) must be <= 4096");
  uint8_t* base = nullptr;
  kv_status st;
  if ((st = scratch_ptr(&base)) != KV_OK) return st;
  double* ttl_dev = reinterpret_cast<double*>(base);
  KV_HIP(hipMemcpyAsync(ttl_dev, ttl_host, (size_t)n_ttl * sizeof(double),
                        hipMemcpyHostToDevice, s));
  return ttl_curves_into(t, ttl_dev, n_ttl,
                         reinterpret_cast<unsigned long long*>(base + kScratchTtlBytes), hits,
                         hitw, store, s);
}

kv_status ttl_curves(Trace& t, const double* ttl_dev, uint32_t n_ttl, uint64_t* hits,
                     uint64_t* hitw, double* store, hipStream_t s) {
  const uint32_t G = t.n_groups;
  const uint32_t bins = G * (n_ttl + 1);
  if (n_ttl > kTtlMax || bins > kTtlBins)
    return fail(KV_ERR_UNSUPPORTED, "kv_ttl_curves: n_groups * (n_ttl + 1) must be <= 4096");
  DevBuf& bh = t.ws[22];
  kv_status st;
  if ((st = bh.reserve((uint64_t)bins * 24)) != KV_OK) return st;
  return ttl_curves_into(t, ttl_dev, n_ttl, bh.as<unsigned long long>(), hits, hitw, store, s);
}

kv_status ttl_curves_into(Trace& t, const double* ttl_dev, uint32_t n_ttl,
                          unsigned long long* cnt, uint64_t* hits, uint64_t* hitw,
                          double* store, hipStream_t s) {
  const uint32_t G = t.n_groups;
  const uint32_t bins = G * (n_ttl + 1);
  kv_status st;
  unsigned long long* wsum = cnt + bins;
  double* wd = reinterpret_cast<double*>(wsum + bins);
  StageTimer tm(kStTtl, s);
  if ((st = fill_u64(reinterpret_cast<uint64_t*>(cnt), 0, (uint64_t)bins * 3, s)) != KV_OK)
    return st;
  const uint64_t per_block = (uint64_t)kTtlNT * kTtlU;
  const uint32_t nblk = (uint32_t)std::min<uint64_t>((t.n + per_block - 1) / per_block, 1024);
  hipLaunchKernelGGL(k_ttl_hist, dim3(nblk), dim3(kTtlNT), 0, s, t.shared.key.as<uint32_t>(),
                     t.req.as<uint32_t>(), t.req_time.as<double>(), t.shared.w.as<uint8_t>(),
                     t.shared.g.as<uint8_t>(), t.n, ttl_dev, n_ttl, bins, cnt, wsum, wd);
  KV_HIP(hipGetLastError());
  GroupWeights W{};
  for (uint32_t g = 0; g < KV_MAX_GROUPS; ++g) W.w[g] = t.st.u_w_g[g];
  hipLaunchKernelGGL(k_ttl_fin, dim3(1), dim3(64), 0, s, cnt, wsum, wd, ttl_dev, n_ttl, G, W,
                     hits, hitw, store);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

}  // namespace kv
