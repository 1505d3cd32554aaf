// k_leaf.hip - radix-tree (leaf-first) eviction as a stack algorithm.
//
// A radix KV cache shares blocks through a prefix tree (Section 3.2): the
// blocks of a request form a chain and the cache evicts the least recently
// used leaf.  When requests are prefix chains (a block always follows the
// same parent) and every request fits the cache, the cached set stays
// closed under parents, and the least recently used leaf is the block that
// ranks lowest by (request of its latest access, then deeper first): a
// block's latest request is never older than any of its cached
// descendants', and within that request its descendants come after it.
// That ranking is a priority independent of the capacity, so the policy has
// Mattson's inclusion property, and its stack distances are the LRU stack
// distances of the trace with every request followed by a re-touch of its
// blocks from the deepest to the first (the re-touches leave the request's
// blocks ordered shallowest first on top of the stack; they are not
// accesses and are not counted).  This file checks the trace, measures the
// heaviest request and builds that order; the stack pass then bins the
// trace's own positions only.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

uint32_t grid_for_n(uint64_t m, uint32_t cap = 32768) {
  uint64_t g = (m + 255) / 256;
  if (g > cap) g = cap;
  return (uint32_t)(g ? g : 1);
}

// First position of every request r <= n_req (an empty request starts where
// the next one does).
__global__ __launch_bounds__(256) void k_leaf_rstart(const uint32_t* __restrict__ req, uint64_t n,
                                                     uint32_t n_req, uint32_t* __restrict__ rs) {
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p <= n;
       p += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t lo = p == 0 ? 0u : req[p - 1] + 1u;
    const uint32_t hi = p == n ? n_req : req[p];
    for (uint32_t r = lo; r <= hi && r <= n_req; ++r) rs[r] = (uint32_t)p;
  }
}

// Chains: a re-accessed block's previous access lies in an earlier request
// and has the same parent (the block accessed just before, in the same
// request; none for a request's first block).  Request weights.
__global__ __launch_bounds__(256) void k_leaf_check(const uint32_t* __restrict__ key,
                                                    const uint32_t* __restrict__ bid,
                                                    const uint32_t* __restrict__ req,
                                                    const uint8_t* __restrict__ w8, uint64_t n,
                                                    uint32_t* __restrict__ reqw,
                                                    uint32_t* __restrict__ flag) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t r = req[i];
    atomicAdd(&reqw[r], (uint32_t)w8[i]);
    const uint32_t k = key[i];
    if (!k) continue;
    const uint32_t p = k - 1;
    const uint32_t rp = req[p];
    const uint32_t par_i = (i > 0 && req[i - 1] == r) ? bid[i - 1] : kNone;
    const uint32_t par_p = (p > 0 && req[p - 1] == rp) ? bid[p - 1] : kNone;
    if (rp >= r || par_i != par_p) atomicOr(flag, 1u);
  }
}

__global__ __launch_bounds__(256) void k_leaf_max(const uint32_t* __restrict__ reqw, uint32_t m,
                                                  uint32_t* __restrict__ out) {
  uint32_t x = 0;
  for (uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; r < m;
       r += (uint64_t)gridDim.x * blockDim.x)
    x = max(x, reqw[r]);
  for (int d = 32; d > 0; d >>= 1) x = max(x, (uint32_t)__shfl_down((int)x, d, 64));
  if ((threadIdx.x & 63) == 0 && x) atomicMax(out, x);
}

// Position of access x in the re-touched order: request r = [s, e) becomes
// [2s, 2e): its accesses at 2s .. 2s + (e - s) - 1, then its re-touches,
// deepest first.
__device__ __forceinline__ uint32_t aug_real(uint32_t x, uint32_t s) { return s + x; }
__device__ __forceinline__ uint32_t aug_retouch(uint32_t x, uint32_t s, uint32_t e) {
  return s + 2 * e - 1 - x;
}

__global__ __launch_bounds__(256) void k_leaf_build(const uint32_t* __restrict__ key,
                                                    const uint32_t* __restrict__ nxt,
                                                    const uint32_t* __restrict__ bid,
                                                    const uint8_t* __restrict__ w8,
                                                    const uint8_t* __restrict__ g8,
                                                    const uint32_t* __restrict__ req,
                                                    const uint32_t* __restrict__ rs, uint64_t n,
                                                    uint32_t* __restrict__ akey,
                                                    uint32_t* __restrict__ anxt,
                                                    uint32_t* __restrict__ abid,
                                                    uint8_t* __restrict__ aw,
                                                    uint8_t* __restrict__ ag,
                                                    uint8_t* __restrict__ real) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t x = (uint32_t)i;
    const uint32_t r = req[x];
    const uint32_t s = rs[r], e = rs[r + 1];
    const uint32_t a = aug_real(x, s), v = aug_retouch(x, s, e);
    const uint32_t k = key[x], nx = nxt[x];
    uint32_t pk = 0;  // the previous access's re-touch, + 1
    if (k) {
      const uint32_t p = k - 1, rp = req[p];
      pk = aug_retouch(p, rs[rp], rs[rp + 1]) + 1;
    }
    uint32_t an = kNone;  // the next access, in the new order
    if (nx != kNone) an = aug_real(nx, rs[req[nx]]);
    akey[a] = pk;
    anxt[a] = v;
    akey[v] = a + 1;
    anxt[v] = an;
    abid[a] = abid[v] = bid[x];
    aw[a] = aw[v] = w8[x];
    ag[a] = ag[v] = g8[x];
    real[a] = 1;
    real[v] = 0;
  }
}

}  // namespace

kv_status leaf_prepare(Trace& t, hipStream_t s) {
  if (t.leaf_checked) return KV_OK;
  const uint64_t n = t.n;
  const uint32_t nr = t.st.n_req;
  kv_status st;
  DevBuf rs, reqw, flag;
  if ((st = rs.reserve(((uint64_t)nr + 1) * 4)) != KV_OK) return st;
  if ((st = reqw.reserve((uint64_t)nr * 4)) != KV_OK) return st;
  if ((st = flag.reserve(8)) != KV_OK) return st;
  if ((st = fill_u32(reqw.as<uint32_t>(), 0, nr, s)) != KV_OK) return st;
  if ((st = fill_u32(flag.as<uint32_t>(), 0, 2, s)) != KV_OK) return st;
  const Order& o = t.shared;
  hipLaunchKernelGGL(k_leaf_rstart, dim3(grid_for_n(n + 1)), dim3(256), 0, s,
                     t.req.as<uint32_t>(), n, nr, rs.as<uint32_t>());
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_leaf_check, dim3(grid_for_n(n)), dim3(256), 0, s, o.key.as<uint32_t>(),
                     o.bid.as<uint32_t>(), t.req.as<uint32_t>(), o.w.as<uint8_t>(), n,
                     reqw.as<uint32_t>(), flag.as<uint32_t>());
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_leaf_max, dim3(grid_for_n(nr, 1024)), dim3(256), 0, s,
                     (const uint32_t*)reqw.as<uint32_t>(), nr, flag.as<uint32_t>() + 1);
  KV_HIP(hipGetLastError());
  uint32_t h[2] = {0, 0};
  KV_HIP(hipMemcpyAsync(h, flag.p, sizeof(h), hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  t.leaf_chained = h[0] == 0;
  t.max_req_w = h[1];
  if (t.leaf_chained) {
    Order& a = t.leaf;
    const uint64_t m = 2 * n;
    if ((st = a.key.reserve(m * 4)) != KV_OK) return st;
    if ((st = a.nxt.reserve(m * 4)) != KV_OK) return st;
    if ((st = a.bid.reserve(m * 4)) != KV_OK) return st;
    if ((st = a.w.reserve(m)) != KV_OK) return st;
    if ((st = a.g.reserve(m)) != KV_OK) return st;
    if ((st = t.leaf_real.reserve(m)) != KV_OK) return st;
    hipLaunchKernelGGL(k_leaf_build, dim3(grid_for_n(n)), dim3(256), 0, s, o.key.as<uint32_t>(),
                       o.nxt.as<uint32_t>(), o.bid.as<uint32_t>(), o.w.as<uint8_t>(),
                       o.g.as<uint8_t>(), t.req.as<uint32_t>(), (const uint32_t*)rs.as<uint32_t>(),
                       n, a.key.as<uint32_t>(), a.nxt.as<uint32_t>(), a.bid.as<uint32_t>(),
                       a.w.as<uint8_t>(), a.g.as<uint8_t>(), t.leaf_real.as<uint8_t>());
    KV_HIP(hipGetLastError());
    KV_HIP(hipStreamSynchronize(s));  // the temporaries are released on return
    a.n = m;
    a.seg[0] = 0;
    for (int g = 1; g <= KV_MAX_GROUPS; ++g) a.seg[g] = m;
    a.built = true;
  }
  t.leaf_checked = true;
  return KV_OK;
}

}  // namespace kv
