// k_eval.hip - per-configuration counts, objectives and the Pareto filter.
#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

// cumulative value of field f at capacity `cap` (0 for an absent tier)
__device__ __forceinline__ uint64_t cum_at(const OrderView& ov, uint32_t g, uint64_t cap, int f) {
  if (cap == 0) return 0;
  const uint32_t c = cap > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)cap;
  const uint32_t lo = ov.off[g], hi = ov.off[g + 1];
  const uint32_t m = lower_bound(ov.thr, lo, hi, c);
  return ov.hist[(uint64_t)(m + g) * 4 + f];
}

// LRU records from the stack-distance histograms.
//  inclusive: hit_k = hits(C_k) - hits(M) if C_k > M (M = largest faster
//             capacity), miss_k = N - hits(max(M, C_k)), ins_k = N - hits(C_k),
//             evict_k = ins_k - final residents at C_k.
//  exclusive (uniform weight w0): the tiers are one LRU stack cut at the
//             cumulative block capacities S_k; hit_k = hits(S_k) - hits(S_{k-1}),
//             miss_k = N - hits(S_k), evict_k = N - hits(S_k) - finals(S_k)
//             (a block crosses depth S_k once per reuse interval whose distance
//             exceeds S_k and once more if it ends deeper); ins of the top tier
//             = N - hit_top, of a lower tier = evictions of the tier above.
// Cumulative joint value of field f over accesses (or final blocks, `fin`)
// with stack distance <= cap (cap = ~0: any, cold accesses included) and gap
// <= the TTL value at index k of group g.
__device__ __forceinline__ uint64_t joint_at(const OrderView& ov, const JointView& jv,
                                             uint32_t g, uint64_t cap, uint32_t k, int f,
                                             bool fin) {
  if (cap == 0) return 0;
  const uint32_t lo = ov.off[g], hi = ov.off[g + 1];
  const uint32_t d = cap == ~0ull ? hi - lo
                                  : lower_bound(ov.thr, lo, hi,
                                                cap > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)cap) - lo;
  const uint32_t nt = jv.toff[g + 1] - jv.toff[g] + 1;
  const uint64_t b = jv.jbase[g] + (uint64_t)d * nt + k;
  return (fin ? jv.fh : jv.jh)[2 * b + f];
}

// Tier 2 as a disk TTL tier (trace order): present at an access iff its
// stack distance fits cap2 (unbounded: cap2 = ~0) and its gap fits the TTL;
// the faster tiers' largest capacity M decides which accesses reach it.
__device__ __forceinline__ void ttl_tier_record(const OrderView& ov, const JointView& jv,
                                                const kv_config& C, uint32_t g, uint64_t M,
                                                const GroupStats& s, uint64_t* r,
                                                double* store) {
  const double t = C.ttl[g];
  const uint32_t tlo = jv.toff[g], thi = jv.toff[g + 1];
  const uint32_t k = lower_bound(jv.tthr, tlo, thi, t) - tlo;
  const uint64_t c2 = C.cap[2] ? C.cap[2] : ~0ull;
  const uint64_t N = s.n_g, NW = s.n_w_g;
  const uint64_t pc = joint_at(ov, jv, g, c2, k, 0, false), pw = joint_at(ov, jv, g, c2, k, 1, false);
  const uint64_t lo_cap = (M == 0) ? 0 : (M < c2 ? M : c2);
  const uint64_t mc = joint_at(ov, jv, g, lo_cap, k, 0, false);
  const uint64_t mw = joint_at(ov, jv, g, lo_cap, k, 1, false);
  const uint64_t hc = pc - mc, hw = pw - mw;
  const uint64_t rc = N - cum_at(ov, g, M, 0), rw = NW - cum_at(ov, g, M, 1);  // reach the disk
  r[KV_F_HIT] = hc;
  r[KV_F_HIT_W] = hw;
  r[KV_F_MISS] = rc - hc;
  r[KV_F_MISS_W] = rw - hw;
  r[KV_F_INS] = N - pc;
  r[KV_F_INS_W] = NW - pw;
  r[KV_F_EVICT] = (N - pc) - joint_at(ov, jv, g, c2, k, 0, true);
  r[KV_F_EVICT_W] = (NW - pw) - joint_at(ov, jv, g, c2, k, 1, true);
  if (C.cap[2] == 0) {
    // W_g t + sum over gaps <= t of w gap + t (weight of the longer gaps)
    const double sd = jv.wd[tlo + g + k];
    const uint64_t gapw = NW - s.u_w_g;               // re-accesses
    const uint64_t inw = joint_at(ov, jv, g, ~0ull, k, 1, false);  // re-accesses within t
    *store = ((double)s.u_w_g * t + sd) + t * (double)(gapw - inw);
  }
}

__global__ __launch_bounds__(256) void k_lru_counts(const kv_config* __restrict__ cfg,
                                                    uint32_t n_cfg, uint32_t G, OrderView sh,
                                                    OrderView pt, OrderView px, OrderView lf,
                                                    JointView jv,
                                                    const GroupStats* __restrict__ gs,
                                                    uint32_t mixed,
                                                    uint64_t* __restrict__ counts,
                                                    double* __restrict__ store_cg) {
  const uint64_t tid = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= (uint64_t)n_cfg * G) return;
  const uint32_t c = (uint32_t)(tid / G), g = (uint32_t)(tid % G);
  const kv_config& C = cfg[c];
  const bool part = C.partitioned != 0;
  const uint32_t pol = part ? C.policy[g] : C.policy[0];
  if (pol != KV_POLICY_LRU && pol != KV_POLICY_LEAF) return;
  // an exclusive hierarchy over mixed weights is no split stack: replayed
  if (C.mode == KV_MODE_EXCLUSIVE_DEMOTE && mixed) return;
  // radix-tree eviction: distances of the re-touched order (shared tiers only)
  const OrderView& ov = pol == KV_POLICY_LEAF ? lf : (part && G > 1) ? pt : sh;
  uint64_t cap[3];
  for (int k = 0; k < 3; ++k) cap[k] = part ? C.cap_group[k][g] : C.cap[k];
  const uint64_t N = gs[g].n_g, NW = gs[g].n_w_g;
  uint64_t* out = counts + ((uint64_t)c * G + g) * 3 * 8;
  if (store_cg) store_cg[(uint64_t)c * G + g] = 0.0;
  if (C.disk_ttl) {
    uint64_t M = 0;
    for (int k = 0; k < 2; ++k) {
      uint64_t* r = out + k * 8;
      if (cap[k] == 0) {
        for (int f = 0; f < 8; ++f) r[f] = 0;
        continue;
      }
      const uint64_t Mx = cap[k] > M ? cap[k] : M;
      const uint64_t hC = cum_at(ov, g, cap[k], 0), wC = cum_at(ov, g, cap[k], 1);
      const uint64_t hM = cum_at(ov, g, M, 0), wM = cum_at(ov, g, M, 1);
      const uint64_t hX = cum_at(ov, g, Mx, 0), wX = cum_at(ov, g, Mx, 1);
      r[KV_F_HIT] = cap[k] > M ? hC - hM : 0;
      r[KV_F_HIT_W] = cap[k] > M ? wC - wM : 0;
      r[KV_F_MISS] = N - hX;
      r[KV_F_MISS_W] = NW - wX;
      r[KV_F_INS] = N - hC;
      r[KV_F_INS_W] = NW - wC;
      r[KV_F_EVICT] = (N - hC) - cum_at(ov, g, cap[k], 2);
      r[KV_F_EVICT_W] = (NW - wC) - cum_at(ov, g, cap[k], 3);
      M = Mx;
    }
    double st = 0.0;
    ttl_tier_record(ov, jv, C, g, M, gs[g], out + 2 * 8, &st);
    if (store_cg) store_cg[(uint64_t)c * G + g] = st;
    return;
  }
  if (C.mode == KV_MODE_INCLUSIVE || C.mode == KV_MODE_INCLUSIVE_PREFIX) {
    // which accesses a tier serves: by stack distance, or with prefix reuse
    // by the running maximum over the request; what it holds: by distance
    const OrderView& sv = C.mode == KV_MODE_INCLUSIVE_PREFIX ? px : ov;
    uint64_t M = 0;
    for (int k = 0; k < 3; ++k) {
      uint64_t* r = out + k * 8;
      if (cap[k] == 0) {
        for (int f = 0; f < 8; ++f) r[f] = 0;
        continue;
      }
      const uint64_t Mx = cap[k] > M ? cap[k] : M;
      const uint64_t hC = cum_at(ov, g, cap[k], 0), wC = cum_at(ov, g, cap[k], 1);
      const uint64_t sC = cum_at(sv, g, cap[k], 0), swC = cum_at(sv, g, cap[k], 1);
      const uint64_t sM = cum_at(sv, g, M, 0), swM = cum_at(sv, g, M, 1);
      const uint64_t sX = cum_at(sv, g, Mx, 0), swX = cum_at(sv, g, Mx, 1);
      const uint64_t fC = cum_at(ov, g, cap[k], 2), fwC = cum_at(ov, g, cap[k], 3);
      r[KV_F_HIT] = cap[k] > M ? sC - sM : 0;
      r[KV_F_HIT_W] = cap[k] > M ? swC - swM : 0;
      r[KV_F_MISS] = N - sX;
      r[KV_F_MISS_W] = NW - swX;
      r[KV_F_INS] = N - hC;
      r[KV_F_INS_W] = NW - wC;
      r[KV_F_EVICT] = (N - hC) - fC;
      r[KV_F_EVICT_W] = (NW - wC) - fwC;
      M = Mx;
    }
  } else {
    const uint64_t w0 = gs[g].w0;
    uint64_t S = 0, prev_ev = 0;
    bool top = true;
    for (int k = 0; k < 3; ++k) {
      uint64_t* r = out + k * 8;
      if (cap[k] == 0) {
        for (int f = 0; f < 8; ++f) r[f] = 0;
        continue;
      }
      const uint64_t Sp = S;
      S += cap[k] / w0;
      const uint64_t hS = cum_at(ov, g, S * w0, 0);
      const uint64_t hP = cum_at(ov, g, Sp * w0, 0);
      const uint64_t fS = cum_at(ov, g, S * w0, 2);
      const uint64_t hit = hS - hP;
      const uint64_t miss = N - hS;
      const uint64_t ev = N - hS - fS;
      const uint64_t ins = top ? N - hit : prev_ev;
      r[KV_F_HIT] = hit;
      r[KV_F_MISS] = miss;
      r[KV_F_INS] = ins;
      r[KV_F_EVICT] = ev;
      r[KV_F_HIT_W] = hit * w0;
      r[KV_F_MISS_W] = miss * w0;
      r[KV_F_INS_W] = ins * w0;
      r[KV_F_EVICT_W] = ev * w0;
      prev_ev = ev;
      top = false;
    }
  }
}

struct CostArgs {
  double pg, p0, p1, p2, bw_dram, ssd_base, ssd_per_gib, ssd_max, tpf;
  double gb, tpg, span, n_req;
  uint64_t n_w;
  uint32_t n_media;
  kv_disk_medium media[KV_MAX_MEDIA];
};

// (cost, throughput, latency) in IEEE double, left to right, no contraction.
__global__ __launch_bounds__(256) void k_objectives(const kv_config* __restrict__ cfg,
                                                    uint32_t n_cfg, uint32_t G,
                                                    const uint64_t* __restrict__ counts,
                                                    const double* __restrict__ store_cg,
                                                    CostArgs a, double* __restrict__ obj) {
  const uint32_t c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n_cfg) return;
  uint64_t hw0 = 0, hw1 = 0, hw2 = 0, iw2 = 0;
  for (uint32_t g = 0; g < G; ++g) {
    const uint64_t* r = counts + ((uint64_t)c * G + g) * 24;
    hw0 += r[0 * 8 + KV_F_HIT_W];
    hw1 += r[1 * 8 + KV_F_HIT_W];
    hw2 += r[2 * 8 + KV_F_HIT_W];
    iw2 += r[2 * 8 + KV_F_INS_W];
  }
  const uint64_t rw = a.n_w - (hw0 + hw1 + hw2);
  const double kGiB = 1073741824.0;
  const double c0 = ((double)cfg[c].cap[0] * a.gb) / kGiB;
  const double c1 = ((double)cfg[c].cap[1] * a.gb) / kGiB;
  double c2 = ((double)cfg[c].cap[2] * a.gb) / kGiB;
  if (cfg[c].disk_ttl && cfg[c].cap[2] == 0) {
    // an unbounded TTL tier: its mean occupancy over the span
    double st = 0.0;
    for (uint32_t g = 0; g < G; ++g) st += store_cg[(uint64_t)c * G + g];
    c2 = a.span > 0 ? ((st * a.gb) / kGiB) / a.span : 0.0;
  }
  double p2 = a.p2, base = a.ssd_base, per_gib = a.ssd_per_gib, bmax = a.ssd_max;
  if (a.n_media) {
    const kv_disk_medium& md = a.media[cfg[c].medium];
    p2 = md.price_per_gib_hour;
    base = md.bw_base;
    per_gib = md.bw_per_gib;
    bmax = md.bw_max;
  }
  const double bw_lin = base + per_gib * c2;
  const double bw_ssd = (bmax < bw_lin) ? bmax : bw_lin;
  const double t_dram = ((double)hw1 * a.gb) / a.bw_dram;
  const double t_ssd = ((double)(hw2 + iw2) * a.gb) / bw_ssd;
  const double t_rec = ((double)rw * a.tpg) * a.tpf;
  const double t_busy = (t_rec + t_dram) + t_ssd;
  const double t_wall = (a.span < t_busy) ? t_busy : a.span;
  const double thr = ((double)a.n_w * a.tpg) / t_wall;
  const double lat = t_busy / a.n_req;
  const double cost = (((a.pg + c0 * a.p0) + c1 * a.p1) + c2 * p2) * (t_wall / 3600.0);
  obj[3 * (uint64_t)c + 0] = cost;
  obj[3 * (uint64_t)c + 1] = thr;
  obj[3 * (uint64_t)c + 2] = lat;
}

struct Bounds {
  double b0, b1, b2;
};

__device__ __forceinline__ bool feasible(double o0, double o1, double o2, const Bounds& b) {
  if (o0 != o0 || o1 != o1 || o2 != o2) return false;
  if (b.b0 == b.b0 && !(o0 <= b.b0)) return false;
  if (b.b1 == b.b1 && !(o1 >= b.b1)) return false;
  if (b.b2 == b.b2 && !(o2 <= b.b2)) return false;
  return true;
}

// Flag of every point: 1 if it meets the bounds (and has no NaN), else 0;
// the NaN flag of the call.
__global__ __launch_bounds__(256) void k_pareto_init(const double* __restrict__ obj, uint32_t n,
                                                     Bounds bd, uint8_t* __restrict__ flag,
                                                     uint32_t* __restrict__ counters) {
  const uint32_t b = blockIdx.x * 256 + threadIdx.x;
  if (b >= n) return;
  const double o0 = obj[3 * (uint64_t)b], o1 = obj[3 * (uint64_t)b + 1],
               o2 = obj[3 * (uint64_t)b + 2];
  flag[b] = feasible(o0, o1, o2, bd) ? 1 : 0;
  if (o0 != o0 || o1 != o1 || o2 != o2) atomicOr(&counters[1], 1u);
}

// All-pairs dominance over a grid of (points, candidates) tiles: block
// (x, y) tests points [256 x, 256 x + 256) against the feasible candidates
// of its slice [y * per, (y + 1) * per), staged through LDS 256 at a time,
// and clears the flag of every point a candidate of its segment dominates.
// Every writer stores 0, so the blocks need no ordering; the result is the
// same whichever candidates a block sees as still flagged, as dominance is
// transitive (only the objectives and the bounds decide a candidate).
__global__ __launch_bounds__(256) void k_pareto(const double* __restrict__ obj,
                                                const uint32_t* __restrict__ seg, uint32_t n,
                                                uint32_t per, Bounds bd, uint8_t* __restrict__ flag) {
  __shared__ double so[3][256];
  __shared__ uint32_t ss[256];
  __shared__ uint32_t sf[256];
  const uint32_t b = blockIdx.x * 256 + threadIdx.x;
  double ob0 = 0, ob1 = 0, ob2 = 0;
  uint32_t sb = 0;
  bool live = false;
  if (b < n && flag[b]) {
    ob0 = obj[3 * (uint64_t)b];
    ob1 = obj[3 * (uint64_t)b + 1];
    ob2 = obj[3 * (uint64_t)b + 2];
    sb = seg ? seg[b] : 0u;
    live = true;
  }
  const uint32_t c0 = blockIdx.y * per, c1 = min(n, c0 + per);
  bool dom = false;
  for (uint32_t a0 = c0; a0 < c1; a0 += 256) {
    const uint32_t a = a0 + threadIdx.x;
    if (a < c1) {
      const double x0 = obj[3 * (uint64_t)a], x1 = obj[3 * (uint64_t)a + 1],
                   x2 = obj[3 * (uint64_t)a + 2];
      so[0][threadIdx.x] = x0;
      so[1][threadIdx.x] = x1;
      so[2][threadIdx.x] = x2;
      ss[threadIdx.x] = seg ? seg[a] : 0u;
      sf[threadIdx.x] = feasible(x0, x1, x2, bd) ? 1u : 0u;
    }
    __syncthreads();
    const uint32_t m = min(256u, c1 - a0);
    if (live && !dom) {
      for (uint32_t j = 0; j < m; ++j) {
        if (a0 + j == b || !sf[j] || ss[j] != sb) continue;
        const double x0 = so[0][j], x1 = so[1][j], x2 = so[2][j];
        const bool le = x0 <= ob0 && x1 >= ob1 && x2 <= ob2;
        const bool lt = x0 < ob0 || x1 > ob1 || x2 < ob2;
        if (le && lt) {
          dom = true;
          break;
        }
      }
    }
    __syncthreads();
  }
  if (dom) flag[b] = 0;
}

// Points left on the front.
__global__ __launch_bounds__(256) void k_pareto_count(const uint8_t* __restrict__ flag, uint32_t n,
                                                      uint32_t* __restrict__ counters) {
  const uint32_t b = blockIdx.x * 256 + threadIdx.x;
  const uint64_t on = __ballot(b < n && flag[b]);
  if ((threadIdx.x & 63) == 0 && on) atomicAdd(&counters[0], (uint32_t)__popcll(on));
}

}  // namespace

kv_status lru_counts(const kv_config* cfg_dev, uint32_t n_cfg, uint32_t n_groups,
                     OrderView shared, OrderView part, OrderView prefix, OrderView leaf,
                     JointView joint,
                     const GroupStats* gs_dev, bool mixed, uint64_t* counts, double* store_cg,
                     hipStream_t s) {
  const uint64_t m = (uint64_t)n_cfg * n_groups;
  if (m == 0) return KV_OK;
  StageTimer tm(kStLruCounts, s);
  hipLaunchKernelGGL(k_lru_counts, dim3(div_up(m, 256)), dim3(256), 0, s, cfg_dev, n_cfg,
                     n_groups, shared, part, prefix, leaf, joint, gs_dev, mixed ? 1u : 0u, counts,
                     store_cg);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

kv_status objectives(const kv_config* cfg_dev, uint32_t n_cfg, uint32_t n_groups,
                     const uint64_t* counts, const double* store_cg, const kv_cost_model& m,
                     double gb, double tpg, double span, double n_req, uint64_t n_w,
                     double* obj, hipStream_t s) {
  if (n_cfg == 0) return KV_OK;
  CostArgs a{m.price_gpu_per_hour, m.price_per_gib_hour[0], m.price_per_gib_hour[1],
             m.price_per_gib_hour[2], m.bw_dram, m.ssd_bw_base, m.ssd_bw_per_gib,
             m.ssd_bw_max, m.t_prefill_per_token, gb, tpg, span, n_req, n_w, m.n_media, {}};
  for (uint32_t i = 0; i < KV_MAX_MEDIA; ++i) a.media[i] = m.media[i];
  StageTimer tm(kStObjectives, s);
  hipLaunchKernelGGL(k_objectives, dim3(div_up(n_cfg, 256)), dim3(256), 0, s, cfg_dev, n_cfg,
                     n_groups, counts, store_cg, a, obj);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

kv_status pareto(const double* obj, const uint32_t* segment, uint32_t n, const double* bounds,
                 uint8_t* flag, uint32_t* counters_dev, hipStream_t s) {
  const double nan = __builtin_nan("");
  Bounds bd{bounds ? bounds[0] : nan, bounds ? bounds[1] : nan, bounds ? bounds[2] : nan};
  StageTimer tm(kStPareto, s);
  if (n == 0) return KV_OK;
  // point tiles x candidate slices: about 2,048 blocks, slices of whole tiles
  const uint32_t nt = div_up(n, 256);
  const uint32_t ny = std::max<uint32_t>(1, std::min<uint32_t>(nt, div_up(2048, nt)));
  const uint32_t per = div_up(nt, ny) * 256;
  hipLaunchKernelGGL(k_pareto_init, dim3(nt), dim3(256), 0, s, obj, n, bd, flag, counters_dev);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_pareto, dim3(nt, div_up(n, per)), dim3(256), 0, s, obj, segment, n, per,
                     bd, flag);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_pareto_count, dim3(nt), dim3(256), 0, s, flag, n, counters_dev);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

}  // namespace kv
