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
};

struct JobArgs {
  const uint32_t* bid[2];
  const uint8_t* w8[2];
  const uint8_t* g8[2];
  const uint8_t* blk_w;
  const uint8_t* blk_g;
  uint64_t u;           // distinct blocks
  uint32_t n_groups;
  uint32_t n_class;     // LFU classes per job (max multiplicity + 2)
};

// per-job counters: [job][group][4] = ins, ins_w, evict, evict_w

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

// FIFO, one wavefront per job.  Lanes load and gather a batch of 64 accesses;
// lane 0 resolves them in trace order, then writes back.
__device__ void replay_fifo(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ S,
                            uint64_t* __restrict__ bits, unsigned long long* cnt) {
  __shared__ uint32_t sb[64], sw[64], sg[64];
  __shared__ int sdup[64];
  __shared__ uint64_t ss[64], snew[64];
  __shared__ unsigned long long sins[KV_MAX_GROUPS], sinsw[KV_MAX_GROUPS];
  const uint32_t lane = threadIdx.x;
  const uint32_t o = j.order;
  const uint32_t* __restrict__ bid = a.bid[o];
  const uint8_t* __restrict__ w8 = a.w8[o];
  const uint8_t* __restrict__ g8 = a.g8[o];
  if (lane < KV_MAX_GROUPS) {
    sins[lane] = 0;
    sinsw[lane] = 0;
  }
  uint64_t wcur = 0;
  const uint64_t w0 = j.begin & ~63ull;
  for (uint64_t base = w0; base < j.end; base += 64) {
    const uint64_t i = base + lane;
    const bool in = i >= j.begin && i < j.end;
    const uint32_t b = in ? bid[i] : 0u;
    sb[lane] = b;
    sw[lane] = in ? w8[i] : 0u;
    sg[lane] = in ? g8[i] : 0u;
    ss[lane] = in ? S[b] : 0ull;
    __syncthreads();
    int dup = -1;
    if (in)
      for (int l = (int)lane - 1; l >= 0; --l)
        if (base + l >= j.begin && sb[l] == b) {
          dup = l;
          break;
        }
    sdup[lane] = dup;
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
          sins[sg[l]] += 1;
          sinsw[sg[l]] += sw[l];
        }
      }
      bits[(base >> 6) - j.word0] = word;
    }
    __threadfence_block();
    __syncthreads();
  }
  // residents at the end: insertions - residents = evictions
  __shared__ uint64_t swfin;
  if (lane == 0) swfin = wcur;
  __syncthreads();
  __shared__ unsigned long long sfin[KV_MAX_GROUPS], sfinw[KV_MAX_GROUPS];
  if (lane < KV_MAX_GROUPS) {
    sfin[lane] = 0;
    sfinw[lane] = 0;
  }
  __syncthreads();
  const uint64_t wf = swfin;
  for (uint64_t b = lane; b < a.u; b += 64) {
    const uint64_t s = S[b];
    if (s != kNoIns && wf - s <= j.cap) {
      const uint32_t g = a.blk_g[b];
      atomicAdd(&sfin[g], 1ull);
      atomicAdd(&sfinw[g], (unsigned long long)a.blk_w[b]);
    }
  }
  __syncthreads();
  if (lane < a.n_groups) {
    unsigned long long* c = cnt + (uint64_t)lane * 4;
    c[0] = sins[lane];
    c[1] = sinsw[lane];
    c[2] = sins[lane] - sfin[lane];
    c[3] = sinsw[lane] - sfinw[lane];
  }
}

__device__ __forceinline__ uint32_t next_class(const uint64_t* nz, uint32_t nw, uint32_t f) {
  uint32_t wi = f >> 6;
  if (wi >= nw) return 0xFFFFFFFFu;
  uint64_t m = nz[wi] & (~0ull << (f & 63));
  while (m == 0) {
    if (++wi >= nw) return 0xFFFFFFFFu;
    m = nz[wi];
  }
  return (wi << 6) + (uint32_t)__ffsll((long long)m) - 1u;
}

// LFU, one lane per job (each access depends on the previous one's evictions).
__device__ void replay_lfu(const JobDev& j, const JobArgs& a, uint64_t* __restrict__ st,
                           uint32_t* __restrict__ cls, uint64_t* __restrict__ bits,
                           unsigned long long* cnt) {
  __shared__ unsigned long long sins[KV_MAX_GROUPS], sinsw[KV_MAX_GROUPS], sev[KV_MAX_GROUPS],
      sevw[KV_MAX_GROUPS];
  __shared__ bool sbroken;
  const uint32_t lane = threadIdx.x;
  if (lane < KV_MAX_GROUPS) {
    sins[lane] = 0;
    sinsw[lane] = 0;
    sev[lane] = 0;
    sevw[lane] = 0;
  }
  if (lane == 0) sbroken = false;
  __syncthreads();
  if (lane == 0) {
    const uint32_t o = j.order;
    const uint32_t* __restrict__ bid = a.bid[o];
    const uint8_t* __restrict__ w8 = a.w8[o];
    const uint8_t* __restrict__ g8 = a.g8[o];
    uint32_t* head = cls + j.class_off;
    uint32_t* ccount = head + a.n_class;
    uint64_t* nz = reinterpret_cast<uint64_t*>(ccount + a.n_class);
    const uint32_t nw = (a.n_class + 63) / 64;
    uint64_t used = 0;
    uint32_t fmin = 1;
    uint64_t word = 0;
    bool broken = false;
    for (uint64_t i = j.begin; i < j.end && !broken; ++i) {
      const uint32_t b = bid[i];
      const uint32_t w = w8[i];
      const uint64_t s = st[b];
      const uint32_t f = (uint32_t)s;
      if (f) {
        word |= 1ull << (i & 63);
        const uint32_t f1 = f + 1;
        if (--ccount[f] == 0) nz[f >> 6] &= ~(1ull << (f & 63));
        if (ccount[f1]++ == 0) nz[f1 >> 6] |= 1ull << (f1 & 63);
        if (f == fmin && ccount[f] == 0) fmin = f1;
        st[b] = ((uint64_t)i << 32) | f1;
      } else {
        while (used + w > j.cap) {
          uint32_t q = head[fmin];
          uint32_t v = 0;
          // the oldest live member of class fmin lies before position i;
          // the bound only guards against corrupted state
          for (; q < i; ++q) {
            v = bid[q];
            const uint64_t sv = st[v];
            if ((uint32_t)sv == fmin && (uint32_t)(sv >> 32) == q) break;
          }
          if (q >= i) {
            broken = true;
            break;
          }
          head[fmin] = q + 1;
          st[v] = 0;
          const uint32_t vw = a.blk_w[v], vg = a.blk_g[v];
          used -= vw;
          sev[vg] += 1;
          sevw[vg] += vw;
          if (--ccount[fmin] == 0) {
            nz[fmin >> 6] &= ~(1ull << (fmin & 63));
            const uint32_t nf = next_class(nz, nw, fmin);
            if (nf != 0xFFFFFFFFu) fmin = nf;
          }
        }
        st[b] = ((uint64_t)i << 32) | 1u;
        if (ccount[1]++ == 0) nz[0] |= 2ull;
        fmin = 1;
        used += w;
        const uint32_t g = g8[i];
        sins[g] += 1;
        sinsw[g] += w;
      }
      if ((i & 63) == 63 || i + 1 == j.end) {
        bits[(i >> 6) - j.word0] = word;
        word = 0;
      }
    }
    sbroken = broken;
  }
  __syncthreads();
  if (lane < a.n_groups) {
    unsigned long long* c = cnt + (uint64_t)lane * 4;
    c[0] = sins[lane];
    c[1] = sinsw[lane];
    c[2] = sev[lane];
    c[3] = sevw[lane];
  }
  if (lane == 0 && sbroken) cnt[0] = ~0ull;  // poison: surfaced as an impossible count
}

__global__ __launch_bounds__(64) void k_replay(const JobDev* __restrict__ jobs, JobArgs a,
                                               uint64_t* __restrict__ state,
                                               uint32_t* __restrict__ cls,
                                               uint64_t* __restrict__ bits,
                                               unsigned long long* __restrict__ jcnt) {
  const JobDev j = jobs[blockIdx.x];
  if (j.closed) return;
  unsigned long long* cnt = jcnt + (uint64_t)blockIdx.x * a.n_groups * 4;
  if (j.policy == KV_POLICY_FIFO)
    replay_fifo(j, a, state + j.state_off, bits + j.bits_off, cnt);
  else
    replay_lfu(j, a, state + j.state_off, cls, bits + j.bits_off, cnt);
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
    hipLaunchKernelGGL(k_replay, dim3(nj), dim3(64), 0, s, bj.as<JobDev>(), ja,
                       bstate.as<uint64_t>(), bcls.as<uint32_t>(), bbits.as<uint64_t>(),
                       bjc.as<unsigned long long>());
    KV_HIP(hipGetLastError());
  }
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
