// kv_api.cpp - the C ABI of libkvcfg: validation, planning and launch order.
//
// kv_trace_load canonicalises a trace once; kv_eval_configs then evaluates a
// batch of candidate tier configurations (the planner's candidates and the
// simulator's per-candidate evaluation, Section 4.1):
//   1. host: validate, then collect the capacities the LRU configurations
//      need, per access order and group (the thresholds of the stack pass);
//   2. device: one stack-distance pass per needed order (k_stack.hip) and the
//      closed-form LRU records (k_eval.hip);
//   3. device: one replay per distinct (order, group, policy, capacity) for
//      FIFO / LFU tiers, combined per configuration (k_replay.hip);
//   4. device: (cost, throughput, latency) per configuration (Eq. 1, Eq. 2).
// kv_pareto is the selector's dominance filter (Section 4.1).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <tuple>

#include "kv_internal.h"

namespace kv {

namespace {
thread_local std::string g_last_error;
std::mutex g_reg_mu;
std::set<const void*> g_live;  // live trace handles
std::atomic<uint64_t> g_bytes{0};

uint64_t mem_cap() {
  // Test hook: cap the bytes this library may hold on the device, so that
  // the out-of-memory path can be exercised without exhausting the GPU.
  static const uint64_t cap = [] {
    const char* e = std::getenv("KVCFG_TEST_MEM_CAP");
    return e ? std::strtoull(e, nullptr, 10) : 0ull;
  }();
  return cap;
}

bool is_live(const void* t) {
  std::lock_guard<std::mutex> lk(g_reg_mu);
  return g_live.count(t) != 0;
}

// stage timing: recorded event pairs, resolved in kv_timing_read
std::mutex g_tmu;
bool g_timing = false;
struct EvPair {
  int stage;
  hipEvent_t a, b;
};
std::vector<EvPair> g_pairs;
std::vector<hipEvent_t> g_free_events;
kv_timing g_acc{};

hipEvent_t take_event() {
  if (!g_free_events.empty()) {
    hipEvent_t e = g_free_events.back();
    g_free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

StageTimer::StageTimer(Stage st, hipStream_t stream) : slot(-1), s(stream) {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!g_timing) return;
  hipEvent_t a = take_event(), b = take_event();
  if (!a || !b) return;
  if (hipEventRecord(a, s) != hipSuccess) return;
  g_pairs.push_back(EvPair{(int)st, a, b});
  slot = (int)g_pairs.size() - 1;
}

StageTimer::~StageTimer() {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (slot >= 0 && slot < (int)g_pairs.size()) (void)hipEventRecord(g_pairs[slot].b, s);
}

kv_status fail(kv_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

kv_status hip_fail(hipError_t e, const char* what) {
  if (e == hipErrorOutOfMemory) return fail(KV_ERR_NOMEM, std::string("out of device memory: ") + what);
  return fail(KV_ERR_DEVICE, std::string(hipGetErrorString(e)) + " in " + what);
}

// Device blocks released by DevBufs are kept per device and handed out
// again (a trace's workspaces reach ~100 GiB at full scale; allocating and
// freeing that much for every trace fragments the device's memory and slows
// the random-access kernels that follow).  A failed hipMalloc empties the
// device's cache and tries once more; the cache keeps at most half of the
// device's memory, so that other users of the device are not starved.
namespace {
std::mutex g_pool_mu;
std::multimap<size_t, void*> g_pool[64];  // per device: block size -> block
size_t g_pool_bytes[64] = {};
size_t g_pool_limit[64] = {};

size_t block_size(size_t b) {
  // 256 bytes of slack past the end: kernels may issue (and then discard)
  // vector loads of up to 16 bytes at the last valid index
  const size_t need = b + 256;
  const size_t g = need >= (1u << 20) ? (2u << 20) : 4096;
  return (need + g - 1) / g * g;
}

void pool_flush(int dev) {
  for (auto& kv : g_pool[dev]) (void)hipFree(kv.second);
  g_pool[dev].clear();
  g_pool_bytes[dev] = 0;
}
}  // namespace

kv_status DevBuf::reserve(size_t b) {
  if (b <= bytes && p) return KV_OK;
  release();
  if (b == 0) b = 1;
  const uint64_t cap = mem_cap();
  if (cap && g_bytes.load() + b > cap)
    return fail(KV_ERR_NOMEM, "device memory cap reached (test limit)");
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess || d < 0 || d >= 64) {
    (void)hipGetLastError();
    return fail(KV_ERR_DEVICE, "no current device");
  }
  const size_t sz = block_size(b);
  void* q = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    // a cached block of at least sz and at most twice that
    auto it = g_pool[d].lower_bound(sz);
    if (it != g_pool[d].end() && it->first <= 2 * sz) {
      q = it->second;
      p = q;
      bytes = b;
      cap_bytes = it->first;
      g_pool_bytes[d] -= it->first;
      g_pool[d].erase(it);
    }
  }
  if (!q) {
    hipError_t e = hipMalloc(&q, sz);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      {
        std::lock_guard<std::mutex> lk(g_pool_mu);
        pool_flush(d);
      }
      e = hipMalloc(&q, sz);
      if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(KV_ERR_NOMEM, "hipMalloc of " + std::to_string(b) + " bytes failed");
      }
    }
    p = q;
    bytes = b;
    cap_bytes = sz;
  }
  dev = d;
  g_bytes += b;
  return KV_OK;
}

void DevBuf::release() {
  if (p) {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    if (!g_pool_limit[dev]) {
      size_t fr = 0, tot = 0;
      int cur = 0;
      if (hipGetDevice(&cur) == hipSuccess && cur == dev && hipMemGetInfo(&fr, &tot) == hipSuccess)
        g_pool_limit[dev] = tot / 2;
      (void)hipGetLastError();
    }
    if (g_pool_bytes[dev] + cap_bytes <= g_pool_limit[dev]) {
      g_pool[dev].emplace(cap_bytes, p);
      g_pool_bytes[dev] += cap_bytes;
    } else {
      (void)hipFree(p);
    }
    g_bytes -= bytes;
  }
  p = nullptr;
  bytes = 0;
}

Trace::~Trace() {
  if (err_ev) (void)hipEventDestroy(err_ev);
  if (err_host) (void)hipHostFree(err_host);
}

kv_status check_device_error(Trace& t, bool wait, const char* who) {
  if (!t.err_pending) return KV_OK;
  if (wait) {
    KV_HIP(hipEventSynchronize(t.err_ev));
  } else {
    const hipError_t q = hipEventQuery(t.err_ev);
    if (q == hipErrorNotReady) return KV_OK;  // that call is still running
    if (q != hipSuccess) return hip_fail(q, "hipEventQuery");
  }
  t.err_pending = false;
  const uint32_t code = t.err_host[0], job = t.err_host[1];
  if (code == 0) return KV_OK;
  t.err_host[0] = t.err_host[1] = 0;
  KV_HIP(hipMemset(t.err.p, 0, 2 * sizeof(uint32_t)));
  std::string what = "replay job " + std::to_string(job);
  if (code == 2) {
    what = "the exclusive hierarchy of configuration " + std::to_string(job);
  } else if (job < t.err_jobs.size()) {
    const ReplayJobInfo& j = t.err_jobs[job];
    what += std::string(" (") + (j.policy == KV_POLICY_LFU ? "LFU" : "FIFO") + ", capacity " +
            std::to_string(j.cap) + " granules, " +
            (j.group == KV_MAX_GROUPS ? std::string("shared") : "group " + std::to_string(j.group)) +
            ")";
  }
  return fail(KV_ERR_DEVICE, std::string(who) + ": an earlier kv_eval_configs call on this trace "
              "returned invalid counts: " + what + " failed its internal state check");
}

namespace {

bool finite_pos(double x) { return std::isfinite(x) && x > 0; }
bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0; }

kv_status validate_model(const kv_cost_model* m) {
  if (!m) return fail(KV_ERR_INVALID, "kv_eval_configs: model is NULL");
  if (!finite_nonneg(m->price_gpu_per_hour) || !finite_nonneg(m->price_per_gib_hour[0]) ||
      !finite_nonneg(m->price_per_gib_hour[1]) || !finite_nonneg(m->price_per_gib_hour[2]))
    return fail(KV_ERR_INVALID, "kv_eval_configs: prices must be finite and >= 0");
  if (!finite_pos(m->bw_dram) || !finite_pos(m->ssd_bw_base) || !finite_pos(m->ssd_bw_max) ||
      !finite_nonneg(m->ssd_bw_per_gib) || !finite_pos(m->t_prefill_per_token))
    return fail(KV_ERR_INVALID, "kv_eval_configs: bandwidths and t_prefill must be finite and > 0");
  if (m->n_media > KV_MAX_MEDIA || m->reserved)
    return fail(KV_ERR_INVALID, "kv_eval_configs: n_media must be <= 4 and reserved 0");
  for (uint32_t i = 0; i < m->n_media; ++i) {
    const kv_disk_medium& d = m->media[i];
    if (!finite_nonneg(d.price_per_gib_hour) || !finite_pos(d.bw_base) ||
        !finite_nonneg(d.bw_per_gib) || !finite_pos(d.bw_max))
      return fail(KV_ERR_INVALID, "kv_eval_configs: a disk medium has a bad price or bandwidth");
  }
  return KV_OK;
}

uint32_t group_policy(const kv_config& c, uint32_t g) {
  return c.partitioned ? c.policy[g] : c.policy[0];
}

uint64_t group_cap(const kv_config& c, int k, uint32_t g) {
  return c.partitioned ? c.cap_group[k][g] : c.cap[k];
}

kv_status validate_configs(const Trace& t, const kv_config* cfg, uint32_t n_cfg,
                           uint32_t n_media) {
  const uint32_t G = t.n_groups;
  const uint64_t wmax = t.st.w_max;
  for (uint32_t c = 0; c < n_cfg; ++c) {
    const kv_config& C = cfg[c];
    const std::string at = "kv_eval_configs: config " + std::to_string(c) + ": ";
    if (C.mode > KV_MODE_INCLUSIVE_PREFIX) return fail(KV_ERR_INVALID, at + "unknown mode");
    if (C.partitioned > 1) return fail(KV_ERR_INVALID, at + "partitioned must be 0 or 1");
    for (int r = 0; r < 4; ++r)
      if (C.reserved[r]) return fail(KV_ERR_INVALID, at + "reserved bytes must be zero");
    if (C.medium >= std::max<uint32_t>(n_media, 1))
      return fail(KV_ERR_INVALID, at + "the disk medium is not in the cost model");
    if (C.disk_ttl > 1) return fail(KV_ERR_INVALID, at + "disk_ttl must be 0 or 1");
    if (C.disk_ttl) {
      for (uint32_t g = 0; g < G; ++g)
        if (!finite_nonneg(C.ttl[g]))
          return fail(KV_ERR_INVALID, at + "disk TTLs must be finite and >= 0");
      if (C.mode != KV_MODE_INCLUSIVE || C.partitioned || C.policy[0] != KV_POLICY_LRU)
        return fail(KV_ERR_UNSUPPORTED,
                    at + "a disk TTL tier needs the inclusive mode, LRU and shared tiers");
      if (C.cap[2])
        for (uint32_t g = 1; g < G; ++g)
          if (C.ttl[g] != C.ttl[0])
            return fail(KV_ERR_UNSUPPORTED, at + "a bounded disk TTL tier needs one TTL");
    }
    for (int k = 0; k < 3; ++k)
      if (C.cap[k] != 0 && C.cap[k] < wmax)
        return fail(KV_ERR_INVALID, at + "a tier capacity is below the largest block weight");
    const uint32_t ng = C.partitioned ? G : 1;
    for (uint32_t g = 0; g < ng; ++g) {
      if (C.policy[g] > KV_POLICY_LEAF) return fail(KV_ERR_INVALID, at + "unknown policy");
      if (C.policy[g] == KV_POLICY_LEAF &&
          (C.partitioned || C.mode != KV_MODE_INCLUSIVE || C.disk_ttl))
        return fail(KV_ERR_UNSUPPORTED,
                    at + "radix-tree eviction needs the inclusive mode on shared tiers");
    }
    if (C.partitioned) {
      for (int k = 0; k < 3; ++k) {
        uint64_t sum = 0;
        for (uint32_t g = 0; g < G; ++g) {
          const uint64_t x = C.cap_group[k][g];
          if (x != 0 && x < wmax)
            return fail(KV_ERR_INVALID, at + "a group capacity is below the largest block weight");
          sum += x;
          if (sum < x) return fail(KV_ERR_INVALID, at + "group capacities overflow");
        }
        if (sum > C.cap[k]) return fail(KV_ERR_INVALID, at + "group capacities exceed the tier");
      }
    }
    if (C.mode == KV_MODE_INCLUSIVE_PREFIX &&
        (C.partitioned || C.policy[0] != KV_POLICY_LRU))
      return fail(KV_ERR_UNSUPPORTED, at + "prefix reuse supports shared LRU tiers only");
  }
  return KV_OK;
}

uint32_t clamp32(uint64_t x) { return x > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)x; }

// Capacities the closed-form LRU records will look up, per group.
void add_thresholds(std::vector<std::vector<uint32_t>>& per_group, const kv_config& C, uint32_t g,
                    uint32_t slot, uint64_t w0) {
  if (C.mode == KV_MODE_INCLUSIVE || C.mode == KV_MODE_INCLUSIVE_PREFIX) {
    for (int k = 0; k < 3; ++k) {
      const uint64_t x = group_cap(C, k, g);
      if (x) per_group[slot].push_back(clamp32(x));
    }
  } else {
    uint64_t S = 0;
    for (int k = 0; k < 3; ++k) {
      const uint64_t x = group_cap(C, k, g);
      if (!x) continue;
      S += x / w0;
      per_group[slot].push_back(clamp32(S * w0));
    }
  }
}

void finish_set(ThresholdSet& ts, std::vector<std::vector<uint32_t>>& per_group, uint32_t G) {
  ts.values.clear();
  ts.n_groups = G;
  ts.off[0] = 0;
  for (uint32_t g = 0; g < G; ++g) {
    auto& v = per_group[g];
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
    ts.values.insert(ts.values.end(), v.begin(), v.end());
    ts.off[g + 1] = (uint32_t)ts.values.size();
  }
  for (uint32_t g = G + 1; g <= KV_MAX_GROUPS; ++g) ts.off[g] = ts.off[G];
}

// The disk TTL tiers' bins: per group its sorted distinct TTL values, the
// joint histograms' layout (bins of group g: (capacities + 1) x (TTLs + 1)),
// zeroed device histograms.  Needs the shared threshold set built.
kv_status plan_joint(Trace& t, std::vector<std::vector<double>>& per_group, JointArgs& ja,
                     JointView& jv, hipStream_t s) {
  const uint32_t G = t.n_groups;
  TtlSet& ts = t.ttl_ts;
  ts.values.clear();
  ts.n_groups = G;
  ts.off[0] = 0;
  std::vector<uint32_t> jbase(G + 1, 0);
  for (uint32_t g = 0; g < G; ++g) {
    auto& v = per_group[g];
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
    if (v.size() > 1024)
      return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: more than 1,024 disk TTLs in one group");
    ts.values.insert(ts.values.end(), v.begin(), v.end());
    ts.off[g + 1] = (uint32_t)ts.values.size();
    const uint64_t nd = (uint64_t)t.shared_ts.off[g + 1] - t.shared_ts.off[g] + 1;
    const uint64_t nb = (uint64_t)jbase[g] + nd * (v.size() + 1);
    if (nb > 0x7FFFFFFFull) return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: too many joint bins");
    jbase[g + 1] = (uint32_t)nb;
  }
  const uint32_t nt = (uint32_t)ts.values.size(), nj = jbase[G];
  // device: TTL values (doubles), then toff and jbase (u32)
  t.joint_stage.assign(2 * nt + 2 * (G + 1), 0);
  std::memcpy(t.joint_stage.data(), ts.values.data(), nt * sizeof(double));
  for (uint32_t g = 0; g <= G; ++g) {
    t.joint_stage[2 * nt + g] = ts.off[g];
    t.joint_stage[2 * nt + G + 1 + g] = jbase[g];
  }
  kv_status st;
  DevBuf& bt = t.ws[27];
  DevBuf& bh = t.ws[28];
  if ((st = bt.reserve(t.joint_stage.size() * 4)) != KV_OK) return st;
  const uint64_t hwords = 4ull * nj + nt + G;
  if ((st = bh.reserve(hwords * 8)) != KV_OK) return st;
  KV_HIP(hipMemcpyAsync(bt.p, t.joint_stage.data(), t.joint_stage.size() * 4,
                        hipMemcpyHostToDevice, s));
  if ((st = fill_u64(bh.as<uint64_t>(), 0, hwords, s)) != KV_OK) return st;
  ja.tthr = bt.as<double>();
  ja.toff = bt.as<uint32_t>() + 2 * nt;
  ja.jbase = ja.toff + G + 1;
  ja.n_tthr = nt;
  ja.n_joint = nj;
  ja.jh = bh.as<uint64_t>();
  ja.fh = ja.jh + 2ull * nj;
  ja.wd = reinterpret_cast<double*>(ja.fh + 2ull * nj);
  jv.tthr = ja.tthr;
  jv.toff = ja.toff;
  jv.jbase = ja.jbase;
  jv.jh = ja.jh;
  jv.fh = ja.fh;
  jv.wd = ja.wd;
  return KV_OK;
}

struct StackSlot {
  int ws_thr, ws_hist, ws_phist;  // ws_phist < 0: no prefix-reuse histogram
};

kv_status run_stack(Trace& t, Order& o, bool partitioned, ThresholdSet& ts, StackSlot slot,
                    OrderView& view, OrderView& pview, const JointArgs* ja, const uint8_t* real,
                    hipStream_t s) {
  kv_status st;
  DevBuf& bt = t.ws[slot.ws_thr];
  DevBuf& bh = t.ws[slot.ws_hist];
  const uint64_t nthr = ts.values.size();
  if ((st = bt.reserve((nthr + KV_MAX_GROUPS + 1) * 4)) != KV_OK) return st;
  const uint64_t nbins = ts.total_bins();
  if ((st = bh.reserve(nbins * 4 * 8)) != KV_OK) return st;
  uint32_t* thr = bt.as<uint32_t>();
  uint32_t* off = thr + nthr;
  if (nthr) KV_HIP(hipMemcpyAsync(thr, ts.values.data(), nthr * 4, hipMemcpyHostToDevice, s));
  KV_HIP(hipMemcpyAsync(off, ts.off, (KV_MAX_GROUPS + 1) * 4, hipMemcpyHostToDevice, s));
  if ((st = fill_u64(bh.as<uint64_t>(), 0, nbins * 4, s)) != KV_OK) return st;
  uint64_t* ph = nullptr;
  if (slot.ws_phist >= 0) {
    DevBuf& bp = t.ws[slot.ws_phist];
    if ((st = bp.reserve(nbins * 4 * 8)) != KV_OK) return st;
    if ((st = fill_u64(bp.as<uint64_t>(), 0, nbins * 4, s)) != KV_OK) return st;
    ph = bp.as<uint64_t>();
  }
  if ((st = stack_pass(t, o, partitioned, ts, thr, off, bh.as<uint64_t>(), ph, ja, real, s)) !=
      KV_OK)
    return st;
  view.thr = thr;
  view.off = off;
  view.hist = bh.as<uint64_t>();
  pview = view;
  if (ph) pview.hist = ph;
  return KV_OK;
}

// kv_pareto's device counters, one set per device, kept until the process
// ends; `done` is recorded after each call's last use of them.
struct PareCounters {
  std::mutex mu;
  DevBuf buf;
  uint32_t* host = nullptr;  // pinned
  hipEvent_t done = nullptr;
};

kv_status pareto_counters(PareCounters** out) {
  static std::mutex mu;
  static PareCounters* per_dev[64] = {};
  int d = 0;
  KV_HIP(hipGetDevice(&d));
  if (d < 0 || d >= 64) return fail(KV_ERR_DEVICE, "device index out of range");
  std::lock_guard<std::mutex> lk(mu);
  if (!per_dev[d]) {
    auto* pc = new PareCounters();
    kv_status st = pc->buf.reserve(2 * sizeof(uint32_t));
    if (st != KV_OK) {
      delete pc;
      return st;
    }
    hipError_t e = hipHostMalloc((void**)&pc->host, 2 * sizeof(uint32_t), hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&pc->done, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(pc->done, nullptr);
    if (e != hipSuccess) {
      if (pc->done) (void)hipEventDestroy(pc->done);
      if (pc->host) (void)hipHostFree(pc->host);
      delete pc;
      return hip_fail(e, "kv_pareto: counters");
    }
    per_dev[d] = pc;
  }
  *out = per_dev[d];
  return KV_OK;
}

}  // namespace
}  // namespace kv

using namespace kv;

extern "C" {

const char* kv_last_error(void) { return kv::g_last_error.c_str(); }

kv_status kv_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(kv::g_tmu);
  kv::g_timing = on != 0;
  return KV_OK;
}

kv_status kv_timing_read(kv_timing* out, int reset) {
  if (!out) return fail(KV_ERR_INVALID, "kv_timing_read: out is NULL");
  std::lock_guard<std::mutex> lk(kv::g_tmu);
  for (auto& p : kv::g_pairs) {
    KV_HIP(hipEventSynchronize(p.b));
    float ms = 0;
    KV_HIP(hipEventElapsedTime(&ms, p.a, p.b));
    kv::g_acc.calls[p.stage] += 1;
    kv::g_acc.ms[p.stage] += ms;
    kv::g_free_events.push_back(p.a);
    kv::g_free_events.push_back(p.b);
  }
  kv::g_pairs.clear();
  *out = kv::g_acc;
  if (reset) kv::g_acc = kv_timing{};
  return KV_OK;
}

kv_status kv_trace_load(const kv_trace_desc* d, void* stream, kv_trace** out) {
  if (!out) return fail(KV_ERR_INVALID, "kv_trace_load: out is NULL");
  *out = nullptr;
  if (!d) return fail(KV_ERR_INVALID, "kv_trace_load: desc is NULL");
  if (d->n < 1 || d->n > kMaxN)
    return fail(KV_ERR_INVALID, "kv_trace_load: n must be in [1, 2^29]");
  if (!d->hash || !d->req || !d->req_time)
    return fail(KV_ERR_INVALID, "kv_trace_load: hash, req and req_time are required");
  if (d->n_req < 1) return fail(KV_ERR_INVALID, "kv_trace_load: n_req must be >= 1");
  if (d->n_groups < 1 || d->n_groups > KV_MAX_GROUPS)
    return fail(KV_ERR_INVALID, "kv_trace_load: n_groups must be in [1, 16]");
  if (d->tokens_per_granule < 1 || d->granule_bytes < 1)
    return fail(KV_ERR_INVALID, "kv_trace_load: tokens_per_granule and granule_bytes must be >= 1");
  hipStream_t s = (hipStream_t)stream;
  Trace* t = new Trace();
  KV_HIP(hipGetDevice(&t->device));
  kv_status st = canon_build(*t, *d, s);
  if (st == KV_OK && t->st.n_w >= 0xFFFFFFFFull) {
    st = fail(KV_ERR_UNSUPPORTED, "kv_trace_load: total weight must stay below 2^32 granules");
  }
  if (st == KV_OK) st = t->err.reserve(2 * sizeof(uint32_t));
  if (st == KV_OK) st = fill_u32(t->err.as<uint32_t>(), 0, 2, s);
  if (st == KV_OK) {
    hipError_t e = hipHostMalloc((void**)&t->err_host, 2 * sizeof(uint32_t), hipHostMallocDefault);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&t->err_ev, hipEventDisableTiming);
    if (e != hipSuccess) st = hip_fail(e, "kv_trace_load: error record");
    else t->err_host[0] = t->err_host[1] = 0;
  }
  if (st != KV_OK) {
    (void)hipStreamSynchronize(s);
    delete t;
    return st;
  }
  t->magic = kTraceMagic;
  t->gb = d->granule_bytes;
  t->tpg = d->tokens_per_granule;
  {
    std::lock_guard<std::mutex> lk(g_reg_mu);
    g_live.insert(t);
  }
  *out = reinterpret_cast<kv_trace*>(t);
  return KV_OK;
}

kv_status kv_ttl_curves(const kv_trace* h, const double* ttl, uint32_t n_ttl, uint64_t* hits,
                        uint64_t* hitw, double* store, void* stream) {
  if (!h) return fail(KV_ERR_INVALID, "kv_ttl_curves: trace is NULL");
  Trace* t = const_cast<Trace*>(reinterpret_cast<const Trace*>(h));
  if (!is_live(t)) return fail(KV_ERR_INVALID, "kv_ttl_curves: not a live trace handle");
  if (kv_status e = check_device_error(*t, false, "kv_ttl_curves")) return e;
  if (!ttl || !hits || !hitw || !store)
    return fail(KV_ERR_INVALID, "kv_ttl_curves: ttl, hits, hitw and store are required");
  if (n_ttl == 0) return fail(KV_ERR_INVALID, "kv_ttl_curves: n_ttl must be >= 1");
  for (uint32_t k = 0; k < n_ttl; ++k) {
    if (!std::isfinite(ttl[k]) || ttl[k] < 0.0)
      return fail(KV_ERR_INVALID, "kv_ttl_curves: ttl values must be finite and >= 0");
    if (k && ttl[k] < ttl[k - 1])
      return fail(KV_ERR_INVALID, "kv_ttl_curves: ttl values must be non-decreasing");
  }
  if ((uint64_t)t->n_groups * ((uint64_t)n_ttl + 1) > 4096)
    return fail(KV_ERR_UNSUPPORTED, "kv_ttl_curves: n_groups * (n_ttl + 1) must be <= 4096");
  hipStream_t s = (hipStream_t)stream;
  // the thresholds are staged in the trace so they outlive the async copy
  t->ttl_stage.assign(ttl, ttl + n_ttl);
  DevBuf& bt = t->ws[23];
  kv_status st;
  if ((st = bt.reserve((uint64_t)n_ttl * 8)) != KV_OK) return st;
  KV_HIP(hipMemcpyAsync(bt.p, t->ttl_stage.data(), (uint64_t)n_ttl * 8, hipMemcpyHostToDevice, s));
  return ttl_curves(*t, bt.as<double>(), n_ttl, hits, hitw, store, s);
}

kv_status kv_ttl_curves_noalloc(const kv_trace* h, const double* ttl, uint32_t n_ttl,
                                uint64_t* hits, uint64_t* hitw, double* store, void* stream) {
  if (!h) return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: trace is NULL");
  Trace* t = const_cast<Trace*>(reinterpret_cast<const Trace*>(h));
  if (!is_live(t)) return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: not a live trace handle");
  if (kv_status e = check_device_error(*t, false, "kv_ttl_curves_noalloc")) return e;
  if (!ttl || !hits || !hitw || !store)
    return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: ttl, hits, hitw and store are required");
  if (n_ttl == 0) return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: n_ttl must be >= 1");
  for (uint32_t k = 0; k < n_ttl; ++k) {
    if (!std::isfinite(ttl[k]) || ttl[k] < 0.0)
      return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: ttl values must be finite and >= 0");
    if (k && ttl[k] < ttl[k - 1])
      return fail(KV_ERR_INVALID, "kv_ttl_curves_noalloc: ttl values must be non-decreasing");
  }
  return ttl_curves_noalloc(*t, ttl, n_ttl, hits, hitw, store, (hipStream_t)stream);
}

kv_status kv_trace_free(kv_trace* h) {
  if (!h) return KV_OK;
  Trace* t = reinterpret_cast<Trace*>(h);
  {
    std::lock_guard<std::mutex> lk(g_reg_mu);
    if (!g_live.count(t)) return fail(KV_ERR_INVALID, "kv_trace_free: not a live trace handle");
    g_live.erase(t);
  }
  (void)hipDeviceSynchronize();
  t->magic = kDeadMagic;
  delete t;
  return KV_OK;
}

kv_status kv_trace_info(const kv_trace* h, kv_trace_stats* out) {
  if (!h || !out) return fail(KV_ERR_INVALID, "kv_trace_info: NULL argument");
  Trace* t = const_cast<Trace*>(reinterpret_cast<const Trace*>(h));
  if (!is_live(t)) return fail(KV_ERR_INVALID, "kv_trace_info: not a live trace handle");
  *out = t->st;
  return check_device_error(*t, true, "kv_trace_info");
}

kv_status kv_eval_configs(const kv_trace* h, const kv_config* cfg, uint32_t n_cfg,
                          const kv_cost_model* model, uint64_t* counts, double* obj,
                          void* stream) {
  if (!h) return fail(KV_ERR_INVALID, "kv_eval_configs: trace is NULL");
  Trace* t = const_cast<Trace*>(reinterpret_cast<const Trace*>(h));
  if (!is_live(t)) return fail(KV_ERR_INVALID, "kv_eval_configs: not a live trace handle");
  kv_status st;
  if ((st = check_device_error(*t, false, "kv_eval_configs")) != KV_OK) return st;
  if ((st = validate_model(model)) != KV_OK) return st;
  if (n_cfg == 0) return KV_OK;
  if (!cfg || !counts) return fail(KV_ERR_INVALID, "kv_eval_configs: cfg and counts are required");
  if ((st = validate_configs(*t, cfg, n_cfg, model->n_media)) != KV_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  bool need_leaf = false;
  for (uint32_t c = 0; c < n_cfg; ++c) need_leaf |= !cfg[c].partitioned && cfg[c].policy[0] == KV_POLICY_LEAF;
  if (need_leaf) {
    // radix-tree eviction: a trace of prefix-chain requests, each fitting
    // every tier; its stack pass runs over 2N positions, within kMaxN
    if (2 * t->n > kMaxN)
      return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: radix-tree eviction evaluates an order of "
                                      "2N positions, at most " + std::to_string(kMaxN) +
                                      " (N = " + std::to_string(t->n) + ")");
    // that order carries every access's weight twice: its sums stay below 2^32
    if (2 * t->st.n_w >= 0xFFFFFFFFull)
      return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: radix-tree eviction needs the total "
                                      "weight below 2^31 granules");
    if ((st = leaf_prepare(*t, s)) != KV_OK) return st;
    if (!t->leaf_chained)
      return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: radix-tree eviction needs requests that "
                                      "are prefix chains of blocks");
    for (uint32_t c = 0; c < n_cfg; ++c) {
      if (cfg[c].partitioned || cfg[c].policy[0] != KV_POLICY_LEAF) continue;
      for (int k = 0; k < 3; ++k)
        if (cfg[c].cap[k] && cfg[c].cap[k] < t->max_req_w)
          return fail(KV_ERR_UNSUPPORTED, "kv_eval_configs: config " + std::to_string(c) +
                                              ": radix-tree eviction needs every tier to hold "
                                              "the heaviest request (" +
                                              std::to_string(t->max_req_w) + " granules)");
    }
  }
  const uint32_t G = t->n_groups;
  t->cfg_stage.assign(cfg, cfg + n_cfg);

  // ---- plan: thresholds per order, replay jobs
  std::vector<std::vector<uint32_t>> tsh(G), tpt(G), tlf(G);
  std::vector<std::vector<double>> tttl(G);  // disk TTL values per group
  bool need_shared = false, need_part = false, need_prefix = false, need_joint = false;
  const uint64_t w0 = t->st.w_max;
  const bool mixed = t->st.w_min != t->st.w_max;
  bool need_excl = false;
  std::map<std::tuple<uint32_t, uint32_t, uint32_t, uint64_t>, uint32_t> job_index;
  std::vector<ReplayJob> jobs;
  for (uint32_t c = 0; c < n_cfg; ++c) {
    const kv_config& C = cfg[c];
    const bool part_order = C.partitioned && G > 1;
    const uint32_t ng = C.partitioned ? G : 1;
    for (uint32_t g = 0; g < ng; ++g) {
      const uint32_t pol = group_policy(C, g);
      if (excl_replayed(C, g, mixed)) {  // replayed access by access
        need_excl = true;
        continue;
      }
      if (pol == KV_POLICY_LEAF) {
        for (uint32_t gg = 0; gg < G; ++gg) add_thresholds(tlf, C, 0, gg, w0);
        continue;
      }
      if (pol == KV_POLICY_LRU) {
        need_prefix |= C.mode == KV_MODE_INCLUSIVE_PREFIX;
        if (C.disk_ttl) {
          need_joint = true;
          for (uint32_t gg = 0; gg < G; ++gg) tttl[gg].push_back(C.ttl[gg]);
        }
        if (part_order) {
          need_part = true;
          add_thresholds(tpt, C, g, g, w0);
        } else {
          need_shared = true;
          if (C.partitioned) {
            add_thresholds(tsh, C, g, 0, w0);
          } else {
            for (uint32_t gg = 0; gg < G; ++gg) add_thresholds(tsh, C, 0, gg, w0);
          }
        }
        continue;
      }
      for (int k = 0; k < 3; ++k) {
        const uint64_t x = group_cap(C, k, g);
        if (!x) continue;
        const uint32_t ord = part_order ? 1u : 0u;
        const uint32_t grp = part_order ? g : (uint32_t)KV_MAX_GROUPS;
        auto key = std::make_tuple(ord, grp, pol, x);
        if (job_index.count(key)) continue;
        job_index[key] = (uint32_t)jobs.size();
        ReplayJob j{};
        j.order = ord;
        j.group = grp;
        j.policy = pol;
        j.cap = x;
        const uint64_t dw = part_order ? t->st.u_w_g[g] : t->st.distinct_w;
        j.closed = x >= dw ? 1u : 0u;
        jobs.push_back(j);
      }
    }
  }
  if (need_part || (!jobs.empty() && G > 1)) {
    if ((st = canon_partition(*t, s)) != KV_OK) return st;
  }
  for (auto& j : jobs) {
    const Order& o = j.order ? t->part : t->shared;
    j.begin = j.order ? o.seg[j.group] : 0;
    j.end = j.order ? o.seg[j.group + 1] : t->n;
  }

  // ---- device copies of the batch and per-group statistics
  DevBuf& bcfg = t->ws[9];
  DevBuf& bgs = t->ws[10];
  if ((st = bcfg.reserve((uint64_t)n_cfg * sizeof(kv_config))) != KV_OK) return st;
  if ((st = bgs.reserve(sizeof(GroupStats) * KV_MAX_GROUPS)) != KV_OK) return st;
  for (uint32_t g = 0; g < KV_MAX_GROUPS; ++g)
    t->gs_stage[g] = GroupStats{t->st.n_g[g], t->st.n_w_g[g], t->st.u_g[g], w0, t->st.u_w_g[g]};
  KV_HIP(hipMemcpyAsync(bcfg.p, t->cfg_stage.data(), (uint64_t)n_cfg * sizeof(kv_config),
                        hipMemcpyHostToDevice, s));
  KV_HIP(hipMemcpyAsync(bgs.p, t->gs_stage, sizeof(t->gs_stage), hipMemcpyHostToDevice, s));
  const kv_config* cfg_dev = bcfg.as<kv_config>();
  double* store_cg = nullptr;  // unbounded disk TTL tiers' storage integrals
  if (need_joint) {
    if ((st = t->ws[29].reserve((uint64_t)n_cfg * G * sizeof(double))) != KV_OK) return st;
    store_cg = t->ws[29].as<double>();
  }

  // ---- LRU: stack-distance passes + closed forms
  auto lru = [&]() -> kv_status {
    kv_status r;
    OrderView vsh, vpt, vpx, vlf, unused;
    JointArgs ja;
    JointView jv;
    if (need_shared) {
      finish_set(t->shared_ts, tsh, G);
      if (need_joint && (r = plan_joint(*t, tttl, ja, jv, s)) != KV_OK) return r;
      if ((r = run_stack(*t, t->shared, false, t->shared_ts,
                         StackSlot{5, 6, need_prefix ? 24 : -1}, vsh, vpx,
                         need_joint ? &ja : nullptr, nullptr, s)) != KV_OK)
        return r;
    }
    if (need_leaf) {
      finish_set(t->leaf_ts, tlf, G);
      if ((r = run_stack(*t, t->leaf, false, t->leaf_ts, StackSlot{30, 31, -1}, vlf, unused,
                         nullptr, t->leaf_real.as<uint8_t>(), s)) != KV_OK)
        return r;
    }
    if (need_part) {
      finish_set(t->part_ts, tpt, G);
      if ((r = run_stack(*t, t->part, true, t->part_ts, StackSlot{7, 8, -1}, vpt, unused,
                         nullptr, nullptr, s)) != KV_OK)
        return r;
    }
    if (need_shared || need_part || need_leaf)
      return lru_counts(cfg_dev, n_cfg, G, vsh, vpt, vpx, vlf, jv, bgs.as<GroupStats>(), mixed,
                        counts, store_cg, s);
    return KV_OK;
  };
  // ---- FIFO / LFU: replay jobs, with the LRU work running meanwhile
  if (!jobs.empty()) {
    if ((st = replay_run(*t, jobs, cfg, cfg_dev, n_cfg, counts, s, lru)) != KV_OK) return st;
  } else if ((st = lru()) != KV_OK) {
    return st;
  }
  // ---- exclusive hierarchies without a split stack
  if (need_excl && (st = excl_run(*t, cfg, cfg_dev, n_cfg, counts, s)) != KV_OK) return st;
  // ---- objectives
  if (obj) {
    st = objectives(cfg_dev, n_cfg, G, counts, store_cg, *model, (double)t->gb, (double)t->tpg,
                    t->st.span, (double)t->st.n_req, t->st.n_w, obj, s);
    if (st != KV_OK) return st;
  }
  return KV_OK;
}

kv_status kv_pareto(const double* obj, const uint32_t* segment, uint32_t n, const double* bounds,
                    uint8_t* on_front, uint32_t* n_front, void* stream) {
  if (n == 0) {
    if (n_front) *n_front = 0;
    return KV_OK;
  }
  if (!obj || !on_front) return fail(KV_ERR_INVALID, "kv_pareto: obj and on_front are required");
  if (n > (1u << 26)) return fail(KV_ERR_INVALID, "kv_pareto: n must be <= 2^26");
  hipStream_t s = (hipStream_t)stream;
  // the per-device counters {flagged rows, NaN seen}, allocated on the first
  // call; calls on different streams take turns through `done`
  PareCounters* pc = nullptr;
  kv_status st = pareto_counters(&pc);
  if (st != KV_OK) return st;
  std::lock_guard<std::mutex> lk(pc->mu);
  KV_HIP(hipStreamWaitEvent(s, pc->done, 0));
  uint32_t* counters = pc->buf.as<uint32_t>();
  st = fill_u32(counters, 0, 2, s);
  if (st == KV_OK) st = pareto(obj, segment, n, bounds, on_front, counters, s);
  if (st == KV_OK && n_front) {
    hipError_t e = hipMemcpyAsync(pc->host, counters, 2 * sizeof(uint32_t),
                                  hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) st = hip_fail(e, "kv_pareto result copy");
  }
  KV_HIP(hipEventRecord(pc->done, s));
  if (st != KV_OK) return st;
  if (n_front) {
    KV_HIP(hipEventSynchronize(pc->done));
    *n_front = pc->host[0];
    if (pc->host[1]) return fail(KV_ERR_INVALID, "kv_pareto: an objective is NaN");
  }
  return KV_OK;
}

}  // extern "C"
