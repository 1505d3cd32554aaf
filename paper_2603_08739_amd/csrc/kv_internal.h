// kv_internal.h - internal declarations shared by the HIP translation units
// of libkvcfg (never installed; the public contract is include/kvcfg.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <functional>
#include <vector>

#include "../../include/kvcfg.h"

namespace kv {

constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr int kSdLogB = 13;                 // stack-distance position block: 8192
constexpr uint32_t kSdB = 1u << kSdLogB;
constexpr uint64_t kMaxN = 1ull << 29;

// ---------------------------------------------------------------------------
// error state
// ---------------------------------------------------------------------------
kv_status fail(kv_status s, const std::string& msg);
kv_status hip_fail(hipError_t e, const char* what);

#define KV_HIP(call)                                          \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return ::kv::hip_fail(e_, #call);   \
  } while (0)

// A device allocation owned by its holder; released blocks return to a
// per-device cache for the next reserve.
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;      // bytes asked for
  size_t cap_bytes = 0;  // size of the block held
  int dev = 0;           // device the block lives on
  DevBuf() = default;
  DevBuf(const DevBuf&) = delete;
  DevBuf& operator=(const DevBuf&) = delete;
  ~DevBuf() { release(); }
  void release();
  // Grow to at least `b` bytes (contents are not preserved on growth).
  kv_status reserve(size_t b);
  template <class T>
  T* as() const { return static_cast<T*>(p); }
};

// One order of the accesses: the trace order, or the accesses regrouped
// stably by tenant group (for per-group partitioned caches).
struct Order {
  DevBuf key;   // u32[n]: previous occurrence + 1 in this order, 0 = first access
  DevBuf nxt;   // u32[n]: next occurrence in this order, kNone = last access
  DevBuf bid;   // u32[n]: dense block id
  DevBuf w;     // u8[n]
  DevBuf g;     // u8[n]
  uint64_t seg[KV_MAX_GROUPS + 1] = {0};  // group segments (partitioned order)
  uint64_t n = 0;                          // positions (0: the trace's accesses)
  bool built = false;
};

struct ThresholdSet {
  // thresholds (granules, clamped to u32) per group, concatenated; bins per
  // group = count + 1 (the last bin collects distances above every threshold)
  std::vector<uint32_t> values;
  uint32_t off[KV_MAX_GROUPS + 1] = {0};  // thresholds of group g: [off[g], off[g+1])
  uint32_t n_groups = 1;
  uint32_t total_bins() const { return off[n_groups] + n_groups; }
  uint32_t bin_base(uint32_t g) const { return off[g] + g; }
};

// What an error message needs to name a replay job.
struct ReplayJobInfo {
  uint32_t policy, group;
  uint64_t cap;
};

struct GroupStats {
  uint64_t n_g, n_w_g, u_g, w0;  // accesses, weight, distinct blocks, uniform weight
  uint64_t u_w_g;                // distinct weight
};

// The TTL values disk TTL tiers use, per group (sorted, distinct).
struct TtlSet {
  std::vector<double> values;
  uint32_t off[KV_MAX_GROUPS + 1] = {0};
  uint32_t n_groups = 1;
};

// Disk TTL tiers (trace order): per group, a joint histogram of accesses by
// (stack-distance bin, gap bin) and of blocks by (final-depth bin, end-age
// bin), bin (d, t) of group g at jbase[g] + d * (tbins of g) + t; gap bins
// cut at the group's TTL values (bin t = #{ttl < gap}; no gap = last bin).
struct JointArgs {
  const double* tthr = nullptr;    // [toff[G]] TTL values, device
  const uint32_t* toff = nullptr;  // [G + 1], device
  const uint32_t* jbase = nullptr; // [G + 1], device
  uint32_t n_tthr = 0, n_joint = 0;
  uint64_t* jh = nullptr;          // [n_joint][2] count, weight (zeroed)
  uint64_t* fh = nullptr;          // [n_joint][2] count, weight (zeroed)
  double* wd = nullptr;            // [n_tthr + G] sum of w * gap per (group, gap bin) (zeroed)
};

struct Trace {
  uint64_t magic = 0;
  int device = 0;
  kv_trace_stats st{};
  uint64_t n = 0, u = 0;
  uint32_t n_groups = 1;
  uint64_t gb = 0;    // granule bytes
  uint32_t tpg = 0;   // tokens per granule
  Order shared;       // trace order
  Order part;         // partitioned order (built on first use when n_groups > 1)
  // Radix-tree eviction: the trace with every request followed by a re-touch
  // of its blocks, deepest first (built on first use); `leaf_real` flags
  // the positions that are accesses of the trace.
  Order leaf;
  DevBuf leaf_real;   // u8[2n]
  bool leaf_checked = false, leaf_chained = false;
  uint64_t max_req_w = 0;  // heaviest request (granules)
  DevBuf blk_w;       // u8[u]  weight per dense block id
  DevBuf blk_g;       // u8[u]  group per dense block id
  DevBuf req;         // u32[n] request of each access (trace order)
  DevBuf req_time;    // f64[n_req] arrival time of each request
  // workspace reused across kv_eval_configs calls on this trace
  DevBuf ws[32];
  // Device error record {code, job} written by a replay kernel that fails
  // its internal state check; copied after every kv_eval_configs call that
  // replays into `err_host` (pinned), with `err_ev` recorded after the copy.
  DevBuf err;
  uint32_t* err_host = nullptr;
  hipEvent_t err_ev = nullptr;
  bool err_pending = false;
  std::vector<ReplayJobInfo> err_jobs;  // the replayed jobs of the latest call
  ~Trace();
  // host staging of the latest kv_eval_configs call (alive across its copies)
  ThresholdSet shared_ts, part_ts, leaf_ts;
  TtlSet ttl_ts;
  std::vector<uint32_t> joint_stage;
  std::vector<kv_config> cfg_stage;
  GroupStats gs_stage[KV_MAX_GROUPS];
  std::vector<uint8_t> job_stage, rec_stage, src_stage;
  std::vector<double> ttl_stage;
  std::vector<unsigned long long> jc_stage;
  std::vector<uint8_t> excl_stage;
};

constexpr uint64_t kTraceMagic = 0x6b7663666774726bull;  // "kvcfgtrk"
constexpr uint64_t kDeadMagic = 0x646561646b766366ull;

// ---------------------------------------------------------------------------
// stage timing (kv_timing_enable / kv_timing_read)
// ---------------------------------------------------------------------------
enum Stage {
  kStLoadValidate = 0, kStLoadSort, kStLoadLinks, kStPartition, kStStackMatrix,
  kStStackLocal, kStStackAssemble, kStStackFinal, kStLruCounts, kStReplayInit, kStReplay,
  kStCombine, kStObjectives, kStPareto, kStReplayFifo, kStTtl, kStReplayExcl
};
// Records an event pair around a scope when timing is enabled.
struct StageTimer {
  StageTimer(Stage st, hipStream_t s);
  ~StageTimer();
  int slot;
  hipStream_t s;
};

// ---------------------------------------------------------------------------
// launchers (each defined in the .hip file that holds its kernels)
// ---------------------------------------------------------------------------
// exclusive (inclusive=false) or inclusive prefix sum of u32, any length;
// `scratch` holds scan_scratch_elems(m) u32 of device memory.  in == out is allowed.
uint64_t scan_scratch_elems(uint64_t m);
kv_status scan_u32(const uint32_t* in, uint32_t* out, uint64_t m, bool inclusive,
                   uint32_t* scratch, hipStream_t s);
kv_status fill_u32(uint32_t* p, uint32_t v, uint64_t m, hipStream_t s);
kv_status fill_u64(uint64_t* p, uint64_t v, uint64_t m, hipStream_t s);

// canonicalisation (k_canon.hip)
kv_status canon_build(Trace& t, const kv_trace_desc& d, hipStream_t s);
kv_status canon_partition(Trace& t, hipStream_t s);

// radix-tree eviction (k_leaf.hip): checks once whether the requests are
// prefix chains and finds the heaviest request; if they are chains, builds
// t.leaf and t.leaf_real.
kv_status leaf_prepare(Trace& t, hipStream_t s);

// stack-distance pass (k_stack.hip)
// hist: u64[total_bins][4] = {count, weight, final count, final weight},
// made cumulative over the bins of each group on return.
// thr_dev / off_dev: device copies of ts.values / ts.off; hist must be zeroed.
// phist (zeroed, same layout, or NULL; trace order only): fields 0 and 1
// count the accesses by their request-prefix distance (prefix reuse).
// ja (or NULL; trace order only): the joint histograms of disk TTL tiers,
// made cumulative over both bin dimensions (and wd over gap bins) on return.
// real (or NULL): per position, whether it is binned (the radix-tree order's
// re-touches are not).
kv_status stack_pass(Trace& t, Order& o, bool partitioned, const ThresholdSet& ts,
                     const uint32_t* thr_dev, const uint32_t* off_dev, uint64_t* hist,
                     uint64_t* phist, const JointArgs* ja, const uint8_t* real, hipStream_t s);

// per-configuration evaluation (k_eval.hip)

// Device view of one order's threshold sets and cumulative histograms.
struct OrderView {
  const uint32_t* thr = nullptr;
  const uint32_t* off = nullptr;
  const uint64_t* hist = nullptr;
};
// Device view of the cumulative joint histograms (trace order).
struct JointView {
  const double* tthr = nullptr;
  const uint32_t* toff = nullptr;
  const uint32_t* jbase = nullptr;
  const uint64_t* jh = nullptr;
  const uint64_t* fh = nullptr;
  const double* wd = nullptr;
};
// Writes the records of every (config, group) whose policy is LRU, except
// exclusive hierarchies over blocks of mixed weights (`mixed`), which are
// replayed.  Groups of
// partitioned configs read `part` when n_groups > 1, `shared` otherwise;
// prefix-reuse configs take their hits from `prefix` (trace order).
// Disk TTL tiers take tier 2 from `joint` and write the storage-time
// integral of each unbounded one per (config, group) to store_cg.
kv_status lru_counts(const kv_config* cfg_dev, uint32_t n_cfg, uint32_t n_groups,
                     OrderView shared, OrderView part, OrderView prefix, OrderView leaf,
                     JointView joint,
                     const GroupStats* gs_dev, bool mixed, uint64_t* counts, double* store_cg,
                     hipStream_t s);
// store_cg: [n_cfg][n_groups] or NULL (no disk TTL tier in the batch).
kv_status objectives(const kv_config* cfg_dev, uint32_t n_cfg, uint32_t n_groups,
                     const uint64_t* counts, const double* store_cg, const kv_cost_model& m,
                     double gb, double tpg, double span, double n_req, uint64_t n_w,
                     double* obj, hipStream_t s);
kv_status pareto(const double* obj, const uint32_t* segment, uint32_t n, const double* bounds,
                 uint8_t* flag, uint32_t* counters_dev, hipStream_t s);

// TTL curves (k_ttl.hip): validated arguments; ttl_dev holds the n_ttl
// thresholds on the device.
kv_status ttl_curves(Trace& t, const double* ttl_dev, uint32_t n_ttl, uint64_t* hits,
                     uint64_t* hitw, double* store, hipStream_t s);
// The same with the histograms at `hist` (3 * n_groups * (n_ttl + 1) words).
kv_status ttl_curves_into(Trace& t, const double* ttl_dev, uint32_t n_ttl,
                          unsigned long long* hist, uint64_t* hits, uint64_t* hitw,
                          double* store, hipStream_t s);
// The same in the library's per-device scratch array (no allocation); the
// TTL values are copied from the host through the stream.
kv_status ttl_curves_noalloc(Trace& t, const double* ttl_host, uint32_t n_ttl, uint64_t* hits,
                             uint64_t* hitw, double* store, hipStream_t s);

// Reports (and clears) a replay failure recorded on the device by an earlier
// kv_eval_configs call on `t`: with `wait`, waits for that call's error
// copy; otherwise reports only what has already arrived.
kv_status check_device_error(Trace& t, bool wait, const char* who);

// replay of non-LRU policies (k_replay.hip)
struct ReplayJob {
  uint32_t order;     // 0 = trace order, 1 = partitioned order
  uint32_t group;     // partitioned: the group; shared: KV_MAX_GROUPS
  uint32_t policy;    // KV_POLICY_FIFO or KV_POLICY_LFU
  uint32_t closed;    // 1: capacity covers every distinct block -> no replay
  uint64_t cap;       // granules
  uint64_t begin, end;  // positions [begin, end) in the order
};
// Replays FIFO/LFU jobs on two forked streams; `meanwhile` enqueues other
// work on s (it runs concurrently), then the streams are joined and the
// per-configuration records are combined on s.
kv_status replay_run(Trace& t, const std::vector<ReplayJob>& jobs, const kv_config* cfg_host,
                     const kv_config* cfg_dev, uint32_t n_cfg, uint64_t* counts,
                     hipStream_t s, const std::function<kv_status()>& meanwhile);

// exclusive hierarchies replayed access by access (k_excl.hip)
// Whether hierarchy g of C (group g when partitioned, 0 otherwise) is
// replayed there: the exclusive mode under FIFO or LFU, or under LRU when
// the trace's blocks have mixed weights (otherwise a split stack serves it).
bool excl_replayed(const kv_config& C, uint32_t g, bool mixed);
// Writes the records of every replayed hierarchy of the batch (the records
// of a shared hierarchy: every group).
kv_status excl_run(Trace& t, const kv_config* cfg_host, const kv_config* cfg_dev,
                   uint32_t n_cfg, uint64_t* counts, hipStream_t s);

}  // namespace kv
