// kvoracle.cpp - CPU ORACLE for the batched KV-tier configuration evaluator.
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
// benchmark's CPU-baseline leg load this library.  It shares no source with
// the GPU library: no headers, no helpers, no tables.  It is deliberately
// plain and slow: every configuration replays the whole trace literally,
// access after access, through standard-library containers keyed by the raw
// 64-bit block hash.
//
// What it computes (the paper's simulator replays a historical trace of
// KV-block hashes through a multi-tier storage model and reports hit rates
// per tier, Sections 3.2 and 4.1; the objectives follow Eq. 1 and Eq. 2 and
// the selector's dominance rule follows Section 4.1):
//
//   oracle_replay      per configuration, per tenant group, per tier:
//                      {hit, miss, ins, evict} and their granule-weighted twins.
//   oracle_objectives  (cost, throughput, latency) from those counts.
//   oracle_pareto      non-dominated flags under optional bounds.
//
// Cache rules (the paper names LRU for tier eviction, Section 2.1; FIFO and
// LFU are the benchmark's extra policies):
//   * A tier of capacity 0 is absent: it holds nothing and records nothing.
//   * Lookup happens before any update for the access.
//   * A miss inserts the block, first evicting victims until used + w <= C.
//     LRU evicts the least recently used block; FIFO the oldest insertion;
//     LFU the minimum (in-cache frequency, last access index) - frequency
//     starts at 1 on insertion, +1 per hit, and is forgotten on eviction.
//   * Inclusive hierarchy: every tier is an independent cache that sees every
//     access; the access is served by the fastest tier holding the block; then
//     every present tier applies its hit update and every other tier inserts.
//   * Inclusive hierarchy with prefix reuse (LRU, shared caches): contents
//     evolve exactly as in the inclusive hierarchy, but a request reuses only
//     a run of its blocks from its first block on, as a radix-tree cache
//     does (Section 3.2's prefix-shared KV blocks): per tier, block j of a
//     request is available iff the tier holds it and block j-1 of the same
//     request was available there (the first block needs only presence); the
//     access is served by the fastest tier where it is available.
//   * Exclusive hierarchy with write-back demotion (LRU only): a block lives
//     in at most one tier; a hit in a lower tier removes it there and promotes
//     it to the top tier; an overfull tier demotes its LRU block to the next
//     tier's MRU end; blocks pushed past the last tier are dropped.
//   * Counts: hit_k = accesses served by k; miss_k = accesses that reached k
//     (not served by a faster tier) and were not served by k; ins_k = blocks
//     that entered k; evict_k = blocks that left k for lack of room (a
//     demotion counts as an eviction of the source tier).  Evictions are
//     charged to the evicted block's group.
//
// Build: g++ -O2 -std=c++17 -ffp-contract=off -fPIC -shared -pthread
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <list>
#include <set>
#include <thread>
#include <tuple>
#include <unordered_map>
#include <vector>

namespace {

constexpr int kMaxGroups = 16;
constexpr int kTiers = 3;
constexpr int kFields = 8;  // hit, miss, ins, evict, hit_w, miss_w, ins_w, evict_w
enum Field { F_HIT = 0, F_MISS, F_INS, F_EVICT, F_HIT_W, F_MISS_W, F_INS_W, F_EVICT_W };
enum Policy { P_LRU = 0, P_FIFO = 1, P_LFU = 2 };
enum Mode { M_INCLUSIVE = 0, M_EXCLUSIVE = 1, M_INCLUSIVE_PREFIX = 2 };

struct Block {
  uint64_t hash;
  uint32_t w;
  uint32_t g;
  uint32_t req;
};

// Counts of one configuration: [group][tier][field].
struct Counts {
  uint64_t v[kMaxGroups][kTiers][kFields];
};

// ---------------------------------------------------------------------------
// One tier cache.  Subclasses implement one eviction policy each.
// ---------------------------------------------------------------------------
class Tier {
 public:
  explicit Tier(uint64_t cap) : cap_(cap) {}
  virtual ~Tier() = default;
  virtual bool contains(uint64_t h) const = 0;
  virtual void hit(uint64_t h, uint64_t t) = 0;
  // Insert a missing block; every victim is reported through `ev`.
  template <class F>
  void insert(const Block& b, uint64_t t, F&& ev) {
    while (used_ + b.w > cap_) {
      Block v = pop_victim();
      used_ -= v.w;
      ev(v);
    }
    push(b, t);
    used_ += b.w;
  }
  uint64_t used() const { return used_; }

 protected:
  virtual Block pop_victim() = 0;
  virtual void push(const Block& b, uint64_t t) = 0;
  uint64_t cap_;
  uint64_t used_ = 0;
};

// LRU: list front = most recently used.
class LruTier : public Tier {
 public:
  using Tier::Tier;
  bool contains(uint64_t h) const override { return pos_.count(h) != 0; }
  void hit(uint64_t h, uint64_t) override {
    auto it = pos_.at(h);
    order_.splice(order_.begin(), order_, it);
  }

 protected:
  Block pop_victim() override {
    Block v = order_.back();
    order_.pop_back();
    pos_.erase(v.hash);
    return v;
  }
  void push(const Block& b, uint64_t) override {
    order_.push_front(b);
    pos_[b.hash] = order_.begin();
  }
  std::list<Block> order_;
  std::unordered_map<uint64_t, std::list<Block>::iterator> pos_;
};

// FIFO: list front = newest insertion; hits do not reorder.
class FifoTier : public Tier {
 public:
  using Tier::Tier;
  bool contains(uint64_t h) const override { return pos_.count(h) != 0; }
  void hit(uint64_t, uint64_t) override {}

 protected:
  Block pop_victim() override {
    Block v = order_.back();
    order_.pop_back();
    pos_.erase(v.hash);
    return v;
  }
  void push(const Block& b, uint64_t) override {
    order_.push_front(b);
    pos_[b.hash] = order_.begin();
  }
  std::list<Block> order_;
  std::unordered_map<uint64_t, std::list<Block>::iterator> pos_;
};

// LFU: ordered set of (frequency, last access index, hash); victim = smallest.
class LfuTier : public Tier {
 public:
  using Tier::Tier;
  bool contains(uint64_t h) const override { return info_.count(h) != 0; }
  void hit(uint64_t h, uint64_t t) override {
    Info& in = info_.at(h);
    order_.erase(std::make_tuple(in.freq, in.last, h));
    in.freq += 1;
    in.last = t;
    order_.insert(std::make_tuple(in.freq, in.last, h));
  }

 protected:
  struct Info {
    uint64_t freq, last;
    Block b;
  };
  Block pop_victim() override {
    auto first = *order_.begin();
    order_.erase(order_.begin());
    uint64_t h = std::get<2>(first);
    Block v = info_.at(h).b;
    info_.erase(h);
    return v;
  }
  void push(const Block& b, uint64_t t) override {
    info_[b.hash] = Info{1, t, b};
    order_.insert(std::make_tuple(uint64_t(1), t, b.hash));
  }
  std::set<std::tuple<uint64_t, uint64_t, uint64_t>> order_;
  std::unordered_map<uint64_t, Info> info_;
};

Tier* make_tier(int policy, uint64_t cap) {
  if (policy == P_LRU) return new LruTier(cap);
  if (policy == P_FIFO) return new FifoTier(cap);
  return new LfuTier(cap);
}

void add(Counts& c, uint32_t g, int k, Field f, uint64_t cnt_field_weight) {
  c.v[g][k][f] += cnt_field_weight;
}

// Inclusive hierarchy over the accesses listed in `idx`; with `prefix`, a
// block is available from a tier only while its request's earlier blocks
// were.
void replay_inclusive(const std::vector<Block>& acc, const std::vector<uint32_t>& idx,
                      const uint64_t cap[kTiers], int policy, bool prefix, Counts& out) {
  Tier* tier[kTiers] = {nullptr, nullptr, nullptr};
  for (int k = 0; k < kTiers; ++k)
    if (cap[k] > 0) tier[k] = make_tier(policy, cap[k]);
  bool run[kTiers] = {false, false, false};  // the request's blocks so far all available
  bool first = true;
  uint32_t cur_req = 0;
  for (uint32_t i : idx) {
    const Block& b = acc[i];
    if (first || b.req != cur_req) {
      for (int k = 0; k < kTiers; ++k) run[k] = true;
      cur_req = b.req;
      first = false;
    }
    bool present[kTiers] = {false, false, false};
    int served = -1;
    for (int k = 0; k < kTiers; ++k) {
      if (!tier[k]) continue;
      present[k] = tier[k]->contains(b.hash);
      const bool avail = present[k] && (!prefix || run[k]);
      run[k] = avail;
      if (avail && served < 0) served = k;
    }
    for (int k = 0; k < kTiers; ++k) {
      if (!tier[k]) continue;
      if (served == k) {
        add(out, b.g, k, F_HIT, 1);
        add(out, b.g, k, F_HIT_W, b.w);
      } else if (served < 0 || served > k) {
        add(out, b.g, k, F_MISS, 1);
        add(out, b.g, k, F_MISS_W, b.w);
      }
    }
    for (int k = 0; k < kTiers; ++k) {
      if (!tier[k]) continue;
      if (present[k]) {
        tier[k]->hit(b.hash, i);
      } else {
        add(out, b.g, k, F_INS, 1);
        add(out, b.g, k, F_INS_W, b.w);
        tier[k]->insert(b, i, [&](const Block& v) {
          add(out, v.g, k, F_EVICT, 1);
          add(out, v.g, k, F_EVICT_W, v.w);
        });
      }
    }
  }
  for (int k = 0; k < kTiers; ++k) delete tier[k];
}

// Exclusive LRU hierarchy with write-back demotion over the accesses in `idx`.
void replay_exclusive(const std::vector<Block>& acc, const std::vector<uint32_t>& idx,
                      const uint64_t cap[kTiers], Counts& out) {
  // Each tier: list front = MRU.  where[h] = (tier, iterator).
  std::list<Block> lst[kTiers];
  uint64_t used[kTiers] = {0, 0, 0};
  std::unordered_map<uint64_t, std::pair<int, std::list<Block>::iterator>> where;
  std::vector<int> live;  // non-absent tiers, fastest first
  for (int k = 0; k < kTiers; ++k)
    if (cap[k] > 0) live.push_back(k);
  if (live.empty()) return;
  const int top = live[0];
  for (uint32_t i : idx) {
    const Block& b = acc[i];
    auto it = where.find(b.hash);
    int at = (it == where.end()) ? -1 : it->second.first;
    for (int k : live) {
      if (k == at) {
        add(out, b.g, k, F_HIT, 1);
        add(out, b.g, k, F_HIT_W, b.w);
        break;
      }
      add(out, b.g, k, F_MISS, 1);
      add(out, b.g, k, F_MISS_W, b.w);
    }
    if (at == top) {  // plain LRU hit in the top tier
      lst[top].splice(lst[top].begin(), lst[top], it->second.second);
      continue;
    }
    if (at >= 0) {  // hit in a lower tier: take it out for promotion
      lst[at].erase(it->second.second);
      used[at] -= b.w;
      where.erase(it);
    }
    lst[top].push_front(b);
    used[top] += b.w;
    where[b.hash] = {top, lst[top].begin()};
    add(out, b.g, top, F_INS, 1);
    add(out, b.g, top, F_INS_W, b.w);
    // cascade demotions down the hierarchy
    for (size_t li = 0; li < live.size(); ++li) {
      int k = live[li];
      while (used[k] > cap[k]) {
        Block v = lst[k].back();
        lst[k].pop_back();
        used[k] -= v.w;
        add(out, v.g, k, F_EVICT, 1);
        add(out, v.g, k, F_EVICT_W, v.w);
        if (li + 1 < live.size()) {
          int n = live[li + 1];
          lst[n].push_front(v);
          used[n] += v.w;
          where[v.hash] = {n, lst[n].begin()};
          add(out, v.g, n, F_INS, 1);
          add(out, v.g, n, F_INS_W, v.w);
        } else {
          where.erase(v.hash);
        }
      }
    }
  }
}

struct ConfigView {
  const uint64_t* cap;        // [3]
  const uint64_t* cap_group;  // [3][16]
  uint8_t mode;
  uint8_t partitioned;
  const uint8_t* policy;  // [16]
};

int replay_one(const std::vector<Block>& acc, const std::vector<std::vector<uint32_t>>& by_group,
               const std::vector<uint32_t>& all, uint32_t n_groups, uint32_t w_max,
               const ConfigView& c, Counts& out) {
  auto bad_cap = [&](uint64_t x) { return x > 0 && x < w_max; };
  if (c.partitioned) {
    for (uint32_t g = 0; g < n_groups; ++g) {
      uint64_t cg[kTiers];
      for (int k = 0; k < kTiers; ++k) {
        cg[k] = c.cap_group[k * kMaxGroups + g];
        if (bad_cap(cg[k])) return -1;
      }
      if (c.mode == M_INCLUSIVE_PREFIX) return -4;
      if (c.mode == M_EXCLUSIVE) {
        if (c.policy[g] != P_LRU) return -4;
        replay_exclusive(acc, by_group[g], cg, out);
      } else {
        replay_inclusive(acc, by_group[g], cg, c.policy[g], false, out);
      }
    }
  } else {
    for (int k = 0; k < kTiers; ++k)
      if (bad_cap(c.cap[k])) return -1;
    if (c.mode == M_EXCLUSIVE) {
      if (c.policy[0] != P_LRU) return -4;
      replay_exclusive(acc, all, c.cap, out);
    } else if (c.mode == M_INCLUSIVE_PREFIX) {
      if (c.policy[0] != P_LRU) return -4;
      replay_inclusive(acc, all, c.cap, P_LRU, true, out);
    } else {
      replay_inclusive(acc, all, c.cap, c.policy[0], false, out);
    }
  }
  return 0;
}

}  // namespace

extern "C" {

// Replays every configuration literally.  counts: uint64[n_cfg][n_groups][3][8].
// req: request of every access (NULL: one request per access).  Returns 0,
// or -1 for an invalid capacity (between 0 and the largest block), -4 for an
// exclusive or prefix hierarchy with a policy other than LRU (or a
// partitioned prefix one), -2 for bad sizes.
int oracle_replay(uint64_t n, const uint64_t* hash, const uint8_t* group, const uint8_t* weight,
                  const uint32_t* req, uint32_t n_groups, uint32_t n_cfg, const uint64_t* cap,
                  const uint64_t* cap_group, const uint8_t* mode, const uint8_t* partitioned,
                  const uint8_t* policy, uint32_t n_threads, uint64_t* counts) {
  if (n_groups < 1 || n_groups > (uint32_t)kMaxGroups) return -2;
  std::vector<Block> acc(n);
  std::vector<std::vector<uint32_t>> by_group(n_groups);
  std::vector<uint32_t> all(n);
  uint32_t w_max = 1;
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t g = group ? group[i] : 0;
    uint32_t w = weight ? weight[i] : 1;
    if (g >= n_groups || w == 0) return -2;
    acc[i] = Block{hash[i], w, g, req ? req[i] : (uint32_t)i};
    by_group[g].push_back((uint32_t)i);
    all[i] = (uint32_t)i;
    w_max = std::max(w_max, w);
  }
  std::atomic<uint32_t> next{0};
  std::atomic<int> status{0};
  auto work = [&]() {
    Counts* c = new Counts;
    for (;;) {
      uint32_t j = next.fetch_add(1);
      if (j >= n_cfg) break;
      std::fill(&c->v[0][0][0], &c->v[0][0][0] + kMaxGroups * kTiers * kFields, 0);
      ConfigView v{cap + 3 * (size_t)j, cap_group + 3 * kMaxGroups * (size_t)j, mode[j],
                   partitioned[j], policy + kMaxGroups * (size_t)j};
      int rc = replay_one(acc, by_group, all, n_groups, w_max, v, *c);
      if (rc != 0) status.store(rc);
      uint64_t* dst = counts + (size_t)j * n_groups * kTiers * kFields;
      for (uint32_t g = 0; g < n_groups; ++g)
        for (int k = 0; k < kTiers; ++k)
          for (int f = 0; f < kFields; ++f) dst[(g * kTiers + k) * kFields + f] = c->v[g][k][f];
    }
    delete c;
  };
  uint32_t nt = std::max<uint32_t>(1, std::min<uint32_t>(n_threads, n_cfg));
  std::vector<std::thread> th;
  for (uint32_t t = 1; t < nt; ++t) th.emplace_back(work);
  work();
  for (auto& t : th) t.join();
  return status.load();
}

// Objectives per configuration (cost, throughput, latency), all fp64, each
// step in the order written.  cost_model: [price_gpu_per_hour, price_gib_hour[3],
// bw_dram, ssd_bw_base, ssd_bw_per_gib, ssd_bw_max, t_prefill_per_token].
// The counts enter as granule totals over groups: H_w[k] = sum_g hit_w,
// I_w2 = sum_g ins_w of the SSD tier; recompute R_w = N_w - sum_k H_w[k].
//   capGiB[k] = cap[k] * gb / 2^30
//   bw_ssd    = min(ssd_bw_base + ssd_bw_per_gib * capGiB[2], ssd_bw_max)
//   t_dram    = H_w[1] * gb / bw_dram
//   t_ssd     = (H_w[2] + I_w2) * gb / bw_ssd
//   t_rec     = R_w * tpg * t_prefill_per_token
//   T_busy    = t_rec + t_dram + t_ssd;   T_wall = max(span, T_busy)
//   throughput = N_w * tpg / T_wall;      latency = T_busy / n_req
//   cost = (price_gpu + sum_k capGiB[k] * price_k) * T_wall / 3600
int oracle_objectives(uint32_t n_cfg, const uint64_t* cap, const uint64_t* counts,
                      uint32_t n_groups, const double* cm, double gb, double tpg,
                      double span, double n_req, uint64_t n_w, double* obj) {
  const double kGiB = 1073741824.0;
  for (uint32_t j = 0; j < n_cfg; ++j) {
    const uint64_t* c = counts + (size_t)j * n_groups * kTiers * kFields;
    uint64_t hw[kTiers] = {0, 0, 0};
    uint64_t iw2 = 0;
    for (uint32_t g = 0; g < n_groups; ++g) {
      for (int k = 0; k < kTiers; ++k) hw[k] += c[(g * kTiers + k) * kFields + F_HIT_W];
      iw2 += c[(g * kTiers + 2) * kFields + F_INS_W];
    }
    uint64_t rw = n_w - (hw[0] + hw[1] + hw[2]);
    double capgib[kTiers];
    for (int k = 0; k < kTiers; ++k) capgib[k] = ((double)cap[3 * (size_t)j + k] * gb) / kGiB;
    double bw_ssd = std::min(cm[5] + cm[6] * capgib[2], cm[7]);
    double t_dram = ((double)hw[1] * gb) / cm[4];
    double t_ssd = ((double)(hw[2] + iw2) * gb) / bw_ssd;
    double t_rec = ((double)rw * tpg) * cm[8];
    double t_busy = (t_rec + t_dram) + t_ssd;
    double t_wall = std::max(span, t_busy);
    double thr = ((double)n_w * tpg) / t_wall;
    double lat = t_busy / n_req;
    double cost = (((cm[0] + capgib[0] * cm[1]) + capgib[1] * cm[2]) + capgib[2] * cm[3]) *
                  (t_wall / 3600.0);
    obj[3 * (size_t)j + 0] = cost;
    obj[3 * (size_t)j + 1] = thr;
    obj[3 * (size_t)j + 2] = lat;
  }
  return 0;
}

// Non-dominated flags by brute force over all pairs of each segment.
// bounds (NULL or [3], NaN = none): cost <= b0, throughput >= b1, latency <= b2.
// a dominates b: a.cost <= b.cost, a.thr >= b.thr, a.lat <= b.lat, one strict.
// Returns the number of flagged rows, or -1 if an objective is NaN.
int64_t oracle_pareto(uint32_t n, const double* obj, const uint32_t* segment,
                      const double* bounds, uint8_t* flag) {
  for (uint64_t i = 0; i < 3ull * n; ++i)
    if (std::isnan(obj[i])) return -1;
  std::vector<uint8_t> feas(n, 1);
  for (uint32_t i = 0; i < n; ++i) {
    if (!bounds) break;
    const double* o = obj + 3 * (size_t)i;
    if (!std::isnan(bounds[0]) && !(o[0] <= bounds[0])) feas[i] = 0;
    if (!std::isnan(bounds[1]) && !(o[1] >= bounds[1])) feas[i] = 0;
    if (!std::isnan(bounds[2]) && !(o[2] <= bounds[2])) feas[i] = 0;
  }
  int64_t count = 0;
  for (uint32_t b = 0; b < n; ++b) {
    flag[b] = 0;
    if (!feas[b]) continue;
    const double* ob = obj + 3 * (size_t)b;
    bool dominated = false;
    for (uint32_t a = 0; a < n && !dominated; ++a) {
      if (a == b || !feas[a]) continue;
      if (segment && segment[a] != segment[b]) continue;
      const double* oa = obj + 3 * (size_t)a;
      bool le = oa[0] <= ob[0] && oa[1] >= ob[1] && oa[2] <= ob[2];
      bool lt = oa[0] < ob[0] || oa[1] > ob[1] || oa[2] < ob[2];
      dominated = le && lt;
    }
    if (!dominated) {
      flag[b] = 1;
      ++count;
    }
  }
  return count;
}

}  // extern "C"
