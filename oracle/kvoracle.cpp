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
//   oracle_replay_memo the same, replaying each distinct inclusive tier cache
//                      once (inclusive tiers are independent caches) and
//                      classifying every configuration from presence bits.
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
//   * Exclusive hierarchy with write-back demotion: a block lives in at most
//     one tier; a hit in a lower tier removes it there and promotes it to the
//     top tier; an overfull tier demotes its victim to the next tier; blocks
//     pushed past the last tier are dropped.  With LRU the demoted block
//     enters the next tier's MRU end.  With FIFO or LFU a tier takes every
//     block that enters it (a miss, a promotion, a demotion) as its newest
//     member - FIFO: the newest insertion; LFU: frequency 1, touched now,
//     the touches of the whole hierarchy being numbered in one sequence -
//     and first passes its own victims down, each taken by the next tier the
//     same way, before it admits the block.
//   * Counts: hit_k = accesses served by k; miss_k = accesses that reached k
//     (not served by a faster tier) and were not served by k; ins_k = blocks
//     that entered k; evict_k = blocks that left k for lack of room (a
//     demotion counts as an eviction of the source tier).  Evictions are
//     charged to the evicted block's group.
//
// Build: g++ -O2 -std=c++17 -ffp-contract=off -fPIC -shared -pthread
#include <algorithm>
#include <array>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <functional>
#include <memory>
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
enum Policy { P_LRU = 0, P_FIFO = 1, P_LFU = 2, P_LEAF = 3 };
enum Mode { M_INCLUSIVE = 0, M_EXCLUSIVE = 1, M_INCLUSIVE_PREFIX = 2 };

struct Block {
  uint64_t hash;
  uint32_t req;
  uint8_t w;  // granules, 1..255
  uint8_t g;  // tenant group
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
  // Take a resident block out without an eviction (a promotion).
  Block remove(uint64_t h) {
    Block b = take(h);
    used_ -= b.w;
    return b;
  }

 protected:
  // policies of the exclusive mode only (LRU, FIFO, LFU) implement it
  virtual Block take(uint64_t) { std::abort(); }
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
  Block take(uint64_t h) override {
    auto it = pos_.at(h);
    Block b = *it;
    order_.erase(it);
    pos_.erase(h);
    return b;
  }
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
  Block take(uint64_t h) override {
    auto it = pos_.at(h);
    Block b = *it;
    order_.erase(it);
    pos_.erase(h);
    return b;
  }
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
  Block take(uint64_t h) override {
    const Info in = info_.at(h);
    order_.erase(std::make_tuple(in.freq, in.last, h));
    info_.erase(h);
    return in.b;
  }
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

// Radix-tree eviction (the prefix tree of a radix KV cache, Section 3.2):
// the blocks of a request form a chain, each block's parent being the block
// accessed just before it in the same request.  A cached block is a leaf
// when no cached block has it as parent; the victim is the leaf whose latest
// access is the oldest.
class LeafTier : public Tier {
 public:
  LeafTier(uint64_t cap, const std::vector<Block>* acc) : Tier(cap), acc_(acc) {}
  bool contains(uint64_t h) const override { return node_.count(h) != 0; }
  void hit(uint64_t h, uint64_t t) override {
    Node& n = node_.at(h);
    if (n.kids == 0) {
      leaves_.erase({n.last, h});
      leaves_.insert({t, h});
    }
    n.last = t;
  }

 protected:
  struct Node {
    Block b;
    uint64_t last;
    bool has_parent;
    uint64_t parent;
    uint32_t kids;  // cached children
  };
  Block pop_victim() override {
    const auto v = *leaves_.begin();
    leaves_.erase(leaves_.begin());
    const Node n = node_.at(v.second);
    node_.erase(v.second);
    if (n.has_parent) {
      auto it = node_.find(n.parent);
      if (it != node_.end() && --it->second.kids == 0) leaves_.insert({it->second.last, n.parent});
    }
    return n.b;
  }
  void push(const Block& b, uint64_t t) override {
    Node n{b, t, false, 0, 0};
    if (t > 0 && (*acc_)[t - 1].req == b.req) {
      n.has_parent = true;
      n.parent = (*acc_)[t - 1].hash;
      auto it = node_.find(n.parent);
      if (it != node_.end() && it->second.kids++ == 0) leaves_.erase({it->second.last, n.parent});
    }
    node_[b.hash] = n;
    leaves_.insert({t, b.hash});
  }
  const std::vector<Block>* acc_;
  std::unordered_map<uint64_t, Node> node_;
  std::set<std::pair<uint64_t, uint64_t>> leaves_;  // (latest access, hash) of the leaves
};

Tier* make_tier(int policy, uint64_t cap, const std::vector<Block>* acc = nullptr) {
  if (policy == P_LRU) return new LruTier(cap);
  if (policy == P_FIFO) return new FifoTier(cap);
  if (policy == P_LEAF) return new LeafTier(cap, acc);
  return new LfuTier(cap);
}

// Radix-tree eviction needs a trace whose requests are prefix chains (a
// block is re-accessed only in a later request and always after the same
// parent block) and capacities that hold any one request (a request never
// evicts its own blocks).  Returns 0 or -4.
// Whether the requests are prefix chains, and the heaviest request.
void leaf_trace_info(const std::vector<Block>& acc, bool* chained, uint64_t* max_req_w) {
  std::unordered_map<uint64_t, std::pair<uint64_t, uint64_t>> seen;  // hash -> (parent+1, req)
  uint64_t req_w = 0;
  *chained = true;
  *max_req_w = 0;
  for (size_t i = 0; i < acc.size(); ++i) {
    const bool same = i > 0 && acc[i - 1].req == acc[i].req;
    const uint64_t par = same ? acc[i - 1].hash + 1 : 0;  // +1: 0 means no parent
    req_w = same ? req_w + acc[i].w : acc[i].w;
    *max_req_w = std::max(*max_req_w, req_w);
    auto it = seen.find(acc[i].hash);
    if (it != seen.end() && (it->second.first != par || it->second.second == acc[i].req))
      *chained = false;
    seen[acc[i].hash] = {par, acc[i].req};
  }
}

int check_leaf(const std::vector<Block>& acc, const uint64_t cap[kTiers]) {
  bool chained;
  uint64_t max_req_w;
  leaf_trace_info(acc, &chained, &max_req_w);
  if (!chained) return -4;
  for (int k = 0; k < kTiers; ++k)
    if (cap[k] && cap[k] < max_req_w) return -4;
  return 0;
}

// The disk TTL tier: a block is held for ttl[g] seconds after each of its
// accesses (g = the block's group); with a capacity it is also evicted least
// recently accessed first when full (then every group has the same ttl, so
// blocks also expire in that order).  Expired blocks are dropped by
// expire(now) before each lookup.  The tier integrates its occupancy:
// every residency adds weight x (its last access + ttl - its insertion).
struct TtlSpec {
  const double* ttl;       // [kMaxGroups] seconds, by group
  const double* req_time;  // request times
  const std::vector<Block>* acc;
};

class TtlTier : public Tier {
 public:
  TtlTier(uint64_t cap, const TtlSpec& s, uint32_t n_groups)
      : Tier(cap ? cap : ~0ull), bounded_(cap != 0), s_(s), lists_(cap ? 1 : n_groups) {}
  bool contains(uint64_t h) const override { return pos_.count(h) != 0; }
  void hit(uint64_t h, uint64_t t) override {
    auto it = pos_.at(h);
    it->last = time_of(t);
    auto& l = lists_[list_of(it->b)];
    l.splice(l.begin(), l, it);
  }
  template <class F>
  void expire(double now, F&& ev) {
    for (size_t l = 0; l < lists_.size(); ++l) {
      auto& lst = lists_[l];
      while (!lst.empty()) {
        const Entry& e = lst.back();
        const double ttl = s_.ttl[bounded_ ? 0 : l];
        if (!(e.last + ttl < now)) break;
        store_ += (double)e.b.w * ((e.last + ttl) - e.since);
        used_ -= e.b.w;
        ev(e.b);
        pos_.erase(e.b.hash);
        lst.pop_back();
      }
    }
  }
  // occupancy of the blocks still held, each until its last access + ttl
  double finish() {
    for (size_t l = 0; l < lists_.size(); ++l)
      for (const Entry& e : lists_[l])
        store_ += (double)e.b.w * ((e.last + s_.ttl[bounded_ ? 0 : l]) - e.since);
    return store_;
  }

 protected:
  struct Entry {
    Block b;
    double last, since;  // latest access, insertion (seconds)
  };
  double time_of(uint64_t t) const { return s_.req_time[(*s_.acc)[t].req]; }
  size_t list_of(const Block& b) const { return bounded_ ? 0 : b.g; }
  Block pop_victim() override {
    auto& lst = lists_[0];  // bounded: one list, least recent at the back
    Entry e = lst.back();
    lst.pop_back();
    pos_.erase(e.b.hash);
    return e.b;
  }
  void push(const Block& b, uint64_t t) override {
    const double now = time_of(t);
    auto& l = lists_[list_of(b)];
    l.push_front(Entry{b, now, now});
    pos_[b.hash] = l.begin();
  }
  bool bounded_;
  TtlSpec s_;
  std::vector<std::list<Entry>> lists_;
  std::unordered_map<uint64_t, std::list<Entry>::iterator> pos_;
  double store_ = 0.0;
};

void add(Counts& c, uint32_t g, int k, Field f, uint64_t cnt_field_weight) {
  c.v[g][k][f] += cnt_field_weight;
}

// Inclusive hierarchy over the accesses listed in `idx`; with `prefix`, a
// block is available from a tier only while its request's earlier blocks
// were.
void replay_inclusive(const std::vector<Block>& acc, const std::vector<uint32_t>& idx,
                      const uint64_t cap[kTiers], int policy, bool prefix, Counts& out,
                      const TtlSpec* ttl = nullptr, uint32_t n_groups = 1,
                      double* store = nullptr) {
  Tier* tier[kTiers] = {nullptr, nullptr, nullptr};
  TtlTier* tt = nullptr;
  for (int k = 0; k < kTiers; ++k)
    if (cap[k] > 0 && !(k == 2 && ttl)) tier[k] = make_tier(policy, cap[k], &acc);
  if (ttl) tier[2] = tt = new TtlTier(cap[2], *ttl, n_groups);
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
    if (tt)
      tt->expire(ttl->req_time[b.req], [&](const Block& v) {
        add(out, v.g, 2, F_EVICT, 1);
        add(out, v.g, 2, F_EVICT_W, v.w);
      });
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
  if (tt && store) {
    const double s = tt->finish();
    if (cap[2] == 0) *store += s;  // an unbounded tier is billed by occupancy
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

// Exclusive hierarchy with write-back demotion under FIFO or LFU over the
// accesses in `idx`: every tier is a cache of the policy; a block that enters
// a tier is its newest member (LFU: frequency 1, touch number now), and the
// tier passes its victims down before admitting it.
void replay_exclusive_policy(const std::vector<Block>& acc, const std::vector<uint32_t>& idx,
                             const uint64_t cap[kTiers], int policy, Counts& out) {
  std::vector<int> live;  // non-absent tiers, fastest first
  for (int k = 0; k < kTiers; ++k)
    if (cap[k] > 0) live.push_back(k);
  if (live.empty()) return;
  std::vector<std::unique_ptr<Tier>> tier(kTiers);
  for (int k : live) tier[k].reset(make_tier(policy, cap[k]));
  std::unordered_map<uint64_t, int> where;  // hash -> tier holding it
  uint64_t touch = 0;                       // one sequence for the hierarchy
  // block b enters live tier number li; victims go to li + 1 first
  std::function<void(size_t, const Block&)> enter = [&](size_t li, const Block& b) {
    const int k = live[li];
    tier[k]->insert(b, touch++, [&](const Block& v) {
      where.erase(v.hash);
      add(out, v.g, k, F_EVICT, 1);
      add(out, v.g, k, F_EVICT_W, v.w);
      if (li + 1 < live.size()) enter(li + 1, v);
    });
    where[b.hash] = k;
    add(out, b.g, k, F_INS, 1);
    add(out, b.g, k, F_INS_W, b.w);
  };
  const int top = live[0];
  for (uint32_t i : idx) {
    const Block& b = acc[i];
    auto it = where.find(b.hash);
    const int at = (it == where.end()) ? -1 : it->second;
    for (int k : live) {
      if (k == at) {
        add(out, b.g, k, F_HIT, 1);
        add(out, b.g, k, F_HIT_W, b.w);
        break;
      }
      add(out, b.g, k, F_MISS, 1);
      add(out, b.g, k, F_MISS_W, b.w);
    }
    if (at == top) {  // a hit in the top tier: the policy's update
      tier[top]->hit(b.hash, touch++);
      continue;
    }
    if (at >= 0) {  // a hit in a lower tier: taken out for promotion
      tier[at]->remove(b.hash);
      where.erase(b.hash);
    }
    enter(0, b);
  }
}

struct ConfigView {
  const uint64_t* cap;        // [3]
  const uint64_t* cap_group;  // [3][16]
  uint8_t mode;
  uint8_t partitioned;
  const uint8_t* policy;  // [16]
  uint8_t disk_ttl;       // tier 2 is a TTL tier
  const double* ttl;      // [16] seconds by group
};

// A disk TTL tier is supported in the inclusive LRU shared mode; a bounded
// one needs the same ttl in every group.  0, -1 (invalid) or -4.
int check_ttl(const ConfigView& c, uint32_t n_groups) {
  if (!c.disk_ttl) return 0;
  if (c.disk_ttl > 1) return -1;
  for (uint32_t g = 0; g < n_groups; ++g)
    if (!std::isfinite(c.ttl[g]) || c.ttl[g] < 0) return -1;
  if (c.mode != M_INCLUSIVE || c.partitioned || c.policy[0] != P_LRU) return -4;
  if (c.cap[2])
    for (uint32_t g = 1; g < n_groups; ++g)
      if (c.ttl[g] != c.ttl[0]) return -4;
  return 0;
}

int replay_one(const std::vector<Block>& acc, const std::vector<std::vector<uint32_t>>& by_group,
               const std::vector<uint32_t>& all, uint32_t n_groups, uint32_t w_max,
               const ConfigView& c, Counts& out, const double* req_time = nullptr,
               double* store = nullptr) {
  auto bad_cap = [&](uint64_t x) { return x > 0 && x < w_max; };
  if (const int rc = check_ttl(c, n_groups)) return rc;
  if (c.disk_ttl) {
    for (int k = 0; k < kTiers; ++k)
      if (bad_cap(c.cap[k])) return -1;
    const TtlSpec spec{c.ttl, req_time, &acc};
    replay_inclusive(acc, all, c.cap, P_LRU, false, out, &spec, n_groups, store);
    return 0;
  }
  for (uint32_t g = 0; g < (c.partitioned ? n_groups : 1u); ++g)
    if (c.policy[g] > P_LEAF) return -1;
  if (c.policy[0] == P_LEAF || (c.partitioned && std::count(c.policy, c.policy + n_groups, P_LEAF))) {
    if (c.partitioned || c.mode != M_INCLUSIVE) return -4;
    for (int k = 0; k < kTiers; ++k)
      if (bad_cap(c.cap[k])) return -1;
    if (const int rc = check_leaf(acc, c.cap)) return rc;
    replay_inclusive(acc, all, c.cap, P_LEAF, false, out);
    return 0;
  }
  if (c.partitioned) {
    for (uint32_t g = 0; g < n_groups; ++g) {
      uint64_t cg[kTiers];
      for (int k = 0; k < kTiers; ++k) {
        cg[k] = c.cap_group[k * kMaxGroups + g];
        if (bad_cap(cg[k])) return -1;
      }
      if (c.mode == M_INCLUSIVE_PREFIX) return -4;
      if (c.mode == M_EXCLUSIVE) {
        if (c.policy[g] == P_LRU) replay_exclusive(acc, by_group[g], cg, out);
        else replay_exclusive_policy(acc, by_group[g], cg, c.policy[g], out);
      } else {
        replay_inclusive(acc, by_group[g], cg, c.policy[g], false, out);
      }
    }
  } else {
    for (int k = 0; k < kTiers; ++k)
      if (bad_cap(c.cap[k])) return -1;
    if (c.mode == M_EXCLUSIVE) {
      if (c.policy[0] == P_LRU) replay_exclusive(acc, all, c.cap, out);
      else replay_exclusive_policy(acc, all, c.cap, c.policy[0], out);
    } else if (c.mode == M_INCLUSIVE_PREFIX) {
      if (c.policy[0] != P_LRU) return -4;
      replay_inclusive(acc, all, c.cap, P_LRU, true, out);
    } else {
      replay_inclusive(acc, all, c.cap, c.policy[0], false, out);
    }
  }
  return 0;
}

// ---------------------------------------------------------------------------
// Memo mode.  In the inclusive hierarchy every tier is an independent cache
// that sees every access of its partition, so what one tier does depends only
// on (partition, policy, capacity).  Memo mode replays each distinct such
// cache once, literally, keeping one presence bit per access and its own
// insert / eviction tallies, then classifies every configuration from its
// tiers' bits: served by k = present in k and in no faster present tier.
// Non-inclusive configurations take the literal path above.
// ---------------------------------------------------------------------------
struct MemoJob {
  uint32_t part;    // index into the partition lists (group g, or n_groups = shared)
  int policy;       // P_*, or -1 for a disk TTL tier
  uint64_t cap;
  double ttl[kMaxGroups] = {};  // TTL tier: seconds by group
  double store = 0.0;           // TTL tier: occupancy integral (unbounded)
  std::vector<uint64_t> bits;  // presence before the access, one bit per list entry
  uint64_t ins[kMaxGroups] = {}, ins_w[kMaxGroups] = {}, ev[kMaxGroups] = {}, ev_w[kMaxGroups] = {};
};

void memo_run(const std::vector<Block>& acc, const std::vector<uint32_t>& idx, MemoJob& j,
              const double* req_time, uint32_t n_groups) {
  TtlTier* tt = nullptr;
  TtlSpec spec{j.ttl, req_time, &acc};
  Tier* t = j.policy < 0 ? (tt = new TtlTier(j.cap, spec, n_groups))
                         : make_tier(j.policy, j.cap, &acc);
  j.bits.assign((idx.size() + 63) / 64, 0);
  for (int g = 0; g < kMaxGroups; ++g) j.ins[g] = j.ins_w[g] = j.ev[g] = j.ev_w[g] = 0;
  for (size_t q = 0; q < idx.size(); ++q) {
    const uint32_t i = idx[q];
    const Block& b = acc[i];
    if (tt)
      tt->expire(req_time[b.req], [&](const Block& v) {
        j.ev[v.g] += 1;
        j.ev_w[v.g] += v.w;
      });
    if (t->contains(b.hash)) {
      j.bits[q >> 6] |= 1ull << (q & 63);
      t->hit(b.hash, i);
    } else {
      j.ins[b.g] += 1;
      j.ins_w[b.g] += b.w;
      t->insert(b, i, [&](const Block& v) {
        j.ev[v.g] += 1;
        j.ev_w[v.g] += v.w;
      });
    }
  }
  if (tt) {
    const double st = tt->finish();
    j.store = j.cap == 0 ? st : 0.0;
  }
  delete t;
}

// Per-list masks: one bit plane per group and per weight bit.
struct ListMasks {
  std::vector<std::vector<uint64_t>> group;   // [g] -> words
  std::vector<std::vector<uint64_t>> wplane;  // [bit] -> words
  std::vector<uint64_t> valid;
};

void build_masks(const std::vector<Block>& acc, const std::vector<uint32_t>& idx,
                 uint32_t n_groups, ListMasks& m) {
  const size_t W = (idx.size() + 63) / 64;
  m.group.assign(n_groups, std::vector<uint64_t>(W, 0));
  m.wplane.assign(8, std::vector<uint64_t>(W, 0));
  m.valid.assign(W, 0);
  for (size_t q = 0; q < idx.size(); ++q) {
    const Block& b = acc[idx[q]];
    const uint64_t bit = 1ull << (q & 63);
    m.valid[q >> 6] |= bit;
    m.group[b.g][q >> 6] |= bit;
    for (int p = 0; p < 8; ++p)
      if ((b.w >> p) & 1u) m.wplane[p][q >> 6] |= bit;
  }
}

uint64_t popc(uint64_t x) { return (uint64_t)__builtin_popcountll(x); }

// Adds the (hit, miss) counts and weights of one partition of one
// configuration: tiers[k] = job or NULL (absent).
void memo_classify(const ListMasks& m, uint32_t n_groups, const MemoJob* tiers[kTiers],
                   Counts& out) {
  const size_t W = m.valid.size();
  bool wp[8];
  for (int p = 0; p < 8; ++p) {
    wp[p] = false;
    for (size_t x = 0; x < W && !wp[p]; ++x) wp[p] = m.wplane[p][x] != 0;
  }
  for (size_t x = 0; x < W; ++x) {
    uint64_t seen = 0;  // present in some faster (or this) present tier
    for (int k = 0; k < kTiers; ++k) {
      if (!tiers[k]) continue;
      const uint64_t pk = tiers[k]->bits[x];
      const uint64_t hit = pk & ~seen;
      seen |= pk;
      const uint64_t miss = m.valid[x] & ~seen;
      for (uint32_t g = 0; g < n_groups; ++g) {
        const uint64_t gm = m.group[g][x];
        const uint64_t h = hit & gm, ms = miss & gm;
        if (!(h | ms)) continue;
        out.v[g][k][F_HIT] += popc(h);
        out.v[g][k][F_MISS] += popc(ms);
        for (int p = 0; p < 8; ++p) {
          if (!wp[p]) continue;
          out.v[g][k][F_HIT_W] += popc(h & m.wplane[p][x]) << p;
          out.v[g][k][F_MISS_W] += popc(ms & m.wplane[p][x]) << p;
        }
      }
    }
  }
  for (int k = 0; k < kTiers; ++k) {
    if (!tiers[k]) continue;
    for (uint32_t g = 0; g < n_groups; ++g) {
      out.v[g][k][F_INS] += tiers[k]->ins[g];
      out.v[g][k][F_INS_W] += tiers[k]->ins_w[g];
      out.v[g][k][F_EVICT] += tiers[k]->ev[g];
      out.v[g][k][F_EVICT_W] += tiers[k]->ev_w[g];
    }
  }
}

template <class F>
void parallel_for(uint32_t n, uint32_t n_threads, F&& f) {
  std::atomic<uint32_t> next{0};
  auto work = [&]() {
    for (;;) {
      const uint32_t j = next.fetch_add(1);
      if (j >= n) break;
      f(j);
    }
  };
  const uint32_t nt = std::max<uint32_t>(1, std::min<uint32_t>(n_threads, n));
  std::vector<std::thread> th;
  for (uint32_t t = 1; t < nt; ++t) th.emplace_back(work);
  work();
  for (auto& t : th) t.join();
}

}  // namespace

extern "C" {

// Replays every configuration literally.  counts: uint64[n_cfg][n_groups][3][8].
// req: request of every access (NULL: one request per access).  Returns 0,
// or -1 for an invalid capacity (between 0 and the largest block), -4 for a
// prefix hierarchy with a policy other than LRU (or a partitioned one), for
// radix-tree eviction outside the shared inclusive mode, or for a disk TTL
// tier outside the shared inclusive LRU mode, -2 for bad sizes.
int oracle_replay(uint64_t n, const uint64_t* hash, const uint8_t* group, const uint8_t* weight,
                  const uint32_t* req, uint32_t n_groups, uint32_t n_cfg, const uint64_t* cap,
                  const uint64_t* cap_group, const uint8_t* mode, const uint8_t* partitioned,
                  const uint8_t* policy, const uint8_t* disk_ttl, const double* ttl,
                  const double* req_time, uint32_t n_threads, uint64_t* counts, double* store) {
  if (n_groups < 1 || n_groups > (uint32_t)kMaxGroups) return -2;
  std::vector<Block> acc(n);
  std::vector<std::vector<uint32_t>> by_group(n_groups);
  std::vector<uint32_t> all(n);
  uint32_t w_max = 1;
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t g = group ? group[i] : 0;
    uint32_t w = weight ? weight[i] : 1;
    if (g >= n_groups || w == 0) return -2;
    acc[i] = Block{hash[i], req ? req[i] : (uint32_t)i, (uint8_t)w, (uint8_t)g};
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
                   partitioned[j], policy + kMaxGroups * (size_t)j, disk_ttl[j],
                   ttl + kMaxGroups * (size_t)j};
      double st = 0.0;
      int rc = replay_one(acc, by_group, all, n_groups, w_max, v, *c, req_time, &st);
      if (rc != 0) status.store(rc);
      store[j] = st;
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
// bw_dram, ssd_bw_base, ssd_bw_per_gib, ssd_bw_max, t_prefill_per_token,
// n_media, then per medium (price_gib_hour, bw_base, bw_per_gib, bw_max)].
// The counts enter as granule totals over groups: H_w[k] = sum_g hit_w,
// I_w2 = sum_g ins_w of the SSD tier; recompute R_w = N_w - sum_k H_w[k].
//   capGiB[k] = cap[k] * gb / 2^30, except an unbounded disk TTL tier:
//               capGiB[2] = (store * gb / 2^30) / span (mean occupancy; 0 if span = 0)
//   (p2, base, per_gib, max) = the disk's price and bandwidth terms, from
//               media[medium] when n_media > 0
//   bw_ssd    = min(base + per_gib * capGiB[2], max)
//   t_dram    = H_w[1] * gb / bw_dram
//   t_ssd     = (H_w[2] + I_w2) * gb / bw_ssd
//   t_rec     = R_w * tpg * t_prefill_per_token
//   T_busy    = t_rec + t_dram + t_ssd;   T_wall = max(span, T_busy)
//   throughput = N_w * tpg / T_wall;      latency = T_busy / n_req
//   cost = (price_gpu + capGiB[0] * p0 + capGiB[1] * p1 + capGiB[2] * p2) * T_wall / 3600
int oracle_objectives(uint32_t n_cfg, const uint64_t* cap, const uint64_t* counts,
                      uint32_t n_groups, const double* cm, double gb, double tpg,
                      double span, double n_req, uint64_t n_w, const uint8_t* disk_ttl,
                      const uint8_t* medium, const double* store, double* obj) {
  const double kGiB = 1073741824.0;
  const uint32_t n_media = (uint32_t)cm[9];
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
    if (disk_ttl[j] && cap[3 * (size_t)j + 2] == 0)
      capgib[2] = span > 0 ? ((store[j] * gb) / kGiB) / span : 0.0;
    double p2 = cm[3], base = cm[5], per_gib = cm[6], bmax = cm[7];
    if (n_media) {
      const double* md = cm + 10 + 4 * (size_t)medium[j];
      p2 = md[0];
      base = md[1];
      per_gib = md[2];
      bmax = md[3];
    }
    double bw_ssd = std::min(base + per_gib * capgib[2], bmax);
    double t_dram = ((double)hw[1] * gb) / cm[4];
    double t_ssd = ((double)(hw[2] + iw2) * gb) / bw_ssd;
    double t_rec = ((double)rw * tpg) * cm[8];
    double t_busy = (t_rec + t_dram) + t_ssd;
    double t_wall = std::max(span, t_busy);
    double thr = ((double)n_w * tpg) / t_wall;
    double lat = t_busy / n_req;
    double cost = (((cm[0] + capgib[0] * cm[1]) + capgib[1] * cm[2]) + capgib[2] * p2) *
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

extern "C" {

// Memo-mode replay: the same results as oracle_replay (same arguments and
// return codes), with every distinct inclusive tier cache (partition,
// policy, capacity) replayed once and shared by the configurations that
// use it.  Exclusive and prefix-reuse configurations replay literally.
int oracle_replay_memo(uint64_t n, const uint64_t* hash, const uint8_t* group,
                       const uint8_t* weight, const uint32_t* req, uint32_t n_groups,
                       uint32_t n_cfg, const uint64_t* cap, const uint64_t* cap_group,
                       const uint8_t* mode, const uint8_t* partitioned, const uint8_t* policy,
                       const uint8_t* disk_ttl, const double* ttl, const double* req_time,
                       uint32_t n_threads, uint64_t* counts, double* store) {
  if (n_groups < 1 || n_groups > (uint32_t)kMaxGroups) return -2;
  std::vector<Block> acc(n);
  // partition lists: [g] = group g's accesses, [n_groups] = every access
  // (with one group the two are the same list, kept once)
  std::vector<std::vector<uint32_t>> lists(n_groups + 1);
  const uint32_t all_list = n_groups == 1 ? 0u : n_groups;
  uint32_t w_max = 1;
  for (uint64_t i = 0; i < n; ++i) {
    uint32_t g = group ? group[i] : 0;
    uint32_t w = weight ? weight[i] : 1;
    if (g >= n_groups || w == 0) return -2;
    acc[i] = Block{hash[i], req ? req[i] : (uint32_t)i, (uint8_t)w, (uint8_t)g};
    lists[g].push_back((uint32_t)i);
    if (all_list != 0) lists[all_list].push_back((uint32_t)i);
    w_max = std::max(w_max, w);
  }
  std::vector<std::vector<uint32_t>> by_group;
  if (n_groups > 1) by_group.assign(lists.begin(), lists.begin() + n_groups);
  auto bad_cap = [&](uint64_t x) { return x > 0 && x < w_max; };

  // plan: distinct (partition, policy, capacity) caches of the inclusive configs
  std::vector<MemoJob> jobs;
  bool leaf_known = false, leaf_chained = false;
  uint64_t leaf_max_w = 0;
  // per config and partition, the job of each tier (-1 absent)
  std::vector<std::vector<std::array<int64_t, kTiers>>> use(n_cfg);
  std::vector<uint8_t> literal(n_cfg, 0);
  auto job_of = [&](uint32_t part, int pol, uint64_t c, const double* tl) -> int64_t {
    for (size_t q = 0; q < jobs.size(); ++q) {
      const MemoJob& j = jobs[q];
      if (j.part != part || j.policy != pol || j.cap != c) continue;
      if (pol < 0 && !std::equal(j.ttl, j.ttl + n_groups, tl)) continue;
      return (int64_t)q;
    }
    MemoJob j;
    j.part = part;
    j.policy = pol;
    j.cap = c;
    if (pol < 0) std::copy(tl, tl + n_groups, j.ttl);
    jobs.push_back(std::move(j));
    return (int64_t)jobs.size() - 1;
  };
  for (uint32_t c = 0; c < n_cfg; ++c) {
    const uint64_t* cp = cap + 3 * (size_t)c;
    const uint64_t* cg = cap_group + 3 * kMaxGroups * (size_t)c;
    const uint8_t* pol = policy + kMaxGroups * (size_t)c;
    const double* tl = ttl + kMaxGroups * (size_t)c;
    for (int k = 0; k < kTiers; ++k)
      if (bad_cap(cp[k])) return -1;
    const ConfigView cv{cp, cg, mode[c], partitioned[c], pol, disk_ttl[c], tl};
    if (const int rc = check_ttl(cv, n_groups)) return rc;
    for (uint32_t g = 0; g < (partitioned[c] ? n_groups : 1u); ++g)
      if (pol[g] > P_LEAF) return -1;
    if (pol[0] == P_LEAF || (partitioned[c] && std::count(pol, pol + n_groups, P_LEAF))) {
      if (partitioned[c] || mode[c] != M_INCLUSIVE) return -4;
      if (!leaf_known) {
        leaf_trace_info(acc, &leaf_chained, &leaf_max_w);
        leaf_known = true;
      }
      if (!leaf_chained) return -4;
      for (int k = 0; k < kTiers; ++k)
        if (cp[k] && cp[k] < leaf_max_w) return -4;
    }
    if (mode[c] != M_INCLUSIVE) {
      literal[c] = 1;
      continue;
    }
    if (partitioned[c]) {
      for (uint32_t g = 0; g < n_groups; ++g) {
        std::array<int64_t, kTiers> t{-1, -1, -1};
        for (int k = 0; k < kTiers; ++k) {
          const uint64_t x = cg[k * kMaxGroups + g];
          if (bad_cap(x)) return -1;
          if (x) t[k] = job_of(g, pol[g], x, nullptr);
        }
        use[c].push_back(t);
      }
    } else {
      std::array<int64_t, kTiers> t{-1, -1, -1};
      for (int k = 0; k < kTiers; ++k)
        if (cp[k] && !(k == 2 && disk_ttl[c])) t[k] = job_of(all_list, pol[0], cp[k], nullptr);
      if (disk_ttl[c]) t[2] = job_of(all_list, -1, cp[2], tl);
      use[c].push_back(t);
    }
  }

  // replay every distinct cache once
  parallel_for((uint32_t)jobs.size(), n_threads, [&](uint32_t q) {
    memo_run(acc, lists[jobs[q].part], jobs[q], req_time, n_groups);
  });
  std::vector<ListMasks> masks(n_groups + 1);
  parallel_for(n_groups + 1, n_threads, [&](uint32_t p) {
    if (p == 0 || p < n_groups || p == all_list) build_masks(acc, lists[p], n_groups, masks[p]);
  });

  // classify every configuration
  std::atomic<int> status{0};
  parallel_for(n_cfg, n_threads, [&](uint32_t c) {
    Counts* out = new Counts;
    std::fill(&out->v[0][0][0], &out->v[0][0][0] + kMaxGroups * kTiers * kFields, 0);
    store[c] = 0.0;
    if (literal[c]) {
      ConfigView v{cap + 3 * (size_t)c, cap_group + 3 * kMaxGroups * (size_t)c, mode[c],
                   partitioned[c], policy + kMaxGroups * (size_t)c, disk_ttl[c],
                   ttl + kMaxGroups * (size_t)c};
      const int rc = replay_one(acc, n_groups > 1 ? by_group : lists, lists[all_list], n_groups,
                                w_max, v, *out, req_time, &store[c]);
      if (rc != 0) status.store(rc);
    } else {
      for (size_t u = 0; u < use[c].size(); ++u) {
        const uint32_t part = partitioned[c] ? (uint32_t)u : all_list;
        const MemoJob* t[kTiers];
        for (int k = 0; k < kTiers; ++k) t[k] = use[c][u][k] >= 0 ? &jobs[use[c][u][k]] : nullptr;
        memo_classify(masks[part], n_groups, t, *out);
        if (disk_ttl[c] && t[2]) store[c] += t[2]->store;
      }
    }
    uint64_t* dst = counts + (size_t)c * n_groups * kTiers * kFields;
    for (uint32_t g = 0; g < n_groups; ++g)
      for (int k = 0; k < kTiers; ++k)
        for (int f = 0; f < kFields; ++f) dst[(g * kTiers + k) * kFields + f] = out->v[g][k][f];
    delete out;
  });
  return status.load();
}

}  // extern "C"
