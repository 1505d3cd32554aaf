// k_canon.hip - trace canonicalisation.
//
// The paper's simulator consumes traces of salted KV-block hashes, 16 tokens
// per block (Section 3.3, trace description; Section 4.1, simulator).  Every
// later step needs, per access, the position of the previous and of the next
// access to the same block, and a dense id per distinct block.  They come
// from one stable LSD radix sort of (hash, position) pairs: equal hashes end
// up adjacent and in trace order, so neighbours in the sorted array are the
// previous / next occurrences.
//
// Radix pass layout: 4096-item tiles (256 threads x 16 items).  Ranking is
// stable and needs no shared sort buffer: each 64-lane wavefront ranks 64
// consecutive items per round by matching digits with 8 ballots, keeping a
// running count per digit in LDS; waves own contiguous quarters of the tile.
#include "kv_device.h"
#include "kv_internal.h"

namespace kv {
namespace {

constexpr int kRsNT = 1024;
constexpr int kRsItems = 8;
constexpr uint32_t kRsTile = kRsNT * kRsItems;  // 8192
constexpr int kRsDigits = 256;                   // 8-bit digits
constexpr int kRsWaves = kRsNT / 64;

enum : uint32_t {
  kErrGroup = 1u,
  kErrWeight = 2u,
  kErrReq = 4u,
  kErrInconsistent = 8u,
  kErrTime = 16u,
};

struct DevStats {
  unsigned long long n_g[KV_MAX_GROUPS];
  unsigned long long n_w_g[KV_MAX_GROUPS];
  unsigned long long u_g[KV_MAX_GROUPS];
  unsigned long long u_w_g[KV_MAX_GROUPS];
  unsigned long long mult;
  uint32_t w_min, w_max, err, pad;
};

// Per access: check group / weight / request index, copy group and weight
// into the trace order, seed the sort with (hash, position), accumulate
// per-group totals.
__global__ __launch_bounds__(256) void k_validate(const uint64_t* __restrict__ hash,
                                                  const uint32_t* __restrict__ req,
                                                  const uint8_t* __restrict__ group,
                                                  const uint8_t* __restrict__ weight, uint64_t n,
                                                  uint32_t n_req, uint32_t n_groups,
                                                  uint8_t* __restrict__ g8, uint8_t* __restrict__ w8,
                                                  uint64_t* __restrict__ keys,
                                                  uint32_t* __restrict__ vals, DevStats* st) {
  __shared__ unsigned long long sn[KV_MAX_GROUPS], sw[KV_MAX_GROUPS];
  __shared__ uint32_t smin, smax, serr;
  if (threadIdx.x < KV_MAX_GROUPS) {
    sn[threadIdx.x] = 0;
    sw[threadIdx.x] = 0;
  }
  if (threadIdx.x == 0) {
    smin = 0xFFFFFFFFu;
    smax = 0;
    serr = 0;
  }
  __syncthreads();
  uint32_t err = 0, wmin = 0xFFFFFFFFu, wmax = 0;
  // per-group totals add up in registers while the thread's group stays
  // the same (always, with one group) and go to LDS when it changes: LDS
  // atomics of a wavefront on one address are taken one lane at a time
  uint32_t cg = 0xFFFFFFFFu;
  unsigned long long cn = 0, cw = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    uint32_t g = group ? group[i] : 0u;
    uint32_t w = weight ? weight[i] : 1u;
    uint32_t r = req[i];
    if (g >= n_groups) { err |= kErrGroup; g = 0; }
    if (w == 0) err |= kErrWeight;
    if (r >= n_req || (i + 1 < n && req[i + 1] < r)) err |= kErrReq;
    g8[i] = (uint8_t)g;
    w8[i] = (uint8_t)w;
    keys[i] = hash[i];
    vals[i] = (uint32_t)i;
    if (g != cg) {
      if (cn) {
        atomicAdd(&sn[cg], cn);
        atomicAdd(&sw[cg], cw);
      }
      cg = g;
      cn = 0;
      cw = 0;
    }
    ++cn;
    cw += w;
    wmin = min(wmin, w);
    wmax = max(wmax, w);
  }
  if (cn) {
    atomicAdd(&sn[cg], cn);
    atomicAdd(&sw[cg], cw);
  }
  atomicMin(&smin, wmin);
  atomicMax(&smax, wmax);
  if (err) atomicOr(&serr, err);
  __syncthreads();
  if (threadIdx.x < n_groups) {
    if (sn[threadIdx.x]) atomicAdd(&st->n_g[threadIdx.x], sn[threadIdx.x]);
    if (sw[threadIdx.x]) atomicAdd(&st->n_w_g[threadIdx.x], sw[threadIdx.x]);
  }
  if (threadIdx.x == 0) {
    atomicMin(&st->w_min, smin);
    atomicMax(&st->w_max, smax);
    if (serr) atomicOr(&st->err, serr);
  }
}

__global__ void k_check_times(const double* __restrict__ t, uint32_t n_req, DevStats* st) {
  uint32_t bad = 0;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i + 1 < n_req;
       i += gridDim.x * blockDim.x)
    if (!(t[i] <= t[i + 1])) bad = 1;
  if (n_req && blockIdx.x == 0 && threadIdx.x == 0 && t[0] != t[0]) bad = 1;
  if (bad) atomicOr(&st->err, kErrTime);
}

// Digit histogram of one tile: counts[digit * ntiles + tile].
__global__ __launch_bounds__(kRsNT) void k_rs_count(const uint64_t* __restrict__ keys, uint64_t n,
                                                    int shift, uint32_t* __restrict__ counts,
                                                    uint32_t ntiles) {
  __shared__ uint32_t h[kRsDigits];
  if (threadIdx.x < kRsDigits) h[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t base = (uint64_t)blockIdx.x * kRsTile;
  const uint32_t lane = lane_id();
#pragma unroll
  for (int e = 0; e < kRsItems; ++e) {
    const uint64_t i = base + (uint64_t)e * kRsNT + threadIdx.x;
    const bool valid = i < n;
    const uint32_t d = valid ? (uint32_t)(keys[i] >> shift) & 255u : 0u;
    // lanes of the wavefront with the same digit (8 ballots): the highest
    // adds their number, so no two lanes of one atomic share an address
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    if (valid && (peers >> lane) == 1ull) atomicAdd(&h[d], (uint32_t)__popcll(peers));
  }
  __syncthreads();
  if (threadIdx.x < kRsDigits) counts[(uint64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one tile given the exclusive digit offsets.  The tile
// is first put in digit order in LDS, then written out position by position,
// so that neighbouring threads write neighbouring words of one digit's run.
__global__ __launch_bounds__(kRsNT) void k_rs_scatter(const uint64_t* __restrict__ kin,
                                                      const uint32_t* __restrict__ vin,
                                                      uint64_t* __restrict__ kout,
                                                      uint32_t* __restrict__ vout, uint64_t n,
                                                      int shift,
                                                      const uint32_t* __restrict__ offsets,
                                                      uint32_t ntiles) {
  __shared__ uint32_t wcnt[kRsWaves][kRsDigits];
  __shared__ uint32_t gbase[kRsDigits];   // the digit's first output position, less its tile start
  __shared__ uint32_t red[kRsWaves];
  __shared__ uint64_t sk[kRsTile];
  __shared__ uint32_t sv[kRsTile];
  const int w = threadIdx.x / 64;
  const uint32_t lane = lane_id();
  for (int d = threadIdx.x; d < kRsWaves * kRsDigits; d += kRsNT) (&wcnt[0][0])[d] = 0;
  const uint32_t g0 =
      threadIdx.x < kRsDigits ? offsets[(uint64_t)threadIdx.x * ntiles + blockIdx.x] : 0u;
  __syncthreads();
  const uint64_t t0 = (uint64_t)blockIdx.x * kRsTile;
  const uint64_t base = t0 + (uint64_t)w * (kRsItems * 64);
  uint64_t k[kRsItems];
  uint32_t v[kRsItems], d[kRsItems], rk[kRsItems];
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int r = 0; r < kRsItems; ++r) {
    const uint64_t i = base + (uint64_t)r * 64 + lane;
    const bool valid = i < n;
    k[r] = valid ? kin[i] : 0ull;
    v[r] = valid ? vin[i] : 0u;
    d[r] = (uint32_t)(k[r] >> shift) & 255u;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d[r] >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    const uint32_t before = (uint32_t)__popcll(peers & lt);
    const uint32_t cnt = (uint32_t)__popcll(peers);
    const uint32_t cur = wcnt[w][d[r]];
    rk[r] = cur + before;
    const bool leader = valid && ((peers >> lane) == 1ull);
    if (leader) wcnt[w][d[r]] = cur + cnt;
  }
  __syncthreads();
  {
    // per digit (one per thread of the first kRsDigits): the tile's count,
    // its start in the tile's digit order (a block scan), and each wave's
    // start inside it
    const int dg = threadIdx.x;
    const bool has = dg < kRsDigits;
    uint32_t tot = 0;
    if (has) {
#pragma unroll
      for (int ww = 0; ww < kRsWaves; ++ww) tot += wcnt[ww][dg];
    }
    uint32_t all;
    const uint32_t ls = block_excl_scan_u32<kRsNT, false>(tot, red, all);
    if (has) {
      uint32_t run = ls;
#pragma unroll
      for (int ww = 0; ww < kRsWaves; ++ww) {
        const uint32_t c = wcnt[ww][dg];
        wcnt[ww][dg] = run;
        run += c;
      }
      gbase[dg] = g0 - ls;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kRsItems; ++r) {
    const uint64_t i = base + (uint64_t)r * 64 + lane;
    if (i < n) {
      const uint32_t lp = wcnt[w][d[r]] + rk[r];
      sk[lp] = k[r];
      sv[lp] = v[r];
    }
  }
  __syncthreads();
  const uint32_t m = (uint32_t)min<uint64_t>(kRsTile, n - t0);
  for (uint32_t p = threadIdx.x; p < m; p += kRsNT) {
    const uint64_t key = sk[p];
    const uint32_t dst = gbase[(uint32_t)(key >> shift) & 255u] + p;
    kout[dst] = key;
    vout[dst] = sv[p];
  }
}

// The sort runs its passes over the hashes' high 32 bits only; hashes that
// share them sit interleaved (in position order) in one run of equal high
// bits, and only such mixed runs are sorted again, by (run, low 32 bits).
// Runs of equal high bits: a flag at each run's first element.
__global__ __launch_bounds__(256) void k_hi_starts(const uint64_t* __restrict__ K, uint64_t n,
                                                   uint32_t* __restrict__ start) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x)
    start[k] = (k == 0 || (K[k - 1] >> 32) != (K[k] >> 32)) ? 1u : 0u;
}

// A run (0-based id = inclusive run count - 1) is mixed when two neighbours
// in it differ in their low bits.
__global__ __launch_bounds__(256) void k_hi_mixed(const uint64_t* __restrict__ K, uint64_t n,
                                                  const uint32_t* __restrict__ runincl,
                                                  uint32_t* __restrict__ mixed) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x + 1; k < n;
       k += (uint64_t)gridDim.x * blockDim.x)
    if (K[k - 1] != K[k] && (K[k - 1] >> 32) == (K[k] >> 32)) mixed[runincl[k] - 1u] = 1u;
}

// Elements of mixed runs.
__global__ __launch_bounds__(256) void k_hi_inmixed(const uint32_t* __restrict__ runincl,
                                                    const uint32_t* __restrict__ mixed,
                                                    uint64_t n, uint32_t* __restrict__ flag) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x)
    flag[k] = mixed[runincl[k] - 1u];
}

// Gathers the elements of mixed runs in order: key (run id, low bits),
// position, and where the element sits.
__global__ __launch_bounds__(256) void k_hi_gather(const uint64_t* __restrict__ K,
                                                   const uint32_t* __restrict__ V, uint64_t n,
                                                   const uint32_t* __restrict__ runincl,
                                                   const uint32_t* __restrict__ flag,
                                                   const uint32_t* __restrict__ at,
                                                   uint64_t* __restrict__ ck,
                                                   uint32_t* __restrict__ cv,
                                                   uint32_t* __restrict__ ci) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x) {
    if (!flag[k]) continue;
    const uint32_t j = at[k];
    ck[j] = ((uint64_t)(runincl[k] - 1u) << 32) | (K[k] & 0xFFFFFFFFull);
    cv[j] = V[k];
    ci[j] = (uint32_t)k;
  }
}

// Puts the sorted elements of the mixed runs back in their runs' slots (the
// gathered slots of a run are contiguous and keep their order).
__global__ __launch_bounds__(256) void k_hi_scatter(const uint64_t* __restrict__ ck,
                                                    const uint32_t* __restrict__ cv,
                                                    const uint32_t* __restrict__ ci, uint64_t m,
                                                    uint64_t* __restrict__ K,
                                                    uint32_t* __restrict__ V) {
  for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < m;
       j += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t k = ci[j];
    K[k] = (K[k] & 0xFFFFFFFF00000000ull) | (ck[j] & 0xFFFFFFFFull);
    V[k] = cv[j];
  }
}

// Run starts in hash order: the first element of every group of equal
// hashes (its first occurrence: ties in the sort go by position).
__global__ __launch_bounds__(256) void k_run_flags(const uint64_t* __restrict__ K, uint64_t n,
                                                   uint32_t* __restrict__ newflag) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x)
    newflag[k] = (k == 0 || K[k - 1] != K[k]) ? 1u : 0u;
}

// Neighbours in hash order are the previous / next occurrences.  Both links
// of a position and its block id go out in one 16-byte scatter (link, next,
// id), split into the three arrays by a pass in position order.  Dense block
// ids follow the order of first occurrence (the rank of the block's first
// position among all first positions), so that blocks met close together in
// the trace sit close together in the per-block state arrays.  At a run
// start the block's weight and group go into the per-block tables.
__global__ __launch_bounds__(256) void k_links(const uint64_t* __restrict__ K,
                                               const uint32_t* __restrict__ V, uint64_t n,
                                               const uint32_t* __restrict__ incl,
                                               const uint32_t* __restrict__ newflag,
                                               const uint32_t* __restrict__ firstpos,
                                               const uint32_t* __restrict__ fincl,
                                               uint4* __restrict__ kn,
                                               uint8_t* __restrict__ blk_w,
                                               uint8_t* __restrict__ blk_g,
                                               uint32_t* __restrict__ runstart,
                                               const uint8_t* __restrict__ w8,
                                               const uint8_t* __restrict__ g8, DevStats* st) {
  __shared__ unsigned long long su[KV_MAX_GROUPS], suw[KV_MAX_GROUPS];
  if (threadIdx.x < KV_MAX_GROUPS) {
    su[threadIdx.x] = 0;
    suw[threadIdx.x] = 0;
  }
  __syncthreads();
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t h = K[k];
    const uint32_t pos = V[k];
    const bool sp = newflag[k] == 0u;
    const bool sn = k + 1 < n && K[k + 1] == h;
    const uint32_t key = sp ? V[k - 1] + 1u : 0u;
    const uint32_t nx = sn ? V[k + 1] : kNone;
    const uint32_t run = incl[k] - 1u;
    const uint32_t id = fincl[firstpos[run]] - 1u;
    // a streaming store: each record lands alone in its line
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 rec = {key, nx, id, 0u};
    __builtin_nontemporal_store(rec, reinterpret_cast<u32x4*>(kn) + pos);
    if (!sp) {
      const uint8_t w = w8[pos], g = g8[pos];
      blk_w[id] = w;
      blk_g[id] = g;
      runstart[run] = (uint32_t)k;
      atomicAdd(&su[g], 1ull);
      atomicAdd(&suw[g], (unsigned long long)w);
    }
  }
  __syncthreads();
  if (threadIdx.x < KV_MAX_GROUPS) {
    if (su[threadIdx.x]) atomicAdd(&st->u_g[threadIdx.x], su[threadIdx.x]);
    if (suw[threadIdx.x]) atomicAdd(&st->u_w_g[threadIdx.x], suw[threadIdx.x]);
  }
}

__global__ __launch_bounds__(256) void k_split_links(const uint4* __restrict__ kn, uint64_t n,
                                                     uint32_t* __restrict__ key,
                                                     uint32_t* __restrict__ nxt,
                                                     uint32_t* __restrict__ bid) {
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n;
       p += (uint64_t)gridDim.x * blockDim.x) {
    const uint4 x = kn[p];
    key[p] = x.x;
    nxt[p] = x.y;
    bid[p] = x.z;
  }
}

// Every access carries its block's weight and group (those of the block's
// first occurrence): read in position order, against the per-block tables.
__global__ __launch_bounds__(256) void k_check_blocks(const uint32_t* __restrict__ bid,
                                                      const uint8_t* __restrict__ blk_w,
                                                      const uint8_t* __restrict__ blk_g,
                                                      const uint8_t* __restrict__ w8,
                                                      const uint8_t* __restrict__ g8, uint64_t n,
                                                      DevStats* st) {
  bool bad = false;
  for (uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n;
       p += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t id = bid[p];
    bad |= w8[p] != blk_w[id] || g8[p] != blk_g[id];
  }
  if (__ballot(bad) != 0ull && lane_id() == 0) atomicOr(&st->err, (uint32_t)kErrInconsistent);
}

// Position of each hash group's first element (its first occurrence), and
// a flag at that position in trace order.
__global__ __launch_bounds__(256) void k_first_pos(const uint32_t* __restrict__ V,
                                                   const uint32_t* __restrict__ incl,
                                                   const uint32_t* __restrict__ newflag,
                                                   uint64_t n, uint32_t* __restrict__ firstpos,
                                                   uint32_t* __restrict__ firstflag) {
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x)
    if (newflag[k]) {
      const uint32_t pos = V[k];
      firstpos[incl[k] - 1u] = pos;
      firstflag[pos] = 1u;
    }
}

__global__ __launch_bounds__(256) void k_mult(const uint32_t* __restrict__ incl,
                                              const uint32_t* __restrict__ newflag, uint64_t n,
                                              const uint32_t* __restrict__ runstart,
                                              DevStats* st) {
  unsigned long long best = 0;
  for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (uint64_t)gridDim.x * blockDim.x) {
    const bool last = (k + 1 == n) || newflag[k + 1];
    if (last) {
      const uint32_t id = incl[k] - 1u;
      best = max(best, (unsigned long long)(k - runstart[id] + 1));
    }
  }
#pragma unroll
  for (int dd = 32; dd >= 1; dd >>= 1) best = max(best, (unsigned long long)__shfl_xor(best, dd, 64));
  // one global atomic per block: atomics of many blocks on one address
  // are taken one at a time
  __shared__ unsigned long long sb[256 / 64];
  if (lane_id() == 0) sb[threadIdx.x / 64] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long m = 0;
    for (int w = 0; w < 256 / 64; ++w) m = max(m, sb[w]);
    if (m) atomicMax(&st->mult, m);
  }
}

// Partitioned order: inverse permutation and remapped links.
__global__ __launch_bounds__(256) void k_part_inverse(const uint32_t* __restrict__ perm,
                                                      uint64_t n, uint32_t* __restrict__ ppos) {
  for (uint64_t q = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n;
       q += (uint64_t)gridDim.x * blockDim.x)
    ppos[perm[q]] = (uint32_t)q;
}

__global__ __launch_bounds__(256) void k_part_build(
    const uint32_t* __restrict__ perm, const uint32_t* __restrict__ ppos, uint64_t n,
    const uint32_t* __restrict__ key, const uint32_t* __restrict__ nxt,
    const uint32_t* __restrict__ bid, const uint8_t* __restrict__ w8,
    const uint8_t* __restrict__ g8, uint32_t* __restrict__ pkey, uint32_t* __restrict__ pnxt,
    uint32_t* __restrict__ pbid, uint8_t* __restrict__ pw, uint8_t* __restrict__ pg) {
  for (uint64_t q = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n;
       q += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t i = perm[q];
    const uint32_t kk = key[i];
    const uint32_t nx = nxt[i];
    pkey[q] = kk ? ppos[kk - 1u] + 1u : 0u;
    pnxt[q] = (nx != kNone) ? ppos[nx] : kNone;
    pbid[q] = bid[i];
    pw[q] = w8[i];
    pg[q] = g8[i];
  }
}

__global__ void k_group_keys(const uint8_t* __restrict__ g8, uint64_t n,
                             uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (uint64_t)gridDim.x * blockDim.x) {
    keys[i] = g8[i];
    vals[i] = (uint32_t)i;
  }
}

uint32_t grid_of(uint64_t m, uint64_t cap = 32768) {
  uint64_t g = (m + 255) / 256;
  if (g > cap) g = cap;
  return (uint32_t)(g ? g : 1);
}

// Grids of the kernels that end with global atomics on one address per
// block (trace statistics): a few blocks per compute unit, so that few
// atomics queue on each address.
constexpr uint64_t kReduceGrid = 1024;

// Traces from this length on are sorted by their hashes' high bits first;
// KVCFG_TEST_HIGH_FIRST=1 (read at every load) takes that path for any
// length, so that short test traces reach it.
constexpr uint64_t kHighFirstN = 1ull << 23;
bool high_first_forced() {
  const char* e = std::getenv("KVCFG_TEST_HIGH_FIRST");
  return e && e[0] == '1';
}

// One stable LSD pass over (keys, vals) on digit `shift`.
kv_status radix_pass(const uint64_t* kin, const uint32_t* vin, uint64_t* kout, uint32_t* vout,
                     uint64_t n, int shift, uint32_t* counts, uint32_t* scan_scratch,
                     hipStream_t s) {
  const uint32_t ntiles = div_up(n, kRsTile);
  hipLaunchKernelGGL(k_rs_count, dim3(ntiles), dim3(kRsNT), 0, s, kin, n, shift, counts, ntiles);
  KV_HIP(hipGetLastError());
  kv_status st = scan_u32(counts, counts, (uint64_t)ntiles * 256, false, scan_scratch, s);
  if (st != KV_OK) return st;
  hipLaunchKernelGGL(k_rs_scatter, dim3(ntiles), dim3(kRsNT), 0, s, kin, vin, kout, vout, n,
                     shift, counts, ntiles);
  KV_HIP(hipGetLastError());
  return KV_OK;
}

}  // namespace

kv_status canon_build(Trace& t, const kv_trace_desc& d, hipStream_t s) {
  const uint64_t n = d.n;
  kv_status st;
  Order& o = t.shared;
  if ((st = o.key.reserve(n * 4)) != KV_OK) return st;
  if ((st = o.nxt.reserve(n * 4)) != KV_OK) return st;
  if ((st = o.bid.reserve(n * 4)) != KV_OK) return st;
  if ((st = o.w.reserve(n)) != KV_OK) return st;
  if ((st = o.g.reserve(n)) != KV_OK) return st;

  const uint32_t ntiles = div_up(n, kRsTile);
  const uint64_t ncount = (uint64_t)ntiles * 256;
  const uint64_t scratch_elems = std::max(scan_scratch_elems(ncount), scan_scratch_elems(n));
  DevBuf ka, kb, va, vb, kn, fl, counts, scratch, dst;
  if ((st = ka.reserve(n * 8)) != KV_OK) return st;
  if ((st = kb.reserve(n * 8)) != KV_OK) return st;
  if ((st = va.reserve(n * 4)) != KV_OK) return st;
  if ((st = vb.reserve(n * 4)) != KV_OK) return st;
  if ((st = kn.reserve(n * 16)) != KV_OK) return st;
  // trace-order first-occurrence flags, their inclusive sums, the groups'
  // first positions (u <= n)
  if ((st = fl.reserve(n * 12)) != KV_OK) return st;
  if ((st = counts.reserve(std::max<uint64_t>(ncount, 1) * 4)) != KV_OK) return st;
  if ((st = scratch.reserve(std::max<uint64_t>(scratch_elems, 1) * 4)) != KV_OK) return st;
  if ((st = dst.reserve(sizeof(DevStats))) != KV_OK) return st;
  DevStats* dstats = dst.as<DevStats>();
  KV_HIP(hipMemsetAsync(dstats, 0, sizeof(DevStats), s));
  KV_HIP(hipMemsetAsync(&dstats->w_min, 0xFF, 4, s));
  // the request of every access and the request times, kept for the
  // inter-arrival times of the TTL curves
  if ((st = t.req.reserve(n * 4)) != KV_OK) return st;
  if ((st = t.req_time.reserve((uint64_t)d.n_req * 8)) != KV_OK) return st;
  KV_HIP(hipMemcpyAsync(t.req.p, d.req, n * 4, hipMemcpyDeviceToDevice, s));
  KV_HIP(hipMemcpyAsync(t.req_time.p, d.req_time, (uint64_t)d.n_req * 8,
                        hipMemcpyDeviceToDevice, s));

  {
  StageTimer tm(kStLoadValidate, s);
  hipLaunchKernelGGL(k_validate, dim3(grid_of(n, 4 * kReduceGrid)), dim3(256), 0, s, d.hash, d.req,
                     d.group, d.weight, n, d.n_req, d.n_groups, o.g.as<uint8_t>(),
                     o.w.as<uint8_t>(),
                     ka.as<uint64_t>(), va.as<uint32_t>(), dstats);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_check_times, dim3(std::min<uint32_t>(div_up(d.n_req, 256), 4096)),
                     dim3(256), 0, s, d.req_time, d.n_req, dstats);
  KV_HIP(hipGetLastError());
  }

  // (hash, position) sorted by hash, ties by position.  Long traces: 4
  // stable passes of 8 bits over the high 32 bits, then the runs of equal
  // high bits that mix hashes sorted again by (run, low 32 bits) - for
  // random hashes a few thousand short runs, in the worst case every element.
  // Shorter ones: all 8 passes (the second sort's launches and its host
  // round trip would cost more than the 4 passes they save).
  uint64_t *kin = ka.as<uint64_t>(), *kout = kb.as<uint64_t>();
  uint32_t *vin = va.as<uint32_t>(), *vout = vb.as<uint32_t>();
  const bool high_first = n >= kHighFirstN || high_first_forced();
  {
    StageTimer tm(kStLoadSort, s);
    for (int shift = high_first ? 32 : 0; shift < 64; shift += 8) {
      st = radix_pass(kin, vin, kout, vout, n, shift, counts.as<uint32_t>(),
                      scratch.as<uint32_t>(), s);
      if (st != KV_OK) return st;
      std::swap(kin, kout);
      std::swap(vin, vout);
    }
  }
  if (high_first) {
    StageTimer tm(kStLoadSort, s);
    // free now: kout (2n u32), vout (n u32), fl (3n u32), kn (4n u32)
    uint32_t* flag = vout;
    uint32_t* runincl = reinterpret_cast<uint32_t*>(kout);
    uint32_t* mixed = runincl + n;  // per run, run ids < n
    uint32_t* at = fl.as<uint32_t>();
    hipLaunchKernelGGL(k_hi_starts, dim3(grid_of(n)), dim3(256), 0, s, kin, n, flag);
    KV_HIP(hipGetLastError());
    if ((st = scan_u32(flag, runincl, n, true, scratch.as<uint32_t>(), s)) != KV_OK) return st;
    if ((st = fill_u32(mixed, 0u, n, s)) != KV_OK) return st;
    hipLaunchKernelGGL(k_hi_mixed, dim3(grid_of(n)), dim3(256), 0, s, kin, n, runincl, mixed);
    KV_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_hi_inmixed, dim3(grid_of(n)), dim3(256), 0, s, runincl, mixed, n, flag);
    KV_HIP(hipGetLastError());
    if ((st = scan_u32(flag, at, n, false, scratch.as<uint32_t>(), s)) != KV_OK) return st;
    uint32_t last[3] = {0, 0, 0};
    KV_HIP(hipMemcpyAsync(&last[0], at + (n - 1), 4, hipMemcpyDeviceToHost, s));
    KV_HIP(hipMemcpyAsync(&last[1], flag + (n - 1), 4, hipMemcpyDeviceToHost, s));
    KV_HIP(hipMemcpyAsync(&last[2], runincl + (n - 1), 4, hipMemcpyDeviceToHost, s));
    KV_HIP(hipStreamSynchronize(s));
    const uint64_t m = (uint64_t)last[0] + last[1];
    // the second sort's key: run id (below the run count) above the low 32 bits
    int key_bits = 32;
    while (key_bits < 64 && (uint64_t)(last[2] - 1) >> (key_bits - 32)) ++key_bits;
    if (m) {
      uint64_t* ck = reinterpret_cast<uint64_t*>(kn.p);  // m u64, then m more
      uint64_t* ck2 = ck + m;
      uint32_t* cv = at + n;                             // m u32, then m more
      uint32_t* cv2 = cv + m;
      uint32_t* ci = mixed;                              // free after k_hi_inmixed
      hipLaunchKernelGGL(k_hi_gather, dim3(grid_of(n)), dim3(256), 0, s, kin, vin, n, runincl,
                         flag, at, ck, cv, ci);
      KV_HIP(hipGetLastError());
      for (int shift = 0; shift < key_bits; shift += 8) {
        st = radix_pass(ck, cv, ck2, cv2, m, shift, counts.as<uint32_t>(),
                        scratch.as<uint32_t>(), s);
        if (st != KV_OK) return st;
        std::swap(ck, ck2);
        std::swap(cv, cv2);
      }
      hipLaunchKernelGGL(k_hi_scatter, dim3(grid_of(m)), dim3(256), 0, s, ck, cv, ci, m, kin,
                         vin);
      KV_HIP(hipGetLastError());
    }
  }
  // kin / vin now hold the sorted pairs; the other pair of buffers is free.
  uint32_t* newflag = reinterpret_cast<uint32_t*>(kout);          // n u32
  uint32_t* incl = reinterpret_cast<uint32_t*>(kout) + n;         // n u32
  uint32_t* firstflag = fl.as<uint32_t>();
  uint32_t* fincl = firstflag + n;
  uint32_t* firstpos = fincl + n;
  uint32_t* runstart = vout;  // n >= u entries available
  uint32_t u32 = 0;
  {
  StageTimer tm(kStLoadLinks, s);
  hipLaunchKernelGGL(k_run_flags, dim3(grid_of(n)), dim3(256), 0, s, kin, n, newflag);
  KV_HIP(hipGetLastError());
  if ((st = scan_u32(newflag, incl, n, true, scratch.as<uint32_t>(), s)) != KV_OK) return st;
  if ((st = fill_u32(firstflag, 0u, n, s)) != KV_OK) return st;
  hipLaunchKernelGGL(k_first_pos, dim3(grid_of(n)), dim3(256), 0, s, vin, incl, newflag, n,
                     firstpos, firstflag);
  KV_HIP(hipGetLastError());
  if ((st = scan_u32(firstflag, fincl, n, true, scratch.as<uint32_t>(), s)) != KV_OK) return st;
  }
  KV_HIP(hipMemcpyAsync(&u32, incl + (n - 1), 4, hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  const uint64_t u = u32;
  if ((st = t.blk_w.reserve(u)) != KV_OK) return st;
  if ((st = t.blk_g.reserve(u)) != KV_OK) return st;
  {
  StageTimer tm(kStLoadLinks, s);
  hipLaunchKernelGGL(k_links, dim3(grid_of(n, 4 * kReduceGrid)), dim3(256), 0, s, kin, vin, n,
                     incl, newflag, firstpos, fincl, reinterpret_cast<uint4*>(kn.p),
                     t.blk_w.as<uint8_t>(),
                     t.blk_g.as<uint8_t>(), runstart, o.w.as<uint8_t>(), o.g.as<uint8_t>(),
                     dstats);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_split_links, dim3(grid_of(n)), dim3(256), 0, s,
                     reinterpret_cast<const uint4*>(kn.p), n, o.key.as<uint32_t>(),
                     o.nxt.as<uint32_t>(), o.bid.as<uint32_t>());
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_mult, dim3(grid_of(n, kReduceGrid)), dim3(256), 0, s, incl, newflag, n,
                     runstart, dstats);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_check_blocks, dim3(grid_of(n)), dim3(256), 0, s, o.bid.as<uint32_t>(),
                     t.blk_w.as<uint8_t>(), t.blk_g.as<uint8_t>(), o.w.as<uint8_t>(),
                     o.g.as<uint8_t>(), n, dstats);
  KV_HIP(hipGetLastError());
  }

  DevStats hs;
  double t0 = 0, t1 = 0;
  KV_HIP(hipMemcpyAsync(&hs, dstats, sizeof(DevStats), hipMemcpyDeviceToHost, s));
  KV_HIP(hipMemcpyAsync(&t0, d.req_time, 8, hipMemcpyDeviceToHost, s));
  KV_HIP(hipMemcpyAsync(&t1, d.req_time + (d.n_req - 1), 8, hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  if (hs.err) {
    std::string why;
    if (hs.err & kErrGroup) why += " group id >= n_groups;";
    if (hs.err & kErrWeight) why += " zero weight;";
    if (hs.err & kErrReq) why += " request index out of range or decreasing;";
    if (hs.err & kErrInconsistent) why += " a block hash carries two weights or groups;";
    if (hs.err & kErrTime) why += " request times decreasing or NaN;";
    return fail(KV_ERR_INVALID, "kv_trace_load: invalid trace:" + why);
  }
  kv_trace_stats& ts = t.st;
  ts = kv_trace_stats{};
  ts.n = n;
  ts.n_distinct = u;
  ts.n_req = d.n_req;
  ts.n_groups = d.n_groups;
  ts.w_min = hs.w_min;
  ts.w_max = hs.w_max;
  ts.max_multiplicity = hs.mult;
  ts.span = t1 - t0;
  for (uint32_t g = 0; g < KV_MAX_GROUPS; ++g) {
    ts.n_g[g] = hs.n_g[g];
    ts.n_w_g[g] = hs.n_w_g[g];
    ts.u_g[g] = hs.u_g[g];
    ts.u_w_g[g] = hs.u_w_g[g];
    ts.n_w += hs.n_w_g[g];
    ts.distinct_w += hs.u_w_g[g];
  }
  o.seg[0] = 0;
  o.seg[1] = n;
  for (uint32_t g = 2; g <= KV_MAX_GROUPS; ++g) o.seg[g] = n;
  o.built = true;
  t.n = n;
  t.u = u;
  t.n_groups = d.n_groups;
  return KV_OK;
}

kv_status canon_partition(Trace& t, hipStream_t s) {
  if (t.part.built) return KV_OK;
  const uint64_t n = t.n;
  kv_status st;
  Order& p = t.part;
  Order& o = t.shared;
  if ((st = p.key.reserve(n * 4)) != KV_OK) return st;
  if ((st = p.nxt.reserve(n * 4)) != KV_OK) return st;
  if ((st = p.bid.reserve(n * 4)) != KV_OK) return st;
  if ((st = p.w.reserve(n)) != KV_OK) return st;
  if ((st = p.g.reserve(n)) != KV_OK) return st;
  const uint32_t ntiles = div_up(n, kRsTile);
  const uint64_t ncount = (uint64_t)ntiles * 256;
  DevBuf ka, kb, va, vb, counts, scratch;
  if ((st = ka.reserve(n * 8)) != KV_OK) return st;
  if ((st = kb.reserve(n * 8)) != KV_OK) return st;
  if ((st = va.reserve(n * 4)) != KV_OK) return st;
  if ((st = vb.reserve(n * 4)) != KV_OK) return st;
  if ((st = counts.reserve(ncount * 4)) != KV_OK) return st;
  if ((st = scratch.reserve(std::max<uint64_t>(scan_scratch_elems(ncount), 1) * 4)) != KV_OK)
    return st;
  StageTimer tm(kStPartition, s);
  hipLaunchKernelGGL(k_group_keys, dim3(grid_of(n)), dim3(256), 0, s, o.g.as<uint8_t>(), n,
                     ka.as<uint64_t>(), va.as<uint32_t>());
  KV_HIP(hipGetLastError());
  st = radix_pass(ka.as<uint64_t>(), va.as<uint32_t>(), kb.as<uint64_t>(), vb.as<uint32_t>(), n,
                  0, counts.as<uint32_t>(), scratch.as<uint32_t>(), s);
  if (st != KV_OK) return st;
  const uint32_t* perm = vb.as<uint32_t>();
  uint32_t* ppos = va.as<uint32_t>();
  hipLaunchKernelGGL(k_part_inverse, dim3(grid_of(n)), dim3(256), 0, s, perm, n, ppos);
  KV_HIP(hipGetLastError());
  hipLaunchKernelGGL(k_part_build, dim3(grid_of(n)), dim3(256), 0, s, perm, ppos, n,
                     o.key.as<uint32_t>(), o.nxt.as<uint32_t>(), o.bid.as<uint32_t>(),
                     o.w.as<uint8_t>(), o.g.as<uint8_t>(), p.key.as<uint32_t>(),
                     p.nxt.as<uint32_t>(), p.bid.as<uint32_t>(), p.w.as<uint8_t>(),
                     p.g.as<uint8_t>());
  KV_HIP(hipGetLastError());
  KV_HIP(hipStreamSynchronize(s));
  p.seg[0] = 0;
  for (uint32_t g = 0; g < KV_MAX_GROUPS; ++g)
    p.seg[g + 1] = p.seg[g] + (g < t.n_groups ? t.st.n_g[g] : 0);
  p.built = true;
  return KV_OK;
}

}  // namespace kv
