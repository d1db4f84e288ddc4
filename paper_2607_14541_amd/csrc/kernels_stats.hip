// kernels_stats.hip -- gfx950 kernels of the observed runtime per unit, the
// deployment baseline recorded for every retained (operator, shape) unit
// (§3.1, "Baselines and weights"): count, total, mean, min, max and
// nearest-rank quantiles of the invocation durations of each unit (a key, or
// a (key, phase) pair).
//
// The units and their counts come from the plain device-time group-by (its
// groups are ordered by (key, phase)).  The durations are then placed
// unit by unit (a counting sort: each tile of events reserves one block per
// unit it holds), and the order statistics are read per unit:
//   - up to 64 invocations: one wave sorts them in registers (bitonic);
//   - up to kStatsSmall: one workgroup sorts them in LDS (bitonic);
//   - more: a most-significant-digit radix select over the unit's block, 8
//     bits per round, every requested rank at once, several workgroups per
//     unit adding their digit histograms with global atomics.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t kEmptyU = 0xFFFFFFFFu;
constexpr int64_t kPad = 0x7FFFFFFFFFFFFFFFll;  // sorts after every duration

__device__ __forceinline__ uint64_t unit_rk(uint32_t key, uint32_t ph, bool by_phase) {
  return ((uint64_t)key << 3) | (by_phase ? ph : 0u);
}

__device__ __forceinline__ uint32_t unit_hash(uint64_t rk, uint32_t mask) {
  return hash32((uint32_t)rk ^ (uint32_t)(rk >> 32) * 0x9E3779B1u) & mask;
}

// Unit of a (key, phase); kEmptyU when absent.
__device__ __forceinline__ uint32_t unit_lookup(const StatsTable& t, uint64_t rk) {
  uint32_t h = unit_hash(rk, t.mask);
  for (uint32_t probe = 0; probe <= t.mask; ++probe) {
    const uint64_t k = t.key[h];
    if (k == rk + 1) return t.val[h];
    if (k == 0) return kEmptyU;
    h = (h + 1) & t.mask;
  }
  return kEmptyU;
}

// ---------------------------------------------------------------------------
// Unit heads among the groups: every group (by phase) or each new key.
__global__ void k_stats_heads(const uint32_t* __restrict__ key, uint64_t G, bool by_phase,
                              uint32_t* __restrict__ head) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  head[g] = (by_phase || g == 0 || key[g - 1] != key[g]) ? 1u : 0u;
}

// One thread per unit head: the unit's identity, count, total and mean
// (outputs below the caller's capacity), its count for the segment scan, and
// its entry in the lookup table.  The last group writes the unit count.
__global__ void k_stats_units(SortedGroups g, uint64_t G, bool by_phase, const uint32_t* __restrict__ head,
                              const uint32_t* __restrict__ uidx, StatsOut out, uint64_t cap,
                              uint32_t* __restrict__ ucount, StatsTable t, unsigned long long* __restrict__ words) {
  const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= G) return;
  if (r == G - 1) words[0] = (uint64_t)uidx[r] + head[r];
  if (!head[r]) return;
  const uint32_t k = g.key[r], u = uidx[r];
  u128 tot = 0;
  uint64_t n = 0;
  uint64_t x = r;
  do {  // the unit's groups: this one, and with merged phases the key's others
    tot += make_u128(g.wsum[2 * x], g.wsum[2 * x + 1]);
    n += g.count[x];
    ++x;
  } while (!by_phase && x < G && g.key[x] == k);
  const uint32_t ph = by_phase ? g.phase[r] : 0u;
  ucount[u] = (uint32_t)n;
  if (u < cap) {
    out.key[u] = k;
    out.phase[u] = (uint8_t)ph;
    out.count[u] = n;
    out.total[2 * u] = (uint64_t)tot;
    out.total[2 * u + 1] = (uint64_t)(tot >> 64);
    out.mean[u] = u128_to_f64(tot) / (double)n;  // n < 2^31: exact in fp64
  }
  const uint64_t rk = unit_rk(k, ph, by_phase);
  uint32_t h = unit_hash(rk, t.mask);
  for (uint32_t probe = 0; probe <= t.mask; ++probe) {  // the table holds at least twice the units
    const unsigned long long prev = atomicCAS((unsigned long long*)&t.key[h], 0ull, (unsigned long long)(rk + 1));
    if (prev == 0) {
      t.val[h] = u;
      return;
    }
    h = (h + 1) & t.mask;
  }
}

// ---------------------------------------------------------------------------
// Durations into their units' blocks.  Each workgroup walks its event range
// in tiles of 4 x BLOCK events; a tile counts its events per unit in an LDS
// table, reserves one block per unit it holds (one global atomic each), and
// writes every duration at its place in that block.  The maximum duration
// (for the radix select's digit range) is taken on the way.  Events whose
// unit is missing, whose fields are out of range, or that overrun their
// unit's segment flag the error word and are not written.
constexpr uint32_t kScatterSlots = 8192;  // LDS table of a tile's units (a tile holds 4096 events)

template <int BLOCK, bool VEC>
__global__ __launch_bounds__(BLOCK) void k_stats_scatter(EventsDev ev, uint32_t P, bool by_phase, StatsTable t,
                                                         const uint32_t* __restrict__ seg_start,
                                                         uint32_t* __restrict__ cursor, int64_t* __restrict__ vals,
                                                         unsigned long long* __restrict__ words,
                                                         uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s_tab[];  // 3 x kScatterSlots: unit, count, block start
  uint32_t* s_unit = s_tab;
  uint32_t* s_cnt = s_tab + kScatterSlots;
  uint32_t* s_base = s_tab + 2 * kScatterSlots;
  constexpr uint32_t TILE = 4 * BLOCK;
  const uint64_t n = ev.n;
  const uint64_t per = ((n + gridDim.x - 1) / gridDim.x + 3) / 4 * 4;  // multiple of 4: aligned groups
  const uint64_t b = min(n, (uint64_t)blockIdx.x * per), e = min(n, b + per);
  unsigned long long vmax = 0;
  uint32_t bad = 0;
  for (uint32_t i = threadIdx.x; i < kScatterSlots; i += BLOCK) {
    s_unit[i] = kEmptyU;
    s_cnt[i] = 0;
  }
  __syncthreads();
  for (uint64_t t0 = b; t0 < e; t0 += TILE) {
    uint32_t u[4], slot[4], rank[4];
    int64_t d[4];
    const uint64_t i0 = t0 + 4 * (uint64_t)threadIdx.x;
    uint32_t k4[4] = {0, 0, 0, 0}, p4[4] = {0, 0, 0, 0};
    if (VEC && i0 + 3 < e) {
      const v4u kk = *(const v4u*)(ev.key + i0);
      const uint32_t pp = *(const uint32_t*)(ev.phase + i0);
      const v2l d0 = *(const v2l*)(ev.dur + i0), d1 = *(const v2l*)(ev.dur + i0 + 2);
      k4[0] = kk.x; k4[1] = kk.y; k4[2] = kk.z; k4[3] = kk.w;
      p4[0] = pp & 0xFFu; p4[1] = (pp >> 8) & 0xFFu; p4[2] = (pp >> 16) & 0xFFu; p4[3] = pp >> 24;
      d[0] = d0.x; d[1] = d0.y; d[2] = d1.x; d[3] = d1.y;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool in = i0 + j < e;
        k4[j] = in ? ev.key[i0 + j] : 0u;
        p4[j] = in ? ev.phase[i0 + j] : 0u;
        d[j] = in ? ev.dur[i0 + j] : 0;
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u[j] = kEmptyU;
      slot[j] = kEmptyU;
      if (i0 + j >= e) continue;
      if (p4[j] >= P || d[j] < 0) {
        bad |= ATREX_ERRBIT_RANGE;
        continue;
      }
      u[j] = unit_lookup(t, unit_rk(k4[j], p4[j], by_phase));
      if (u[j] == kEmptyU) {
        bad |= ATREX_ERRBIT_CAPACITY;  // not an event of the aggregated trace
        continue;
      }
      vmax = max(vmax, (unsigned long long)d[j]);
      // the unit's slot in the tile table (linear probing from its hash)
      uint32_t h = hash32(u[j]) & (kScatterSlots - 1);
      for (uint32_t probe = 0; probe < kScatterSlots; ++probe) {
        const uint32_t prev = atomicCAS(&s_unit[h], kEmptyU, u[j]);
        if (prev == kEmptyU || prev == u[j]) break;
        h = (h + 1) & (kScatterSlots - 1);
      }
      slot[j] = h;
      rank[j] = atomicAdd(&s_cnt[h], 1u);
    }
    __syncthreads();
    // one block per unit of the tile
    for (uint32_t i = threadIdx.x; i < kScatterSlots; i += BLOCK)
      if (s_unit[i] != kEmptyU) s_base[i] = atomicAdd(&cursor[s_unit[i]], s_cnt[i]);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (slot[j] == kEmptyU) continue;
      const uint32_t pos = s_base[slot[j]] + rank[j];
      if (pos >= seg_start[u[j] + 1]) {  // more invocations than the group-by counted
        bad |= ATREX_ERRBIT_CAPACITY;
        continue;
      }
      vals[pos] = d[j];
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < kScatterSlots; i += BLOCK) {
      s_unit[i] = kEmptyU;
      s_cnt[i] = 0;
    }
    __syncthreads();
  }
  for (int dd = 32; dd >= 1; dd >>= 1) vmax = max(vmax, (unsigned long long)__shfl_xor(vmax, dd, 64));
  if ((threadIdx.x & 63) == 0) {
    if (vmax) atomicMax(&words[1], vmax);
  }
  for (int dd = 32; dd >= 1; dd >>= 1) bad |= __shfl_xor(bad, dd, 64);
  if (bad && (threadIdx.x & 63) == 0) atomicOr(err, bad);
}

// ---------------------------------------------------------------------------
// The same placement in two passes when the units' counters fit in LDS
// (a counting sort without global atomics): each workgroup counts its
// range's events per unit, an exclusive scan of the unit-major matrix of
// those counts gives every (unit, workgroup) its block, and a second pass
// places the durations with LDS cursors.  The ranges are those of
// k_stats_scatter.  On a wave, the lanes that share the first lane's unit
// take their ranks with one LDS atomic (a unit that dominates the events
// would otherwise serialise the wave's atomics on one address).
constexpr uint32_t kDenseUnits = 24576;     // 96 KB of LDS counters
constexpr uint32_t kDenseUnitsLtab = 4096;  // units when the lookup table sits in LDS too

// rank of this lane's unit u among the wave's lanes (uu: their ballot-shared
// unit) plus the LDS counter's old value, for lanes with `live`
__device__ __forceinline__ uint32_t wave_rank(uint32_t* ctr, uint32_t u, bool live) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t act = __ballot(live);
  if (act == 0) return 0;
  const uint32_t lead = (uint32_t)__ffsll((unsigned long long)act) - 1;
  const uint32_t uu = __builtin_amdgcn_readlane(u, lead);
  const uint64_t same = __ballot(live && u == uu);
  uint32_t base = 0;
  if (lane == lead) base = atomicAdd(&ctr[uu], (uint32_t)__popcll(same));
  base = __builtin_amdgcn_readlane(base, lead);
  if (live && u == uu) return base + (uint32_t)__popcll(same & (((uint64_t)1 << lane) - 1));
  return live ? atomicAdd(&ctr[u], 1u) : 0u;
}

// LTAB: the lookup table is copied into LDS (when it has at most
// kDenseTabSlots slots), beside the counters.  Pass 1 reads only the keys and
// phases; pass 2 reads the durations too and takes their maximum.  Each lane
// keeps the next step's loads in flight while it ranks the current four.
constexpr uint32_t kDenseTabSlots = 8192;  // 96 KB of table + the counters of at most 4096 units

template <bool PLACE>
struct DenseEv {
  uint32_t k[4], p[4];
  int64_t d[4];
};

template <int BLOCK, bool VEC, bool PLACE>
__device__ __forceinline__ void dense_load(const EventsDev& ev, uint64_t i0, uint64_t e, DenseEv<PLACE>& x) {
  if (VEC && i0 + 3 < e) {
    const v4u kk = __builtin_nontemporal_load((const v4u*)(ev.key + i0));
    const uint32_t pp = __builtin_nontemporal_load((const uint32_t*)(ev.phase + i0));
    x.k[0] = kk.x; x.k[1] = kk.y; x.k[2] = kk.z; x.k[3] = kk.w;
    x.p[0] = pp & 0xFFu; x.p[1] = (pp >> 8) & 0xFFu; x.p[2] = (pp >> 16) & 0xFFu; x.p[3] = pp >> 24;
    if (PLACE) {
      const v2l d0 = __builtin_nontemporal_load((const v2l*)(ev.dur + i0));
      const v2l d1 = __builtin_nontemporal_load((const v2l*)(ev.dur + i0 + 2));
      x.d[0] = d0.x; x.d[1] = d0.y; x.d[2] = d1.x; x.d[3] = d1.y;
    } else {
      x.d[0] = x.d[1] = x.d[2] = x.d[3] = 0;
    }
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool in = i0 + j < e;
      x.k[j] = in ? ev.key[i0 + j] : 0u;
      x.p[j] = in ? ev.phase[i0 + j] : 0u;
      x.d[j] = (in && PLACE) ? ev.dur[i0 + j] : 0;
    }
  }
}

// the same count without ranks: no LDS atomic returns its old value
__device__ __forceinline__ void wave_count(uint32_t* ctr, uint32_t u, bool live) {
  const uint32_t lane = threadIdx.x & 63;
  const uint64_t act = __ballot(live);
  if (act == 0) return;
  const uint32_t lead = (uint32_t)__ffsll((unsigned long long)act) - 1;
  const uint32_t uu = __builtin_amdgcn_readlane(u, lead);
  const uint64_t same = __ballot(live && u == uu);
  if (lane == lead) __hip_atomic_fetch_add(&ctr[uu], (uint32_t)__popcll(same), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
  else if (live && u != uu) __hip_atomic_fetch_add(&ctr[u], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int BLOCK, bool VEC, bool PLACE, bool LTAB>
__global__ __launch_bounds__(BLOCK) void k_stats_dense(EventsDev ev, uint32_t P, bool by_phase, StatsTable t,
                                                       uint32_t U, uint32_t* __restrict__ mat,
                                                       const uint32_t* __restrict__ seg_start,
                                                       int64_t* __restrict__ vals,
                                                       unsigned long long* __restrict__ words,
                                                       uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s_ctr[];  // [U] counts (pass 1) or cursors (pass 2), then the table (LTAB)
  const uint32_t nw = gridDim.x, w = blockIdx.x;
  for (uint32_t u = threadIdx.x; u < U; u += BLOCK) s_ctr[u] = PLACE ? mat[(size_t)u * nw + w] : 0u;
  StatsTable lt = t;
  if (LTAB) {  // the lookup table in LDS: keys (8-byte aligned after the counters), then values
    const uint32_t off = (U + 1) & ~1u;
    lt.key = (uint64_t*)(s_ctr + off);
    lt.val = s_ctr + off + 2 * (t.mask + 1);
    for (uint32_t h = threadIdx.x; h <= t.mask; h += BLOCK) {
      lt.key[h] = t.key[h];
      lt.val[h] = t.val[h];
    }
  }
  __syncthreads();
  const uint64_t n = ev.n;
  const uint64_t per = ((n + gridDim.x - 1) / gridDim.x + 3) / 4 * 4;
  const uint64_t b = min(n, (uint64_t)w * per), e = min(n, b + per);
  unsigned long long vmax = 0;
  uint32_t bad = 0;
  const uint64_t nstep = (e - b + 4 * BLOCK - 1) / (4 * BLOCK);  // uniform trip count (wave ballots below)
  DenseEv<PLACE> nxt;
  if (nstep) dense_load<BLOCK, VEC, PLACE>(ev, b + 4 * (uint64_t)threadIdx.x, e, nxt);
  for (uint64_t st = 0; st < nstep; ++st) {
    const uint64_t i0 = b + st * 4 * BLOCK + 4 * (uint64_t)threadIdx.x;
    const DenseEv<PLACE> x = nxt;
    if (st + 1 < nstep) dense_load<BLOCK, VEC, PLACE>(ev, i0 + 4 * BLOCK, e, nxt);
    uint32_t u[4];
    bool live[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      live[j] = i0 + j < e;
      u[j] = kEmptyU;
      if (live[j]) {
        if (x.p[j] >= P || (PLACE && x.d[j] < 0)) {
          bad |= ATREX_ERRBIT_RANGE;
          live[j] = false;
        } else {
          u[j] = unit_lookup(lt, unit_rk(x.k[j], x.p[j], by_phase));
          if (u[j] == kEmptyU || u[j] >= U) {
            bad |= ATREX_ERRBIT_CAPACITY;  // not an event of the aggregated trace
            live[j] = false;
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (!PLACE) {
        wave_count(s_ctr, u[j], live[j]);
        continue;
      }
      const uint32_t pos = wave_rank(s_ctr, u[j], live[j]);
      if (live[j]) {
        vmax = max(vmax, (unsigned long long)x.d[j]);
        if (pos < seg_start[u[j] + 1]) vals[pos] = x.d[j];
        else bad |= ATREX_ERRBIT_CAPACITY;  // more invocations than the group-by counted
      }
    }
  }
  __syncthreads();
  if (!PLACE)
    for (uint32_t u = threadIdx.x; u < U; u += BLOCK) mat[(size_t)u * nw + w] = s_ctr[u];
  for (int dd = 32; dd >= 1; dd >>= 1) {
    vmax = max(vmax, (unsigned long long)__shfl_xor(vmax, dd, 64));
    bad |= __shfl_xor(bad, dd, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    if (PLACE && vmax) atomicMax(&words[1], vmax);
    if (bad) atomicOr(err, bad);
  }
}

// Units by size class: up to 64 invocations, up to kStatsSmall, more (lists
// in any order; their lengths in words[2..4]).
__global__ void k_stats_classify(const uint32_t* __restrict__ ucount, uint64_t U, uint32_t small_max,
                                 uint32_t* __restrict__ tiny, uint32_t* __restrict__ small,
                                 uint32_t* __restrict__ large, unsigned long long* __restrict__ words) {
  const uint64_t u = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= U) return;
  const uint32_t c = ucount[u];
  if (c == 0) return;  // past the last unit (the counts are cleared to the group capacity)
  if (c <= 64) tiny[atomicAdd(&words[2], 1ull)] = (uint32_t)u;
  else if (c <= small_max) small[atomicAdd(&words[3], 1ull)] = (uint32_t)u;
  else large[atomicAdd(&words[4], 1ull)] = (uint32_t)u;
}

// Rank of quantile q (1e-5 steps) among c values, 1-based: ceil(q c / 1e5).
__device__ __forceinline__ uint32_t q_rank(uint32_t q, uint32_t c) {
  return (uint32_t)(((uint64_t)q * c + 99999) / 100000);
}

__device__ __forceinline__ int64_t shfl_i64(int64_t v, int src) {
  const int lo = __shfl((int)(uint32_t)v, src, 64), hi = __shfl((int)(uint32_t)((uint64_t)v >> 32), src, 64);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// One wave per unit of at most 64 invocations: a bitonic sort across the
// lanes (exchanges by shuffles), then the ranks.
__global__ __launch_bounds__(256) void k_stats_tiny(const uint32_t* __restrict__ list, uint64_t nlist,
                                                    const uint32_t* __restrict__ seg_start,
                                                    const int64_t* __restrict__ vals, StatsQ q, StatsOut out,
                                                    uint64_t cap) {
  const uint64_t w = (uint64_t)blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x & 63;
  if (w >= nlist) return;  // wave-uniform
  const uint32_t u = list[w], b = seg_start[u], c = seg_start[u + 1] - b;
  int64_t v = lane < (int)c ? vals[b + lane] : kPad;
  for (int k = 2; k <= 64; k <<= 1) {
    for (int j = k >> 1; j >= 1; j >>= 1) {
      const int64_t o = shfl_i64(v, lane ^ j);
      const bool up = (lane & k) == 0, lower = (lane & j) == 0;
      v = (lower == up) ? min(v, o) : max(v, o);
    }
  }
  if (u >= cap) return;
  const int64_t mn = shfl_i64(v, 0), mx = shfl_i64(v, (int)c - 1);
  if (lane == 0) {
    out.min[u] = mn;
    out.max[u] = mx;
  }
  for (uint32_t j = 0; j < q.n; ++j) {
    const int64_t x = shfl_i64(v, (int)q_rank(q.q[j], c) - 1);
    if (lane == 0) out.quant[(uint64_t)u * q.n + j] = x;
  }
}

// One workgroup per unit of at most kStatsSmall invocations: a bitonic sort
// in LDS over the next power of two (padded), then the ranks.
constexpr uint32_t kStatsSmall = 8192;
__global__ __launch_bounds__(256) void k_stats_small(const uint32_t* __restrict__ list,
                                                     const uint32_t* __restrict__ seg_start,
                                                     const int64_t* __restrict__ vals, StatsQ q, StatsOut out,
                                                     uint64_t cap) {
  extern __shared__ long long s_v[];  // [kStatsSmall]
  const uint32_t u = list[blockIdx.x], b = seg_start[u], c = seg_start[u + 1] - b;
  uint32_t m = 64;
  while (m < c) m <<= 1;
  for (uint32_t i = threadIdx.x; i < m; i += 256) s_v[i] = i < c ? vals[b + i] : kPad;
  __syncthreads();
  for (uint32_t k = 2; k <= m; k <<= 1) {
    for (uint32_t j = k >> 1; j >= 1; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < m / 2; i += 256) {
        // the pair (lo, lo + j) of the i-th comparator of this stage
        const uint32_t lo = 2 * i - (i & (j - 1));
        const uint32_t hi = lo + j;
        const bool up = (lo & k) == 0;
        const long long a = s_v[lo], bb = s_v[hi];
        if ((a > bb) == up) {
          s_v[lo] = bb;
          s_v[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  if (u >= cap) return;
  if (threadIdx.x == 0) {
    out.min[u] = s_v[0];
    out.max[u] = s_v[c - 1];
  }
  for (uint32_t j = threadIdx.x; j < q.n; j += 256) out.quant[(uint64_t)u * q.n + j] = s_v[q_rank(q.q[j], c) - 1];
}

// ---------------------------------------------------------------------------
// Radix select over the large units of one batch (units lu[0..nb)).
// Targets per unit: the q.n quantile ranks, then rank 1 (min), then rank c
// (max).  State per (unit, target): the value's bits fixed so far (prefix)
// and the target's rank among the values that share them (want, 1-based).
constexpr uint32_t kSelChunk = 65536;  // values per workgroup and round

__global__ void k_select_init(const uint32_t* __restrict__ lu, uint32_t nb, const uint32_t* __restrict__ seg_start,
                              StatsQ q, uint64_t* __restrict__ prefix, uint32_t* __restrict__ want,
                              uint32_t* __restrict__ cstart) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nb) return;
  const uint32_t u = lu[i], c = seg_start[u + 1] - seg_start[u];
  const uint32_t T = q.n + 2;
  for (uint32_t j = 0; j < T; ++j) {
    prefix[(size_t)i * T + j] = 0;
    want[(size_t)i * T + j] = j < q.n ? q_rank(q.q[j], c) : (j == q.n ? 1u : c);
  }
  cstart[i] = (c + kSelChunk - 1) / kSelChunk;  // chunk count, scanned by the host into chunk starts
}

// One workgroup per chunk: histogram of digit `shift` of the values whose
// higher bits (above shift + 8) equal each target's prefix.  Targets with
// equal prefixes share one histogram (in the first round all of them do).
// Per wave and prefix, the lanes whose digit equals the first such lane's add
// their count with one LDS atomic: durations crowd into few digits of their
// top bits, which would otherwise serialise the wave on one LDS address.
__global__ __launch_bounds__(1024) void k_select_hist(const uint32_t* __restrict__ lu, uint32_t nb,
                                                      const uint32_t* __restrict__ cstart,
                                                      const uint32_t* __restrict__ seg_start,
                                                      const int64_t* __restrict__ vals, uint32_t T, int shift,
                                                      const uint64_t* __restrict__ prefix,
                                                      uint32_t* __restrict__ hist) {
  __shared__ uint32_t s_h[10 * 256];
  __shared__ uint64_t s_p[10];     // the distinct prefixes
  __shared__ uint32_t s_rep[10];   // target -> its prefix's histogram
  __shared__ uint32_t s_nd;
  // the chunk's unit: the last i with cstart[i] <= blockIdx.x
  uint32_t lo = 0, hi = nb;  // cstart[0] = 0 <= blockIdx.x < cstart[nb]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (cstart[mid] <= blockIdx.x) lo = mid; else hi = mid;
  }
  const uint32_t i = lo, u = lu[i];
  const uint32_t cb = seg_start[u] + (blockIdx.x - cstart[i]) * kSelChunk;
  const uint32_t ce = min(seg_start[u + 1], cb + kSelChunk);
  for (uint32_t x = threadIdx.x; x < T * 256; x += 1024) s_h[x] = 0;
  if (threadIdx.x == 0) {
    uint32_t nd = 0;
    for (uint32_t j = 0; j < T; ++j) {
      const uint64_t pj = prefix[(size_t)i * T + j];
      uint32_t r = nd;
      for (uint32_t k = 0; k < nd; ++k)
        if (s_p[k] == pj) r = k;
      if (r == nd) s_p[nd++] = pj;
      s_rep[j] = r;
    }
    s_nd = nd;
  }
  __syncthreads();
  const uint32_t nd = s_nd, lane = threadIdx.x & 63;
  const int top = shift + 8;  // bits at and above `top` must equal the prefix
  // four values per thread and step, loaded before the first is counted
  const uint32_t steps = (ce - cb + 4095) / 4096;  // uniform over the workgroup: wave ballots below
  for (uint32_t st = 0; st < steps; ++st) {
    uint64_t vv[4];
    bool inv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t x = cb + st * 4096 + (uint32_t)u * 1024 + threadIdx.x;
      inv[u] = x < ce;
      vv[u] = inv[u] ? (uint64_t)vals[x] : 0;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const bool in = inv[u];
      const uint64_t v = vv[u];
      const uint64_t above = top >= 64 ? 0 : v >> top;
      const uint32_t dg = (uint32_t)(v >> shift) & 255u;
      for (uint32_t k = 0; k < nd; ++k) {
        const bool m = in && above == s_p[k];
        const uint64_t act = __ballot(m);
        if (act == 0) continue;  // wave-uniform
        const uint32_t lead = (uint32_t)__ffsll((unsigned long long)act) - 1;
        const uint32_t d0 = __builtin_amdgcn_readlane(dg, lead);
        const uint64_t same = __ballot(m && dg == d0);
        if (lane == lead) atomicAdd(&s_h[k * 256 + d0], (uint32_t)__popcll(same));
        else if (m && dg != d0) atomicAdd(&s_h[k * 256 + dg], 1u);
      }
    }
  }
  __syncthreads();
  for (uint32_t x = threadIdx.x; x < T * 256; x += 1024) {
    const uint32_t c = s_h[s_rep[x / 256] * 256 + (x & 255u)];
    if (c) atomicAdd(&hist[(size_t)i * T * 256 + x], c);
  }
}

// One thread per (unit, target): the digit holding the target's rank.
__global__ void k_select_pick(uint32_t nb, uint32_t T, const uint32_t* __restrict__ hist,
                              uint64_t* __restrict__ prefix, uint32_t* __restrict__ want) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= nb * T) return;
  const uint32_t* h = hist + (size_t)t * 256;
  uint32_t w = want[t], d = 0;
  for (; d < 255; ++d) {
    if (w <= h[d]) break;
    w -= h[d];
  }
  prefix[t] = (prefix[t] << 8) | d;
  want[t] = w;
}

// The selected values of the batch's units into the outputs.
__global__ void k_select_out(const uint32_t* __restrict__ lu, uint32_t nb, StatsQ q,
                             const uint64_t* __restrict__ prefix, StatsOut out, uint64_t cap) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nb) return;
  const uint32_t u = lu[i], T = q.n + 2;
  if (u >= cap) return;
  for (uint32_t j = 0; j < q.n; ++j) out.quant[(uint64_t)u * q.n + j] = (int64_t)prefix[(size_t)i * T + j];
  out.min[u] = (int64_t)prefix[(size_t)i * T + q.n];
  out.max[u] = (int64_t)prefix[(size_t)i * T + q.n + 1];
}

}  // namespace

// ---------------------------------------------------------------------------
// Host launchers
uint32_t stats_small_max() { return kStatsSmall; }
uint32_t stats_sel_chunk() { return kSelChunk; }

void launch_stats_units(hipStream_t s, const SortedGroups& g, uint64_t G, bool by_phase, uint32_t* head,
                        uint32_t* uidx, void* scan_tmp, const StatsOut& out, uint64_t cap, uint32_t* ucount,
                        const StatsTable& t, unsigned long long* words) {
  if (!G) return;
  const uint32_t nb = (uint32_t)((G + 255) / 256);
  hipLaunchKernelGGL(k_stats_heads, dim3(nb), dim3(256), 0, s, g.key, G, by_phase, head);
  exclusive_scan_u32(s, head, uidx, G, scan_tmp);
  hipLaunchKernelGGL(k_stats_units, dim3(nb), dim3(256), 0, s, g, G, by_phase, head, uidx, out, cap, ucount, t,
                     words);
}

void launch_stats_scatter(hipStream_t s, const EventsDev& ev, uint32_t P, bool by_phase, bool vec, uint32_t nblocks,
                          const StatsTable& t, const uint32_t* seg_start, uint32_t* cursor, int64_t* vals,
                          unsigned long long* words, uint32_t* err) {
  const size_t smem = (size_t)3 * kScatterSlots * 4;
  if (vec)
    hipLaunchKernelGGL((k_stats_scatter<1024, true>), dim3(nblocks), dim3(1024), smem, s, ev, P, by_phase, t,
                       seg_start, cursor, vals, words, err);
  else
    hipLaunchKernelGGL((k_stats_scatter<1024, false>), dim3(nblocks), dim3(1024), smem, s, ev, P, by_phase, t,
                       seg_start, cursor, vals, words, err);
}

uint32_t stats_dense_units() { return kDenseUnits; }

void launch_stats_dense(hipStream_t s, const EventsDev& ev, uint32_t P, bool by_phase, bool vec, uint32_t nblocks,
                        const StatsTable& t, uint32_t U, uint32_t* mat, void* scan_tmp, const uint32_t* seg_start,
                        int64_t* vals, unsigned long long* words, uint32_t* err) {
  const bool ltab = t.mask + 1 <= kDenseTabSlots && U <= kDenseUnitsLtab;
  const size_t smem = ltab ? (size_t)((U + 1) & ~1u) * 4 + (size_t)(t.mask + 1) * 12 : (size_t)U * 4;
#define ATREX_DENSE(V, PL, LT)                                                                                        \
  hipLaunchKernelGGL((k_stats_dense<1024, V, PL, LT>), dim3(nblocks), dim3(1024), smem, s, ev, P, by_phase, t, U, mat, \
                     seg_start, vals, words, err)
#define ATREX_DENSE2(PL)                       \
  if (ltab) {                                  \
    if (vec) ATREX_DENSE(true, PL, true);      \
    else ATREX_DENSE(false, PL, true);         \
  } else {                                     \
    if (vec) ATREX_DENSE(true, PL, false);     \
    else ATREX_DENSE(false, PL, false);        \
  }
  ATREX_DENSE2(false);
  exclusive_scan_u32(s, mat, mat, (uint64_t)U * nblocks, scan_tmp);
  ATREX_DENSE2(true);
#undef ATREX_DENSE2
#undef ATREX_DENSE
}

void launch_stats_classify(hipStream_t s, const uint32_t* ucount, uint64_t U, uint32_t* tiny, uint32_t* small,
                           uint32_t* large, unsigned long long* words) {
  if (U)
    hipLaunchKernelGGL(k_stats_classify, dim3((uint32_t)((U + 255) / 256)), dim3(256), 0, s, ucount, U,
                       kStatsSmall, tiny, small, large, words);
}

void launch_stats_sorts(hipStream_t s, const uint32_t* tiny, uint64_t ntiny, const uint32_t* small, uint64_t nsmall,
                        const uint32_t* seg_start, const int64_t* vals, const StatsQ& q, const StatsOut& out,
                        uint64_t cap) {
  if (ntiny)
    hipLaunchKernelGGL(k_stats_tiny, dim3((uint32_t)((ntiny + 3) / 4)), dim3(256), 0, s, tiny, ntiny, seg_start, vals,
                       q, out, cap);
  if (nsmall)
    hipLaunchKernelGGL(k_stats_small, dim3((uint32_t)nsmall), dim3(256), (size_t)kStatsSmall * 8, s, small, seg_start,
                       vals, q, out, cap);
}

void launch_select_init(hipStream_t s, const uint32_t* lu, uint32_t nb, const uint32_t* seg_start, const StatsQ& q,
                        uint64_t* prefix, uint32_t* want, uint32_t* ccount) {
  hipLaunchKernelGGL(k_select_init, dim3((nb + 256) / 256), dim3(256), 0, s, lu, nb, seg_start, q, prefix, want,
                     ccount);
}

void launch_select_round(hipStream_t s, const uint32_t* lu, uint32_t nb, const uint32_t* cstart, uint32_t nchunks,
                         const uint32_t* seg_start, const int64_t* vals, uint32_t T, int shift, uint64_t* prefix,
                         uint32_t* want, uint32_t* hist) {
  launch_fill_u64(s, (uint64_t*)hist, ((uint64_t)nb * T * 256 + 1) / 2, 0);
  hipLaunchKernelGGL(k_select_hist, dim3(nchunks), dim3(1024), 0, s, lu, nb, cstart, seg_start, vals, T, shift, prefix,
                     hist);
  hipLaunchKernelGGL(k_select_pick, dim3((nb * T + 255) / 256), dim3(256), 0, s, nb, T, hist, prefix, want);
}

void launch_select_out(hipStream_t s, const uint32_t* lu, uint32_t nb, const StatsQ& q, const uint64_t* prefix,
                       const StatsOut& out, uint64_t cap) {
  hipLaunchKernelGGL(k_select_out, dim3((nb + 255) / 256), dim3(256), 0, s, lu, nb, q, prefix, out, cap);
}

hipError_t set_stats_smem_limits() {
  hipError_t e = hipFuncSetAttribute((const void*)k_stats_small, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     kStatsSmall * 8);
  const void* sc[] = {(const void*)k_stats_scatter<1024, true>, (const void*)k_stats_scatter<1024, false>};
  for (const void* f : sc) {
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 3 * kScatterSlots * 4);
  }
  const void* dn[] = {
      (const void*)k_stats_dense<1024, true, false, false>, (const void*)k_stats_dense<1024, false, false, false>,
      (const void*)k_stats_dense<1024, true, true, false>,  (const void*)k_stats_dense<1024, false, true, false>,
      (const void*)k_stats_dense<1024, true, false, true>,  (const void*)k_stats_dense<1024, false, false, true>,
      (const void*)k_stats_dense<1024, true, true, true>,   (const void*)k_stats_dense<1024, false, true, true>};
  for (const void* f : dn) {
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
  }
  return e;
}
