// kernels_units.hip -- per-phase weights and Eq. (3) per operator and per key
// (§3.4) over the ordered groups: one workgroup (k_units_small) for up to
// kUnitsSmallMax groups, else three launches for any number of groups:
//
//  1. k_units_tiles (one 1024-group tile per workgroup): copies the groups to
//     the caller's arrays with RN(W) / RN(S[ph]); for each key (its groups are
//     adjacent, at most P of them) U_k = (L_P / |Phi_k|) * sum W; per tile the
//     number of keys and sum U_k; and the tile's operator runs (groups of one
//     operator inside the tile) with their W sums and phase masks.
//  2. k_units_ops (one workgroup): key offsets of the tiles, the operator
//     index of every run (a tile's first run continues the previous tile's
//     operator when the operator spans the boundary), U_i = (L_P / |Phi_i|) *
//     sum W per operator, sum U and w_i = RN(U_i) / RN(sum U).
//  3. k_units_keys (tiles): key ids, U_k and omega_k = RN(U_k) / RN(sum U_k).
//
// Phi (phases in which the unit runs) is the set of phases with a group,
// i.e. with at least one invocation.
#include <algorithm>

#include "atrex_device.hpp"
#include "atrex_kernels.h"
#include "score_rank.hpp"

namespace {

constexpr uint32_t TILE = 1024;
constexpr uint32_t NW = TILE / 64;

__device__ __forceinline__ u128 load_u128(const uint64_t* p, uint64_t i) { return make_u128(p[2 * i], p[2 * i + 1]); }
__device__ __forceinline__ void store_u128(uint64_t* p, uint64_t i, u128 v) {
  p[2 * i] = (uint64_t)v;
  p[2 * i + 1] = (uint64_t)(v >> 64);
}

// Exclusive scan of one u32 per thread over the block; total in `total`.
__device__ uint32_t tile_exscan(uint32_t v, uint32_t* s_w, uint32_t& total) {
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = v;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d, 64);
    if (lane >= (uint32_t)d) inc += y;
  }
  if (lane == 63) s_w[wave] = inc;
  __syncthreads();
  uint32_t off = 0;
  total = 0;
  for (uint32_t w = 0; w < NW; ++w) {
    if (w < wave) off += s_w[w];
    total += s_w[w];
  }
  __syncthreads();
  return off + inc - v;
}

// Block sum of a u128 (valid in every thread after the call).
__device__ u128 tile_sum_u128(u128 v, uint64_t* s_lo, uint64_t* s_hi) {
  const u128 t = wave_sum_u128(v);
  if ((threadIdx.x & 63) == 0) {
    s_lo[threadIdx.x >> 6] = (uint64_t)t;
    s_hi[threadIdx.x >> 6] = (uint64_t)(t >> 64);
  }
  __syncthreads();
  u128 s = 0;
  for (uint32_t w = 0; w < NW; ++w) s += make_u128(s_lo[w], s_hi[w]);
  __syncthreads();
  return s;
}

// L / k where k divides L (k = |Phi| in [1, P], L = lcm(1..P) <= 840): the
// quotient is an integer below 2^10 and the fp32 product L * rcp(k) is within
// 2^-21 relative of it, so rounding it to the nearest integer is exact.
__device__ __forceinline__ uint32_t lcm_over(uint32_t L, uint32_t k) {
  return (uint32_t)rintf((float)L * __builtin_amdgcn_rcpf((float)k));
}

__device__ __forceinline__ double ratio(u128 a, u128 b) { return b == 0 ? 0.0 : u128_to_f64(a) / u128_to_f64(b); }

__global__ __launch_bounds__(TILE) void k_units_tiles(SortedGroups g, uint64_t G, uint32_t P, uint64_t L,
                                                      const uint64_t* __restrict__ S, GroupsOut out, UnitScratch us) {
  __shared__ uint32_t s_w[NW];
  __shared__ uint64_t s_lo[NW], s_hi[NW];
  __shared__ unsigned long long s_rlo[TILE], s_rhi[TILE];
  __shared__ uint32_t s_rmask[TILE];
  const uint32_t t = blockIdx.x, l = threadIdx.x;
  const uint64_t i = (uint64_t)t * TILE + l;
  const bool valid = i < G;
  s_rlo[l] = 0;
  s_rhi[l] = 0;
  s_rmask[l] = 0;
  uint32_t key = 0, ph = 0;
  u128 W = 0;
  bool keyHead = false, opHead = false;
  if (valid) {
    key = g.key[i];
    ph = g.phase[i];
    W = load_u128(g.wsum, i);
    out.key[i] = key;
    out.phase[i] = (uint8_t)ph;
    out.count[i] = g.count[i];
    store_u128(out.wsum, i, W);
    if (out.raw) store_u128(out.raw, i, load_u128(g.raw, i));
    out.weight[i] = ratio(W, load_u128(S, ph));
    const uint32_t prev = i > 0 ? g.key[i - 1] : 0;
    keyHead = i == 0 || prev != key;
    opHead = i == 0 || (prev >> 16) != (key >> 16);
  }
  // keys: the head group sums the key's groups (adjacent, at most P)
  u128 Uk = 0;
  if (keyHead) {
    u128 sum = 0;
    uint32_t mask = 0;
    for (uint64_t e = i; e < G && g.key[e] == key; ++e) {
      sum += load_u128(g.wsum, e);
      mask |= 1u << g.phase[e];
    }
    Uk = (u128)lcm_over((uint32_t)L, (uint32_t)__popc(mask)) * sum;
    store_u128(us.keyU, i, Uk);
  }
  uint32_t nkeys;
  (void)tile_exscan(keyHead ? 1u : 0u, s_w, nkeys);
  const u128 sumUk = tile_sum_u128(Uk, s_lo, s_hi);
  // operator runs inside the tile: a run starts at an operator head or at the
  // tile's first group; its index is the number of run starts before it
  const bool runStart = valid && (opHead || l == 0);
  uint32_t nruns;
  const uint32_t r = tile_exscan(runStart ? 1u : 0u, s_w, nruns) + (runStart ? 1u : 0u) - 1u;  // valid rows only
  // sum each run's W and phase mask: segmented wave sums, one LDS add per run per wave
  {
    const uint32_t lane = l & 63;
    const uint32_t rr = valid ? r : 0xFFFFFFFFu;
    u128 v = valid ? W : (u128)0;
    uint32_t m = valid ? (1u << ph) : 0u;
    for (int d = 1; d < 64; d <<= 1) {  // suffix sums within runs
      const u128 y = shfl_down_u128(v, d);
      const uint32_t ym = __shfl_down(m, d, 64);
      const uint32_t yr = __shfl_down(rr, d, 64);
      if (lane + d < 64 && yr == rr) {
        v += y;
        m |= ym;
      }
    }
    const uint32_t pr = __shfl_up(rr, 1, 64);
    const bool segHead = valid && (lane == 0 || pr != rr);
    if (segHead) {
      const unsigned long long lo = (unsigned long long)(uint64_t)v;
      const unsigned long long old = atomicAdd(&s_rlo[r], lo);
      atomicAdd(&s_rhi[r], (unsigned long long)(uint64_t)(v >> 64) + ((old + lo < old) ? 1ull : 0ull));
      atomicOr(&s_rmask[r], m);
    }
  }
  __syncthreads();
  const size_t rb = (size_t)t * TILE;
  if (runStart) us.runOp[rb + r] = key >> 16;
  if (l < nruns) {
    us.runW[2 * (rb + l)] = s_rlo[l];
    us.runW[2 * (rb + l) + 1] = s_rhi[l];
    us.runMask[rb + l] = s_rmask[l];
  }
  if (l == 0) {
    us.tileKeys[t] = nkeys;
    store_u128(us.tileKeyU, t, sumUk);
    us.tileRuns[t] = nruns;
    us.tileCont[t] = (valid && !opHead) ? 1u : 0u;
  }
}

// One workgroup: key offsets of the tiles, the operator table, counts and totals.
__global__ __launch_bounds__(TILE) void k_units_ops(uint32_t ntiles, uint32_t P, uint64_t L, UnitScratch us,
                                                    UnitTable ops, uint64_t maxOps, const uint64_t* __restrict__ S,
                                                    uint64_t* __restrict__ phase_total,
                                                    unsigned long long* __restrict__ counts,
                                                    uint32_t* __restrict__ err) {
  __shared__ uint32_t s_w[NW];
  __shared__ uint64_t s_lo[NW], s_hi[NW];
  __shared__ uint32_t s_carry[3];
  const uint32_t l = threadIdx.x;
  if (l < P) {
    phase_total[2 * l] = S[2 * l];
    phase_total[2 * l + 1] = S[2 * l + 1];
  }
  // exclusive scans over the tiles: keys, operator heads (runs not continuing), runs
  if (l < 3) s_carry[l] = 0;
  __syncthreads();
  u128 sumUk = 0;
  for (uint32_t t0 = 0; t0 < ntiles; t0 += TILE) {
    const uint32_t t = t0 + l;
    const bool v = t < ntiles;
    const uint32_t nk = v ? us.tileKeys[t] : 0, nr = v ? us.tileRuns[t] : 0;
    const uint32_t nh = v ? nr - us.tileCont[t] : 0;
    if (v) sumUk += load_u128(us.tileKeyU, t);
    uint32_t tk, th, tr;
    const uint32_t ek = tile_exscan(nk, s_w, tk), eh = tile_exscan(nh, s_w, th), er = tile_exscan(nr, s_w, tr);
    if (v) {
      us.keyOff[t] = s_carry[0] + ek;
      us.opBase[t] = s_carry[1] + eh;
      us.runOff[t] = s_carry[2] + er;
    }
    __syncthreads();
    if (l == 0) { s_carry[0] += tk; s_carry[1] += th; s_carry[2] += tr; }
    __syncthreads();
  }
  const uint32_t nkeys = s_carry[0], nops = s_carry[1], nruns = s_carry[2];
  const u128 totUk = tile_sum_u128(sumUk, s_lo, s_hi);
  if (nops > maxOps) {
    if (l == 0) atomicOr(err, ATREX_ERRBIT_CAPACITY);
    return;
  }
  // operator accumulators: U (as W sums first) and the phase masks
  for (uint32_t q = l; q < nops; q += TILE) {
    ops.U[2 * q] = 0;
    ops.U[2 * q + 1] = 0;
    us.opMask[q] = 0;
  }
  __threadfence();
  __syncthreads();
  for (uint32_t x = l; x < nruns; x += TILE) {
    uint32_t lo = 0, hi = ntiles;  // tile of run x: last t with runOff[t] <= x
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) / 2;
      if (us.runOff[mid] <= x) lo = mid; else hi = mid;
    }
    const uint32_t t = lo, rr = x - us.runOff[t];
    const uint32_t q = us.opBase[t] + rr - us.tileCont[t];  // a continuing first run adds to the previous operator
    const size_t ri = (size_t)t * TILE + rr;
    if (rr > 0 || !us.tileCont[t]) ops.id[q] = us.runOp[ri];
    const unsigned long long wlo = us.runW[2 * ri], whi = us.runW[2 * ri + 1];
    const unsigned long long old = atomicAdd((unsigned long long*)&ops.U[2 * q], wlo);
    atomicAdd((unsigned long long*)&ops.U[2 * q + 1], whi + ((old + wlo < old) ? 1ull : 0ull));
    atomicOr(&us.opMask[q], us.runMask[ri]);
  }
  __threadfence();
  __syncthreads();
  u128 sumU = 0;
  for (uint32_t q = l; q < nops; q += TILE) {
    const uint64_t wlo = __hip_atomic_load(&ops.U[2 * q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t whi = __hip_atomic_load(&ops.U[2 * q + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t mask = __hip_atomic_load(&us.opMask[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const u128 U = (u128)lcm_over((uint32_t)L, (uint32_t)__popc(mask)) * make_u128(wlo, whi);
    store_u128(ops.U, q, U);
    sumU += U;
  }
  const u128 totU = tile_sum_u128(sumU, s_lo, s_hi);
  for (uint32_t q = l; q < nops; q += TILE) ops.w[q] = ratio(load_u128(ops.U, q), totU);
  if (l == 0) {
    counts[0] = nops;
    counts[1] = nkeys;
    store_u128(us.totals, 0, totU);
    store_u128(us.totals, 1, totUk);
  }
}

__global__ __launch_bounds__(TILE) void k_units_keys(SortedGroups g, uint64_t G, UnitScratch us, UnitTable keys) {
  __shared__ uint32_t s_w[NW];
  const uint32_t t = blockIdx.x, l = threadIdx.x;
  const uint64_t i = (uint64_t)t * TILE + l;
  bool head = false;
  uint32_t key = 0;
  if (i < G) {
    key = g.key[i];
    head = i == 0 || g.key[i - 1] != key;
  }
  uint32_t n;
  const uint32_t k = us.keyOff[t] + tile_exscan(head ? 1u : 0u, s_w, n);
  if (head) {
    const u128 U = load_u128(us.keyU, i);
    keys.id[k] = key;
    store_u128(keys.U, k, U);
    keys.w[k] = ratio(U, load_u128(us.totals, 1));
  }
}

// ---------------------------------------------------------------------------
// The groups copied to the caller's arrays with RN(W) / RN(S[ph]), one thread
// per group (the per-phase totals by the first threads), for the one-workgroup
// unit kernel below.
__device__ __forceinline__ void group_weights_at(uint32_t i, const SortedGroups& g, uint32_t G, uint32_t P,
                                                 const uint64_t* __restrict__ S, const GroupsOut& out) {
  if (i < P) {
    out.phase_total[2 * i] = S[2 * i];
    out.phase_total[2 * i + 1] = S[2 * i + 1];
  }
  if (i >= G) return;
  const uint32_t ph = g.phase[i];
  const u128 W = load_u128(g.wsum, i);
  out.key[i] = g.key[i];
  out.phase[i] = (uint8_t)ph;
  out.count[i] = g.count[i];
  store_u128(out.wsum, i, W);
  if (out.raw) store_u128(out.raw, i, load_u128(g.raw, i));
  out.weight[i] = ratio(W, load_u128(S, ph));
}

__global__ __launch_bounds__(256) void k_group_weights(SortedGroups g, uint32_t G, uint32_t P,
                                                        const uint64_t* __restrict__ S, GroupsOut out) {
  group_weights_at(blockIdx.x * 256 + threadIdx.x, g, G, P, S, out);
}

// ---------------------------------------------------------------------------
// One workgroup for up to kUnitsSmallMax groups: thread t holds groups
// [8t, 8t + 8) in registers.  A key run has at most P <= 8 groups, so it
// spans at most two threads: the run's part in the previous thread (that
// thread's tail after its last key head) comes by one shuffle.  Operator runs
// are summed with one block-wide segmented scan (a run head restarts the sum).
// Each run's total is taken at its last group; the run indices come from one
// block-wide count of the key and operator heads.  Same outputs as the three
// launches above.
constexpr uint32_t SM_PER = 8;

struct Seg {
  uint32_t f;  // a run head inside
  u128 v;      // sum of W since the last head
  uint32_t m;  // phase mask since the last head
};

__device__ __forceinline__ Seg seg_cat(const Seg& a, const Seg& b) {  // a, then b
  return b.f ? b : Seg{a.f, a.v + b.v, a.m | b.m};
}

__device__ __forceinline__ Seg seg_shfl_up(const Seg& x, int d) {
  Seg y;
  y.f = __shfl_up(x.f, d, 64);
  y.v = shfl_up_u128(x.v, d);
  y.m = __shfl_up(x.m, d, 64);
  return y;
}

// MODE: 1 = the key level only (U_k, omega_k, the key count), 2 = the
// operator level only (U_i, w_i, the operator count), 3 = both.
template <int MODE>
__device__ __forceinline__ void units_small_body(const SortedGroups& g, uint32_t G, uint32_t L, const UnitTable& ops,
                                                 uint64_t maxOps, const UnitTable& keys,
                                                 unsigned long long* __restrict__ counts,
                                                 uint32_t* __restrict__ err) {
  constexpr bool KEYS = (MODE & 1) != 0, OPS = (MODE & 2) != 0;
  __shared__ Seg s_ow[NW];
  __shared__ uint32_t s_n[NW];
  __shared__ uint64_t s_kt[3 * NW];  // each wave's last key tail: sum (lo, hi), phase mask
  __shared__ uint64_t s_lo[NW], s_hi[NW];
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t i0 = tid * SM_PER;
  // this thread's groups, the key before them and the key after them
  uint32_t key[SM_PER], ph[SM_PER];
  u128 W[SM_PER];
#pragma unroll
  for (int j = 0; j < SM_PER; ++j) {
    const uint32_t i = i0 + j;
    key[j] = i < G ? g.key[i] : 0u;
    ph[j] = i < G ? g.phase[i] : 0u;
    W[j] = i < G ? load_u128(g.wsum, i) : (u128)0;
  }
  const uint32_t kprev = (i0 > 0 && i0 <= G) ? g.key[i0 - 1] : 0u;
  const uint32_t knext = i0 + SM_PER < G ? g.key[i0 + SM_PER] : 0u;
  // heads of key runs and operator runs (bit j: group j heads a run), and
  // ends (bit j: group j is the last of its run)
  uint32_t kh = 0, oh = 0, ke = 0, oe = 0;
#pragma unroll
  for (int j = 0; j < SM_PER; ++j) {
    const uint32_t i = i0 + j;
    if (i >= G) continue;
    const uint32_t prev = j == 0 ? kprev : key[j - 1];
    const uint32_t nx = j + 1 < SM_PER ? key[j + 1] : knext;
    const bool last = i + 1 == G;
    if (KEYS && (i == 0 || prev != key[j])) kh |= 1u << j;
    if (OPS && (i == 0 || (prev >> 16) != (key[j] >> 16))) oh |= 1u << j;
    if (KEYS && (last || nx != key[j])) ke |= 1u << j;
    if (OPS && (last || (nx >> 16) != (key[j] >> 16))) oe |= 1u << j;
  }
  // key tail: W and phases after this thread's last key head (all its groups
  // when it has none)
  u128 ktv = 0;
  uint32_t ktm = 0;
  // operator aggregate of this thread, for the block-wide scan
  Seg oa{0, 0, 0};
#pragma unroll
  for (int j = 0; j < SM_PER; ++j) {
    if (i0 + j >= G) continue;
    const bool kf = (kh >> j) & 1, of = (oh >> j) & 1;
    if (KEYS) {
      ktv = (kf ? (u128)0 : ktv) + W[j];
      ktm = (kf ? 0u : ktm) | (1u << ph[j]);
    }
    if (OPS) oa = Seg{oa.f | (of ? 1u : 0u), (of ? (u128)0 : oa.v) + W[j], (of ? 0u : oa.m) | (1u << ph[j])};
  }
  // counts of key heads (low 16 bits) and operator heads (high 16 bits)
  const uint32_t cnt = __popc(kh) | (__popc(oh) << 16);
  Seg oi = oa;
  uint32_t ci = cnt;
  for (int d = 1; d < 64; d <<= 1) {
    Seg oy{0, 0, 0};
    if (OPS) oy = seg_shfl_up(oi, d);
    const uint32_t cy = __shfl_up(ci, d, 64);
    if (lane >= (uint32_t)d) {
      if (OPS) oi = seg_cat(oy, oi);
      ci += cy;
    }
  }
  // the previous thread's key tail (the previous wave's last lane through LDS)
  u128 kin_v = 0;
  uint32_t kin_m = 0;
  if (KEYS) {
    kin_v = shfl_up_u128(ktv, 1);
    kin_m = __shfl_up(ktm, 1, 64);
  }
  if (lane == 63) {
    if (OPS) s_ow[wave] = oi;
    s_n[wave] = ci;
    if (KEYS) {
      s_kt[3 * wave] = (uint64_t)ktv;
      s_kt[3 * wave + 1] = (uint64_t)(ktv >> 64);
      s_kt[3 * wave + 2] = ktm;
    }
  }
  __syncthreads();
  if (KEYS && lane == 0 && wave > 0) {
    kin_v = make_u128(s_kt[3 * (wave - 1)], s_kt[3 * (wave - 1) + 1]);
    kin_m = (uint32_t)s_kt[3 * (wave - 1) + 2];
  }
  Seg oc{0, 0, 0};  // operator carry into this thread
  uint32_t cc = 0, ctot = 0;
  for (uint32_t w = 0; w < NW; ++w) {
    if (w < wave) {
      if (OPS) oc = seg_cat(oc, s_ow[w]);
      cc += s_n[w];
    }
    ctot += s_n[w];
  }
  {  // exclusive within the wave
    Seg oy{0, 0, 0};
    if (OPS) oy = seg_shfl_up(oi, 1);
    const uint32_t cy = __shfl_up(ci, 1, 64);
    if (lane > 0) {
      if (OPS) oc = seg_cat(oc, oy);
      cc += cy;
    }
  }
  const uint32_t nkeys = ctot & 0xFFFFu, nops = ctot >> 16;
  const bool ops_fit = nops <= maxOps;
  // runs ending in this thread: totals, U = (L / |Phi|) * sum W (Eq. (3));
  // RN(U_k) of the key runs is kept for the weights
  u128 sumUk = 0, sumU = 0;
  double dUk[SM_PER];
  {
    u128 kv = kin_v;  // a run continued from the previous thread starts with its tail
    uint32_t km = kin_m;
    Seg orr = oc;
    uint32_t kidx = cc & 0xFFFFu, oidx = cc >> 16;  // heads so far
#pragma unroll
    for (int j = 0; j < SM_PER; ++j) {
      dUk[j] = 0.0;
      if (i0 + j >= G) continue;
      const bool kf = (kh >> j) & 1, of = (oh >> j) & 1;
      if (KEYS) {
        kv = (kf ? (u128)0 : kv) + W[j];
        km = (kf ? 0u : km) | (1u << ph[j]);
        kidx += kf;
        if ((ke >> j) & 1) {
          const u128 U = (u128)lcm_over(L, (uint32_t)__popc(km)) * kv;
          keys.id[kidx - 1] = key[j];
          store_u128(keys.U, kidx - 1, U);
          sumUk += U;
          dUk[j] = u128_to_f64(U);
        }
      }
      if (OPS) {
        orr = Seg{1u, (of ? (u128)0 : orr.v) + W[j], (of ? 0u : orr.m) | (1u << ph[j])};
        oidx += of;
        if ((oe >> j) & 1) {
          const u128 U = (u128)lcm_over(L, (uint32_t)__popc(orr.m)) * orr.v;
          if (ops_fit) {
            ops.id[oidx - 1] = key[j] >> 16;
            store_u128(ops.U, oidx - 1, U);
          }
          sumU += U;
        }
      }
    }
  }
  u128 totU = 0, totUk = 0;
  if (OPS) totU = tile_sum_u128(sumU, s_lo, s_hi);
  if (KEYS) totUk = tile_sum_u128(sumUk, s_lo, s_hi);
  // w_i = RN(U_i) / RN(sum U), omega_k = RN(U_k) / RN(sum U_k): this thread's own runs
  {
    const double dTk = u128_to_f64(totUk);
    uint32_t kidx = cc & 0xFFFFu, oidx = cc >> 16;
#pragma unroll
    for (int j = 0; j < SM_PER; ++j) {
      if (i0 + j >= G) continue;
      kidx += (kh >> j) & 1;
      oidx += (oh >> j) & 1;
      if (KEYS && ((ke >> j) & 1)) keys.w[kidx - 1] = totUk == 0 ? 0.0 : dUk[j] / dTk;
      if (OPS && ops_fit && ((oe >> j) & 1)) ops.w[oidx - 1] = ratio(load_u128(ops.U, oidx - 1), totU);
    }
  }
  if (tid == 0) {
    if (OPS) {
      counts[0] = nops;
      if (!ops_fit) atomicOr(err, ATREX_ERRBIT_CAPACITY);
    }
    if (KEYS) counts[1] = nkeys;
  }
}

__global__ __launch_bounds__(TILE) void k_units_small(SortedGroups g, uint32_t G, uint32_t L, UnitTable ops,
                                                      uint64_t maxOps, UnitTable keys,
                                                      unsigned long long* __restrict__ counts,
                                                      uint32_t* __restrict__ err) {
  units_small_body<3>(g, G, L, ops, maxOps, keys, counts, err);
}

// One launch for three independent steps of the one-call path: workgroups 0
// and 1 run the one-workgroup unit kernel's key level and operator level (the
// longest parts), the next nrank the score ranking, the rest the group
// weights, so that all of them run side by side on different CUs.
// With guard.G set, the group count comes from the device and the unit and
// group-weight parts run only when the ordering finished in one launch with a
// clean error word and at most guard.gmax groups (the caller decides
// afterwards, from the same words, whether their results stand).
__global__ __launch_bounds__(TILE) void k_units_rank(SortedGroups g, uint32_t G, uint32_t P, uint32_t L,
                                                     const uint64_t* __restrict__ S, GroupsOut out, UnitTable ops,
                                                     uint64_t maxOps, UnitTable keys,
                                                     unsigned long long* __restrict__ counts,
                                                     uint32_t* __restrict__ err, ScoreRankArgs sr, uint32_t nrank,
                                                     UnitsGuard guard) {
  extern __shared__ uint64_t smem64[];
  bool units_ok = true;
  if (guard.G) {
    const unsigned long long gd = *guard.G;
    units_ok = *guard.done == 1u &&
               (*guard.err & (ATREX_ERRBIT_RANGE | ATREX_ERRBIT_CAPACITY | ATREX_ERRBIT_SPILL)) == 0 &&
               gd <= guard.gmax;
    G = units_ok ? (uint32_t)gd : 0u;
  }
  if (blockIdx.x == 0) {  // the key level
    if (units_ok) units_small_body<1>(g, G, L, ops, maxOps, keys, counts, err);
  } else if (blockIdx.x == 1) {  // the operator level
    if (units_ok) units_small_body<2>(g, G, L, ops, maxOps, keys, counts, err);
  } else if (blockIdx.x <= nrank + 1) {
    score_rank_block(blockIdx.x - 2, sr.score_key, sr.S, sr.n, sr.sorted_op, sr.sorted_S, sr.err, smem64);
  } else if (units_ok) {
    group_weights_at((blockIdx.x - 2 - nrank) * TILE + threadIdx.x, g, G, P, S, out);
  }
}

}  // namespace

void launch_units_rank(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t L, const uint64_t* S,
                       const GroupsOut& out, const UnitTable& ops, uint64_t maxOps, const UnitTable& keys,
                       unsigned long long* counts, uint32_t* err, const ScoreRankArgs& sr, const UnitsGuard& guard) {
  const uint32_t nrank = (sr.n + kRankPerBlock - 1) / kRankPerBlock;
  const uint64_t gcap = guard.G ? guard.gmax : G;  // groups the weight part covers
  const uint32_t ngw = (uint32_t)std::max<uint64_t>(1, (gcap + TILE - 1) / TILE);
  hipLaunchKernelGGL(k_units_rank, dim3(2 + nrank + ngw), dim3(TILE), (size_t)sr.n * 12, s, g, (uint32_t)G, P,
                     (uint32_t)L, S, out, ops, maxOps, keys, counts, err, sr, nrank, guard);
}

void launch_units(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t L, const uint64_t* S,
                  const GroupsOut& out, const UnitScratch& us, const UnitTable& ops, uint64_t maxOps,
                  const UnitTable& keys, unsigned long long* counts, uint32_t* err) {
  if (G <= kUnitsSmallMax) {
    // independent launches; the one-workgroup kernel first, so that the host
    // enqueues the short one while it runs
    hipLaunchKernelGGL(k_units_small, dim3(1), dim3(TILE), 0, s, g, (uint32_t)G, (uint32_t)L, ops, maxOps, keys,
                       counts, err);
    hipLaunchKernelGGL(k_group_weights, dim3((uint32_t)std::max<uint64_t>(1, (G + 255) / 256)), dim3(256), 0, s, g,
                       (uint32_t)G, P, S, out);
    return;
  }
  const uint32_t nt = (uint32_t)((G + TILE - 1) / TILE);
  launch_fill_u64(s, (uint64_t*)counts, 2, 0);
  if (nt) hipLaunchKernelGGL(k_units_tiles, dim3(nt), dim3(TILE), 0, s, g, G, P, L, S, out, us);
  hipLaunchKernelGGL(k_units_ops, dim3(1), dim3(TILE), 0, s, nt, P, L, us, ops, maxOps, S, out.phase_total, counts,
                     err);
  if (nt) hipLaunchKernelGGL(k_units_keys, dim3(nt), dim3(TILE), 0, s, g, G, us, keys);
}

uint64_t units_tiles(uint64_t G) { return (G + TILE - 1) / TILE; }

hipError_t set_units_smem_limits() {
  return hipFuncSetAttribute((const void*)k_units_rank, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)(kScoreRankMax * 12));
}
