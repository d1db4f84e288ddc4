// kernels_score.hip -- the importance-weighted roofline score (§3.6,
// Eq. (4)-(6)) for up to kScoreRankMax scored units, in two launches:
//
//  1. k_score_rank (one wave per unit): Eq. (4) validation (S_j in
//     (0, 1], NaN = not correct), the duplicate-key check, and each unit's
//     position in the order (operator, S, index) -- NaN after every value of
//     its operator -- counted against every unit staged in LDS; the units are
//     scattered to that order.  No sort.
//  2. k_score_final (one workgroup): operator runs of the ordered units: the
//     median of the correct S_j (Eq. (5); mean of the two middle values for an
//     even count, 0 when none), U_i of the operator from the Eq. (3) table
//     (0 when the operator is not in the trace), w_i = RN(U_i) / RN(sum U over
//     the retained operators) and S_agg = sum w_i S_i (Eq. (6)) as a
//     compensated sum.
#include <math.h>

#include "atrex_device.hpp"
#include "atrex_kernels.h"
#include "score_rank.hpp"

namespace {

constexpr uint32_t NT = 1024;
constexpr uint32_t NW = NT / 64;
constexpr uint32_t MINE = kRankPerBlock;  // units ranked per workgroup: one wave each
constexpr uint64_t kScoreOpsLds = 8192;  // operator table ids staged in LDS up to this size

__global__ __launch_bounds__(NT) void k_score_rank(const uint32_t* __restrict__ score_key,
                                                   const double* __restrict__ S, uint32_t n,
                                                   uint32_t* __restrict__ sorted_op, double* __restrict__ sorted_S,
                                                   uint32_t* __restrict__ err) {
  extern __shared__ uint64_t smem64[];
  score_rank_block(blockIdx.x, score_key, S, n, sorted_op, sorted_S, err, smem64);
}

struct Comp {
  double s, c;
};

__device__ __forceinline__ Comp comp_add(Comp a, double x) {  // Neumaier step
  const double t = a.s + x;
  if (fabs(a.s) >= fabs(x)) a.c += (a.s - t) + x; else a.c += (x - t) + a.s;
  a.s = t;
  return a;
}

__device__ __forceinline__ Comp comp_merge(Comp a, Comp b) {  // TwoSum of the sums
  const double t = a.s + b.s;
  const double bp = t - a.s;
  const double e = (a.s - (t - bp)) + (b.s - bp);
  return Comp{t, a.c + b.c + e};
}

__device__ uint32_t block_exscan(uint32_t v, uint32_t* s_w, uint32_t& total) {
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

// Each thread owns at most SC_PER consecutive ranked units and keeps the
// operators that start among them (U_i, S_i) in registers: one block scan
// numbers the operators, one block sum gives sum U, and the compensated sums
// of w_i S_i are merged in operator order (thread order, then wave order).
constexpr uint32_t SC_PER = kScoreRankMax / NT;

__device__ __forceinline__ Comp comp_shfl_down(Comp a, int d) {
  return Comp{__shfl_down(a.s, d, 64), __shfl_down(a.c, d, 64)};
}

__global__ __launch_bounds__(NT) void k_score_final(const uint32_t* __restrict__ sorted_op,
                                                    const double* __restrict__ sorted_S, uint32_t n, UnitTable opt,
                                                    const unsigned long long* __restrict__ nops_ptr, uint64_t maxOps,
                                                    uint32_t* __restrict__ op_out,
                                                    double* __restrict__ w_out, double* __restrict__ s_out,
                                                    double* __restrict__ s_agg, uint64_t* __restrict__ totU,
                                                    unsigned long long* __restrict__ nret) {
  extern __shared__ uint64_t smem64[];
  double* s_S = (double*)smem64;             // [n]
  uint32_t* s_op = (uint32_t*)(s_S + n);     // [n]
  uint32_t* s_opid = s_op + n;               // [nops_trace] when it fits (kScoreOpsLds)
  const uint64_t nops_trace = min((uint64_t)*nops_ptr, maxOps);
  const bool opid_lds = nops_trace <= kScoreOpsLds;
  __shared__ uint32_t s_w[NW];
  __shared__ uint32_t s_hbits[kScoreRankMax / 32];  // bit i: unit i starts an operator run
  __shared__ uint64_t s_u[2 * NW];
  __shared__ double s_cs[NW], s_cc[NW];
  const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  lds_stage<NT, 8>(s_S, sorted_S, n, [](double v) { return v; });
  lds_stage<NT, 8>(s_op, sorted_op, n, [](uint32_t v) { return v; });
  for (uint32_t j = tid; j < kScoreRankMax / 32; j += NT) s_hbits[j] = 0;
  if (opid_lds) lds_stage<NT, 8>(s_opid, opt.id, (uint32_t)nops_trace, [](uint32_t v) { return v; });
  __syncthreads();
  const uint32_t per = (n + NT - 1) / NT;  // <= SC_PER
  const uint32_t b = min(n, tid * per), e = min(n, b + per);
  uint32_t hmask = 0;  // bit j: unit b + j starts an operator run
#pragma unroll
  for (uint32_t j = 0; j < SC_PER; ++j) {
    const uint32_t i = b + j;
    if (i < e && (i == 0 || s_op[i - 1] != s_op[i])) hmask |= 1u << j;
  }
  if (hmask) {  // this thread's run heads into the bitmap (its units may span two words)
    atomicOr(&s_hbits[b >> 5], hmask << (b & 31));
    if ((b & 31) + per > 32) atomicOr(&s_hbits[(b >> 5) + 1], hmask >> (32 - (b & 31)));
  }
  uint32_t nops;
  const uint32_t ob = block_exscan(__popc(hmask), s_w, nops);  // its barriers also publish the bitmap
  // operator runs starting here: median of the correct S_j (Eq. (5)) and U_i
  u128 U[SC_PER];
  double Si[SC_PER];
  u128 myU = 0;
#pragma unroll
  for (uint32_t j = 0; j < SC_PER; ++j) {
    U[j] = 0;
    Si[j] = 0.0;
    if (!((hmask >> j) & 1u)) continue;
    const uint32_t i = b + j, op = s_op[i];
    // run end: the next run head (the bitmap's next set bit, looked for in
    // four words), else a binary search for the first larger operator
    uint32_t re = n, lo, hi;
    {
      uint32_t wi = (i + 1) >> 5;
      uint32_t bits = i + 1 < n ? s_hbits[wi] & (~0u << ((i + 1) & 31)) : 0u;
      for (int t = 0; t < 3 && !bits && (wi + 1) * 32 < n; ++t) bits = s_hbits[++wi];
      if (bits) {
        re = min(n, wi * 32 + (uint32_t)__builtin_ctz(bits));
      } else if ((wi + 1) * 32 < n) {
        lo = (wi + 1) * 32;
        hi = n;
        while (lo < hi) {
          const uint32_t mid = (lo + hi) / 2;
          if (s_op[mid] <= op) lo = mid + 1; else hi = mid;
        }
        re = lo;
      }
    }
    lo = i;
    hi = re;  // first NaN of the run (NaN sorts last)
    while (lo < hi) {
      const uint32_t mid = (lo + hi) / 2;
      if (!isnan(s_S[mid])) lo = mid + 1; else hi = mid;
    }
    const uint32_t c = lo - i;
    if (c) {
      const uint32_t h = c / 2;
      Si[j] = (c & 1) ? s_S[i + h] : (s_S[i + h - 1] + s_S[i + h]) / 2.0;
    }
    uint64_t x = 0, y = nops_trace;  // the operator's row of the Eq. (3) table
    while (x < y) {
      const uint64_t mid = (x + y) / 2;
      if ((opid_lds ? s_opid[mid] : opt.id[mid]) < op) x = mid + 1; else y = mid;
    }
    if (x < nops_trace && (opid_lds ? s_opid[x] : opt.id[x]) == op) U[j] = make_u128(opt.U[2 * x], opt.U[2 * x + 1]);
    myU += U[j];
  }
  // sum U over the retained operators
  const u128 tu = wave_sum_u128(myU);
  if (lane == 0) {
    s_u[2 * wave] = (uint64_t)tu;
    s_u[2 * wave + 1] = (uint64_t)(tu >> 64);
  }
  __syncthreads();
  u128 T = 0;
  for (uint32_t v = 0; v < NW; ++v) T += make_u128(s_u[2 * v], s_u[2 * v + 1]);
  const double dT = u128_to_f64(T);
  // w_i = RN(U_i) / RN(sum U); Eq. (6) as compensated sums in operator order
  Comp acc{0.0, 0.0};
  uint32_t k = ob;
#pragma unroll
  for (uint32_t j = 0; j < SC_PER; ++j) {
    if (!((hmask >> j) & 1u)) continue;
    const double wk = T == 0 ? 0.0 : u128_to_f64(U[j]) / dT;
    op_out[k] = s_op[b + j];
    s_out[k] = Si[j];
    w_out[k] = wk;
    acc = comp_add(acc, __dmul_rn(wk, Si[j]));
    ++k;
  }
  for (int d = 1; d < 64; d <<= 1) {  // lanes in order: lane l takes l + d when l is a multiple of 2d
    const Comp o = comp_shfl_down(acc, d);
    if ((lane & (2 * d - 1)) == 0) acc = comp_merge(acc, o);
  }
  if (lane == 0) {
    s_cs[wave] = acc.s;
    s_cc[wave] = acc.c;
  }
  __syncthreads();
  if (tid == 0) {
    Comp t{s_cs[0], s_cc[0]};
    for (uint32_t v = 1; v < NW; ++v) t = comp_merge(t, Comp{s_cs[v], s_cc[v]});
    *s_agg = t.s + t.c;
    totU[0] = (uint64_t)T;
    totU[1] = (uint64_t)(T >> 64);
    *nret = nops;
  }
}

}  // namespace

void launch_score_small(hipStream_t s, const uint32_t* score_key, const double* S, uint64_t n, uint32_t* sorted_op,
                        double* sorted_S, const UnitTable& opt, const unsigned long long* nops_trace, uint64_t maxOps,
                        uint32_t* op_out, double* w_out, double* s_out, double* s_agg, uint64_t* totU,
                        unsigned long long* nret, uint32_t* err) {
  const uint32_t nn = (uint32_t)n;
  hipLaunchKernelGGL(k_score_rank, dim3((nn + MINE - 1) / MINE), dim3(NT), (size_t)nn * 12, s, score_key, S, nn,
                     sorted_op, sorted_S, err);
  launch_score_final(s, n, sorted_op, sorted_S, opt, nops_trace, maxOps, op_out, w_out, s_out, s_agg, totU, nret);
}

void launch_score_final(hipStream_t s, uint64_t n, const uint32_t* sorted_op, const double* sorted_S,
                        const UnitTable& opt, const unsigned long long* nops_trace, uint64_t maxOps, uint32_t* op_out,
                        double* w_out, double* s_out, double* s_agg, uint64_t* totU, unsigned long long* nret) {
  const uint32_t nn = (uint32_t)n;
  hipLaunchKernelGGL(k_score_final, dim3(1), dim3(NT), (size_t)nn * 12 + kScoreOpsLds * 4, s, sorted_op, sorted_S, nn,
                     opt, nops_trace, maxOps, op_out, w_out, s_out, s_agg, totU, nret);
}

hipError_t set_score_smem_limits() {
  hipError_t e = hipFuncSetAttribute((const void*)k_score_rank, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)(kScoreRankMax * 12));
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)k_score_final, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)(kScoreRankMax * 12 + kScoreOpsLds * 4));
}
