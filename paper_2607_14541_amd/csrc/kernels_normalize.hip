// kernels_normalize.hip -- per-phase totals of W (§3.4) and the score of
// Eq. (4)-(6) (§3.6) for many scored units: radix-sorted (key) and (operator,
// S) orders, run starts, medians, Eq. (6) as a compensated sum; gfx950.
#include <math.h>

#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr int NB = 256;

// ------------------------------------------------------- u128 block reduction
// Per-phase u128 sums of W over the sorted groups: partials[block][ph].
__global__ __launch_bounds__(NB) void k_phase_totals_part(SortedGroups g, uint64_t G, uint32_t P,
                                                          uint64_t* __restrict__ partials) {
  __shared__ uint64_t s_lo[NB / 64][8], s_hi[NB / 64][8];
  u128 acc[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) acc[p] = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * NB + threadIdx.x; i < G; i += (uint64_t)gridDim.x * NB) {
    const u128 w = make_u128(g.wsum[2 * i], g.wsum[2 * i + 1]);
    const uint32_t ph = g.phase[i];
#pragma unroll
    for (int p = 0; p < 8; ++p) acc[p] += (ph == (uint32_t)p) ? w : (u128)0;
  }
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const u128 t = wave_sum_u128(acc[p]);
    if (lane == 0) { s_lo[wave][p] = (uint64_t)t; s_hi[wave][p] = (uint64_t)(t >> 64); }
  }
  __syncthreads();
  if (threadIdx.x < P) {
    u128 t = 0;
    for (int w = 0; w < NB / 64; ++w) t += make_u128(s_lo[w][threadIdx.x], s_hi[w][threadIdx.x]);
    partials[((size_t)blockIdx.x * P + threadIdx.x) * 2] = (uint64_t)t;
    partials[((size_t)blockIdx.x * P + threadIdx.x) * 2 + 1] = (uint64_t)(t >> 64);
  }
}

// out[c] = sum over r < rows of x[r][c] for c < cols (u128 entries).
__global__ __launch_bounds__(NB) void k_colsum_u128(const uint64_t* __restrict__ x, uint32_t rows, uint32_t cols,
                                                    uint64_t* __restrict__ out) {
  __shared__ uint64_t s_lo[NB / 64], s_hi[NB / 64];
  for (uint32_t c = 0; c < cols; ++c) {
    u128 acc = 0;
    for (uint32_t r = threadIdx.x; r < rows; r += NB)
      acc += make_u128(x[((size_t)r * cols + c) * 2], x[((size_t)r * cols + c) * 2 + 1]);
    const u128 t = wave_sum_u128(acc);
    if ((threadIdx.x & 63) == 0) { s_lo[threadIdx.x >> 6] = (uint64_t)t; s_hi[threadIdx.x >> 6] = (uint64_t)(t >> 64); }
    __syncthreads();
    if (threadIdx.x == 0) {
      u128 s = 0;
      for (int w = 0; w < NB / 64; ++w) s += make_u128(s_lo[w], s_hi[w]);
      out[2 * c] = (uint64_t)s;
      out[2 * c + 1] = (uint64_t)(s >> 64);
    }
    __syncthreads();
  }
}

// Sum of an array of u128: partials[block].
__global__ __launch_bounds__(NB) void k_sum_u128_part(const uint64_t* __restrict__ x, uint64_t n,
                                                      uint64_t* __restrict__ partials) {
  __shared__ uint64_t s_lo[NB / 64], s_hi[NB / 64];
  u128 acc = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * NB + threadIdx.x; i < n; i += (uint64_t)gridDim.x * NB)
    acc += make_u128(x[2 * i], x[2 * i + 1]);
  const u128 t = wave_sum_u128(acc);
  if ((threadIdx.x & 63) == 0) { s_lo[threadIdx.x >> 6] = (uint64_t)t; s_hi[threadIdx.x >> 6] = (uint64_t)(t >> 64); }
  __syncthreads();
  if (threadIdx.x == 0) {
    u128 s = 0;
    for (int w = 0; w < NB / 64; ++w) s += make_u128(s_lo[w], s_hi[w]);
    partials[2 * blockIdx.x] = (uint64_t)s;
    partials[2 * blockIdx.x + 1] = (uint64_t)(s >> 64);
  }
}

// ------------------------------------------------------- run starts

__global__ void k_unit_starts(const uint32_t* __restrict__ flags, const uint32_t* __restrict__ scan, uint64_t G,
                              uint32_t* __restrict__ starts) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < G && flags[i]) starts[scan[i]] = (uint32_t)i;
  if (i == G - 1) starts[scan[i] + flags[i]] = (uint32_t)G;  // sentinel
}



// ------------------------------------------------------- score, Eq. (4)-(6)
__global__ void k_score_validate(const double* __restrict__ S, uint64_t n, uint32_t* __restrict__ err) {
  const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool bad = false;
  if (j < n) {
    const double s = S[j];
    bad = !isnan(s) && !(s > 0.0 && s <= 1.0);  // S_j in (0, 1]; NaN = not correct
  }
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
}

// sort keys: (key), (S bit pattern; NaN after every valid value), index
__global__ void k_score_keys(const uint32_t* __restrict__ score_key, const double* __restrict__ S, uint64_t n,
                             uint64_t* __restrict__ k_key, uint64_t* __restrict__ k_sval, uint32_t* __restrict__ idx) {
  const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  k_key[j] = score_key[j];
  const double s = S[j];
  k_sval[j] = isnan(s) ? ~0ull : (uint64_t)__double_as_longlong(s);  // s > 0: bit order = value order
  idx[j] = (uint32_t)j;
}

__global__ void k_dup_check(const uint64_t* __restrict__ k, uint64_t n, uint32_t* __restrict__ err) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool dup = i > 0 && i < n && k[i] == k[i - 1];
  if (__any(dup) && (threadIdx.x & 63) == 0) atomicOr(err, ATREX_ERRBIT_DUP);
}

__global__ void k_score_opkeys(const uint32_t* __restrict__ score_key, const uint32_t* __restrict__ idx, uint64_t n,
                               uint64_t* __restrict__ k_op) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) k_op[i] = score_key[idx[i]] >> 16;
}

// One thread per retained operator: Eq. (5) median of the correct S_j (they
// come first in the segment, ascending; the first NaN is found by binary
// search), 0 if none; U_i looked up in the operator table of the trace
// (absent: 0).
__global__ void k_score_ops(const uint32_t* __restrict__ score_key, const double* __restrict__ S,
                            const uint32_t* __restrict__ order, const uint32_t* __restrict__ starts, uint64_t nops,
                            UnitTable opt, uint64_t nops_trace, uint32_t* __restrict__ r_op,
                            uint64_t* __restrict__ r_U, double* __restrict__ r_S) {
  const uint64_t u = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= nops) return;
  const uint32_t b = starts[u], e = starts[u + 1];
  const uint32_t op = score_key[order[b]] >> 16;
  uint32_t lo_n = b, hi_n = e;  // first NaN of the segment (NaN sorts after every value)
  while (lo_n < hi_n) {
    const uint32_t mid = (lo_n + hi_n) / 2;
    if (!isnan(S[order[mid]])) lo_n = mid + 1; else hi_n = mid;
  }
  const uint32_t c = lo_n - b;
  double Si = 0.0;
  if (c) {
    const uint32_t h = c / 2;
    Si = (c & 1) ? S[order[b + h]] : (S[order[b + h - 1]] + S[order[b + h]]) / 2.0;
  }
  // binary search op in the trace's operator table
  uint64_t lo = 0, hi = nops_trace;
  while (lo < hi) {
    const uint64_t mid = (lo + hi) / 2;
    if (opt.id[mid] < op) lo = mid + 1; else hi = mid;
  }
  uint64_t Ulo = 0, Uhi = 0;
  if (lo < nops_trace && opt.id[lo] == op) { Ulo = opt.U[2 * lo]; Uhi = opt.U[2 * lo + 1]; }
  r_op[u] = op;
  r_U[2 * u] = Ulo;
  r_U[2 * u + 1] = Uhi;
  r_S[u] = Si;
}

// Operator keys of the scored units in input order, and the identity order.
__global__ void k_score_opiota(const uint32_t* __restrict__ score_key, uint64_t n, uint64_t* __restrict__ k_op,
                               uint32_t* __restrict__ idx) {
  const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  k_op[j] = score_key[j] >> 16;
  idx[j] = (uint32_t)j;
}

// Longest operator segment (starts[0..nseg], nseg = scan[n-1] + flags[n-1]).
__global__ void k_seg_maxlen(const uint32_t* __restrict__ flags, const uint32_t* __restrict__ scan, uint64_t n,
                             const uint32_t* __restrict__ starts, uint32_t* __restrict__ out) {
  const uint32_t nseg = scan[n - 1] + flags[n - 1];
  uint32_t mx = 0;
  for (uint64_t u = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nseg; u += (uint64_t)gridDim.x * blockDim.x)
    mx = max(mx, starts[u + 1] - starts[u]);
  for (int d = 32; d >= 1; d >>= 1) mx = max(mx, (uint32_t)__shfl_xor(mx, d, 64));
  if ((threadIdx.x & 63) == 0 && mx) atomicMax(out, mx);
}

// One workgroup per operator segment of at most kScoreSegMax units (N2 = a
// power of two at least the longest segment): the segment's keys and S bit
// patterns (NaN last) are sorted in LDS; equal neighbouring keys are a
// duplicate; the Eq. (5) median of the correct S_j (mean of the two middle
// values for an even count, 0 when none) and U_i from the operator table of
// the trace (absent: 0).
__device__ __forceinline__ void lds_bitonic(uint64_t* v, uint32_t N2) {
  for (uint32_t k = 2; k <= N2; k <<= 1)
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < N2; i += blockDim.x) {
        const uint32_t l = i ^ j;
        if (l > i) {
          const uint64_t x = v[i], y = v[l];
          if ((x > y) == ((i & k) == 0)) {
            v[i] = y;
            v[l] = x;
          }
        }
      }
      __syncthreads();
    }
}

__global__ __launch_bounds__(256) void k_score_seg(const uint32_t* __restrict__ score_key, const double* __restrict__ S,
                                                   const uint32_t* __restrict__ order,
                                                   const uint32_t* __restrict__ starts, uint32_t N2, UnitTable opt,
                                                   uint64_t nops_trace, uint32_t* __restrict__ r_op,
                                                   uint64_t* __restrict__ r_U, double* __restrict__ r_S,
                                                   uint32_t* __restrict__ err) {
  extern __shared__ uint64_t sm64[];
  uint64_t* sk = sm64;       // [N2] keys, padding ~0
  uint64_t* sv = sm64 + N2;  // [N2] S bit patterns (S > 0: bit order = value order), NaN and padding ~0
  __shared__ uint32_t s_dup;
  const uint32_t u = blockIdx.x, tid = threadIdx.x;
  const uint32_t b = starts[u], m = starts[u + 1] - b;
  if (tid == 0) s_dup = 0;
  for (uint32_t i = tid; i < N2; i += blockDim.x) {
    uint64_t kk = ~0ull, vv = ~0ull;
    if (i < m) {
      const uint32_t j = order[b + i];
      kk = score_key[j];
      const double x = S[j];
      vv = isnan(x) ? ~0ull : (uint64_t)__double_as_longlong(x);
    }
    sk[i] = kk;
    sv[i] = vv;
  }
  __syncthreads();
  lds_bitonic(sk, N2);
  lds_bitonic(sv, N2);
  bool dup = false;
  for (uint32_t i = tid; i + 1 < m; i += blockDim.x) dup |= sk[i] == sk[i + 1];
  if (dup) s_dup = 1u;
  __syncthreads();
  if (tid != 0) return;
  if (s_dup) atomicOr(err, ATREX_ERRBIT_DUP);
  uint32_t lo = 0, hi = m;  // correct S_j: the entries before the first ~0
  while (lo < hi) {
    const uint32_t mid = (lo + hi) / 2;
    if (sv[mid] != ~0ull) lo = mid + 1; else hi = mid;
  }
  const uint32_t c = lo, h = c / 2;
  double Si = 0.0;
  if (c)
    Si = (c & 1) ? __longlong_as_double((long long)sv[h])
                 : (__longlong_as_double((long long)sv[h - 1]) + __longlong_as_double((long long)sv[h])) / 2.0;
  const uint32_t op = (uint32_t)(sk[0] >> 16);
  uint64_t x = 0, y = nops_trace;  // the operator's row of the Eq. (3) table
  while (x < y) {
    const uint64_t mid = (x + y) / 2;
    if (opt.id[mid] < op) x = mid + 1; else y = mid;
  }
  uint64_t Ulo = 0, Uhi = 0;
  if (x < nops_trace && opt.id[x] == op) { Ulo = opt.U[2 * x]; Uhi = opt.U[2 * x + 1]; }
  r_op[u] = op;
  r_U[2 * u] = Ulo;
  r_U[2 * u + 1] = Uhi;
  r_S[u] = Si;
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

// Eq. (6): w_i = RN(U_i) / RN(sum over retained U), S_agg = sum w_i S_i with
// compensated summation (each thread a contiguous run, then a TwoSum tree).
__global__ __launch_bounds__(1024) void k_score_final(const uint32_t* __restrict__ r_op, const uint64_t* __restrict__ r_U,
                                                      const double* __restrict__ r_S, uint64_t nops,
                                                      const uint64_t* __restrict__ totalU, uint32_t* __restrict__ op,
                                                      double* __restrict__ op_weight, double* __restrict__ op_score,
                                                      double* __restrict__ s_agg) {
  __shared__ double s_s[1024], s_c[1024];
  const u128 tot = make_u128(totalU[0], totalU[1]);
  const double dt = u128_to_f64(tot);
  const uint64_t per = (nops + 1023) / 1024;
  const uint64_t b = threadIdx.x * per, e = (b + per < nops) ? b + per : nops;
  Comp acc{0.0, 0.0};
  for (uint64_t u = b; u < e; ++u) {
    const double w = tot == 0 ? 0.0 : u128_to_f64(make_u128(r_U[2 * u], r_U[2 * u + 1])) / dt;
    const double x = __dmul_rn(w, r_S[u]);
    acc = comp_add(acc, x);
    if (op) op[u] = r_op[u];
    if (op_weight) op_weight[u] = w;
    if (op_score) op_score[u] = r_S[u];
  }
  s_s[threadIdx.x] = acc.s;
  s_c[threadIdx.x] = acc.c;
  __syncthreads();
  for (int d = 512; d >= 1; d >>= 1) {
    if (threadIdx.x < (uint32_t)d) {
      const Comp m = comp_merge(Comp{s_s[threadIdx.x], s_c[threadIdx.x]}, Comp{s_s[threadIdx.x + d], s_c[threadIdx.x + d]});
      s_s[threadIdx.x] = m.s;
      s_c[threadIdx.x] = m.c;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *s_agg = s_s[0] + s_c[0];
}

__global__ void k_heads_u64(const uint64_t* __restrict__ k, uint64_t n, uint32_t* __restrict__ flags) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) flags[i] = (i == 0 || k[i] != k[i - 1]) ? 1u : 0u;
}

uint32_t grid_for(uint64_t n, uint32_t b) { return (uint32_t)((n + b - 1) / b); }

}  // namespace

void launch_phase_totals(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t* partials, uint32_t nb,
                         uint64_t* S) {
  hipLaunchKernelGGL(k_phase_totals_part, dim3(nb), dim3(NB), 0, s, g, G, P, partials);
  hipLaunchKernelGGL(k_colsum_u128, dim3(1), dim3(NB), 0, s, partials, nb, P, S);
}



void launch_unit_starts(hipStream_t s, const uint32_t* flags, const uint32_t* scan, uint64_t G, uint32_t* starts) {
  if (G) hipLaunchKernelGGL(k_unit_starts, dim3(grid_for(G, 256)), dim3(256), 0, s, flags, scan, G, starts);
}


void launch_sum_u128(hipStream_t s, const uint64_t* x, uint64_t n, uint64_t* partials, uint32_t nb, uint64_t* out) {
  hipLaunchKernelGGL(k_sum_u128_part, dim3(nb), dim3(NB), 0, s, x, n, partials);
  hipLaunchKernelGGL(k_colsum_u128, dim3(1), dim3(NB), 0, s, partials, nb, 1u, out);
}


void launch_score_validate(hipStream_t s, const double* S, uint64_t n, uint32_t* err) {
  hipLaunchKernelGGL(k_score_validate, dim3(grid_for(n, 256)), dim3(256), 0, s, S, n, err);
}

void launch_score_keys(hipStream_t s, const uint32_t* score_key, const double* S, uint64_t n, uint64_t* k_key,
                       uint64_t* k_sval, uint32_t* idx) {
  hipLaunchKernelGGL(k_score_keys, dim3(grid_for(n, 256)), dim3(256), 0, s, score_key, S, n, k_key, k_sval, idx);
}

void launch_dup_check(hipStream_t s, const uint64_t* sorted_keys, uint64_t n, uint32_t* err) {
  hipLaunchKernelGGL(k_dup_check, dim3(grid_for(n, 256)), dim3(256), 0, s, sorted_keys, n, err);
}

void launch_score_opkeys(hipStream_t s, const uint32_t* score_key, const uint32_t* idx, uint64_t n, uint64_t* k_op) {
  hipLaunchKernelGGL(k_score_opkeys, dim3(grid_for(n, 256)), dim3(256), 0, s, score_key, idx, n, k_op);
}

void launch_heads_u64(hipStream_t s, const uint64_t* k, uint64_t n, uint32_t* flags) {
  hipLaunchKernelGGL(k_heads_u64, dim3(grid_for(n, 256)), dim3(256), 0, s, k, n, flags);
}

void launch_score_ops(hipStream_t s, const uint32_t* score_key, const double* S, const uint32_t* order,
                      const uint32_t* starts, uint64_t nops, uint64_t n, UnitTable opt, uint64_t nops_trace,
                      uint32_t* r_op, uint64_t* r_U, double* r_S) {
  (void)n;
  if (nops)
    hipLaunchKernelGGL(k_score_ops, dim3(grid_for(nops, 256)), dim3(256), 0, s, score_key, S, order, starts, nops, opt,
                       nops_trace, r_op, r_U, r_S);
}

void launch_score_opiota(hipStream_t s, const uint32_t* score_key, uint64_t n, uint64_t* k_op, uint32_t* idx) {
  hipLaunchKernelGGL(k_score_opiota, dim3(grid_for(n, 256)), dim3(256), 0, s, score_key, n, k_op, idx);
}

void launch_seg_maxlen(hipStream_t s, const uint32_t* flags, const uint32_t* scan, uint64_t n, const uint32_t* starts,
                       uint32_t* out) {
  hipLaunchKernelGGL(k_seg_maxlen, dim3(256), dim3(256), 0, s, flags, scan, n, starts, out);
}

void launch_score_seg(hipStream_t s, const uint32_t* score_key, const double* S, const uint32_t* order,
                      const uint32_t* starts, uint64_t nseg, uint32_t maxlen, const UnitTable& opt, uint64_t nops_trace,
                      uint32_t* r_op, uint64_t* r_U, double* r_S, uint32_t* err) {
  uint32_t N2 = 1;
  while (N2 < maxlen) N2 <<= 1;
  if (nseg)
    hipLaunchKernelGGL(k_score_seg, dim3((uint32_t)nseg), dim3(256), (size_t)N2 * 16, s, score_key, S, order, starts,
                       N2, opt, nops_trace, r_op, r_U, r_S, err);
}

void launch_score_final(hipStream_t s, const uint32_t* r_op, const uint64_t* r_U, const double* r_S, uint64_t nops,
                        const uint64_t* totalU, uint32_t* op, double* op_weight, double* op_score, double* s_agg,
                        uint32_t* err) {
  (void)err;
  hipLaunchKernelGGL(k_score_final, dim3(1), dim3(1024), 0, s, r_op, r_U, r_S, nops, totalU, op, op_weight, op_score,
                     s_agg);
}

hipError_t set_normalize_smem_limits() {
  return hipFuncSetAttribute((const void*)k_score_seg, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)(kScoreSegMax * 16));
}
