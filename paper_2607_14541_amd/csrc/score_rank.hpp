// score_rank.hpp -- the ranking step of the importance-weighted roofline score
// (§3.6, Eq. (4)-(6)) for up to kScoreRankMax scored units, as a device
// function of one 1024-thread workgroup, so that the score kernel and the
// one-call path's combined launch share it.
//
// Workgroup `blk` ranks units [16 blk, 16 blk + 16), one wave each: Eq. (4)
// validation (S_j in (0, 1], NaN = not correct), the duplicate-key check, and
// the unit's position in the order (operator, S, index) -- NaN after every
// value of its operator -- counted against every unit staged in LDS (12 B per
// unit of dynamic LDS); the unit is written at that position.  No sort.
#pragma once

#include "atrex_device.hpp"

constexpr uint32_t kRankThreads = 1024;
constexpr uint32_t kRankPerBlock = kRankThreads / 64;  // units ranked per workgroup: one wave each

__device__ __forceinline__ uint64_t score_order_bits(double v) {
  return isnan(v) ? ~0ull : (uint64_t)__double_as_longlong(v);  // S > 0: bits order as values
}

__device__ __forceinline__ void score_rank_block(uint32_t blk, const uint32_t* __restrict__ score_key,
                                                 const double* __restrict__ S, uint32_t n,
                                                 uint32_t* __restrict__ sorted_op, double* __restrict__ sorted_S,
                                                 uint32_t* __restrict__ err, uint64_t* smem64) {
  uint64_t* s_sb = smem64;                  // [n]
  uint32_t* s_key = (uint32_t*)(s_sb + n);  // [n]
  const uint32_t tid = threadIdx.x, lane = tid & 63;
  lds_stage<kRankThreads, 8>(s_sb, S, n, [](double v) { return score_order_bits(v); });
  lds_stage<kRankThreads, 8>(s_key, score_key, n, [](uint32_t k) { return k; });
  __syncthreads();
  const uint32_t m = blk * kRankPerBlock + (tid >> 6);  // this wave's unit
  if (m >= n) return;                                 // wave-uniform
  const uint32_t key_m = s_key[m], op_m = key_m >> 16;
  const uint64_t sb_m = s_sb[m];
  uint32_t below = 0;
  bool dup = false;
#pragma unroll 4
  for (uint32_t j = lane; j < n; j += 64) {
    const uint32_t kj = s_key[j], oj = kj >> 16;
    const uint64_t sj = s_sb[j];
    below += (oj < op_m || (oj == op_m && (sj < sb_m || (sj == sb_m && j < m)))) ? 1u : 0u;
    dup |= kj == key_m && j != m;
  }
  for (int d = 32; d >= 1; d >>= 1) below += __shfl_xor(below, d, 64);
  if (lane == 0) {
    const double v = S[m];
    sorted_op[below] = op_m;
    sorted_S[below] = v;
    if (!isnan(v) && !(v > 0.0 && v <= 1.0)) atomicOr(err, ATREX_ERRBIT_RANGE);
  }
  if (__any(dup) && lane == 0) atomicOr(err, ATREX_ERRBIT_DUP);
}
