// kernels_share.hip -- gfx950 kernels of the plain device-time group-by
// (events that carry no application) and of the target-DSL device-time share
// (§4.1, Metrics: per (operator, shape) the share of device time spent inside
// the target DSL, its mean over each operator's running shapes, and the mean
// of those over the operators where it is defined).
//
// Every mean is exact before its one rounding: a share or an operator mean
// is a double in [2^-110, 1] (or 0), hence an integer multiple of 2^-170 below
// 2^171; the sum of up to 2^16 of them is kept exactly as four 48-bit chunks
// in 64-bit words (no carries between the words: 2^16 terms of < 2^48 each),
// and the quotient by the count is rounded to the nearest double once.  The
// result therefore does not depend on the order in which lanes, waves or
// workgroups add their terms.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr int kFixShift = 905;  // a double with biased exponent E and mantissa m is m 2^(E - 905) units of 2^-170
constexpr uint64_t kChunkMask = ((uint64_t)1 << 48) - 1;

// ---------------------------------------------------------------------------
// Per-phase device time of events without applications: T[ph] += sum of dur
// (u128), cnt[ph] += invocations, with the range checks ph < P and dur >= 0.
// Each thread keeps a private LDS row of P entries (low word, wrap count,
// invocation count): its additions meet no other thread's, so they need no
// atomics.  The workgroup then sums the rows per phase and adds the totals to
// the global words with one atomic per phase.  VEC: four events per thread
// per step with 16-byte loads (16-byte aligned dur, 4-byte aligned phase).
template <int BLOCK, bool VEC>
__global__ __launch_bounds__(BLOCK) void k_time_totals(const uint8_t* __restrict__ phase,
                                                       const int64_t* __restrict__ dur, uint64_t n, uint32_t P,
                                                       unsigned long long* __restrict__ T,
                                                       unsigned long long* __restrict__ cnt,
                                                       uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long s_lo[];    // [P][BLOCK]
  uint32_t* s_wrap = (uint32_t*)(s_lo + P * BLOCK);  // [P][BLOCK]
  uint32_t* s_n = s_wrap + P * BLOCK;                // [P][BLOCK]
  __shared__ unsigned long long s_part[BLOCK / 64][8][3];
  const uint32_t tid = threadIdx.x;
  for (uint32_t p = 0; p < P; ++p) {
    s_lo[p * BLOCK + tid] = 0;
    s_wrap[p * BLOCK + tid] = 0;
    s_n[p * BLOCK + tid] = 0;
  }
  bool bad = false;
  auto one = [&](uint32_t ph, int64_t dd) {
    const bool ok = ph < P && dd >= 0;
    bad |= !ok;
    if (ok) {
      const uint32_t x = ph * BLOCK + tid;
      const unsigned long long lo = s_lo[x], nlo = lo + (unsigned long long)dd;
      s_lo[x] = nlo;
      s_wrap[x] += nlo < lo ? 1u : 0u;
      s_n[x] += 1u;
    }
  };
  const uint64_t stride = (uint64_t)gridDim.x * BLOCK;
  if (VEC) {
    const uint64_t n4 = n / 4;
    for (uint64_t q = (uint64_t)blockIdx.x * BLOCK + tid; q < n4; q += stride) {
      const uint32_t p4 = __builtin_nontemporal_load((const uint32_t*)(phase + 4 * q));
      const v2l d0 = __builtin_nontemporal_load((const v2l*)(dur + 4 * q));
      const v2l d1 = __builtin_nontemporal_load((const v2l*)(dur + 4 * q + 2));
      one(p4 & 0xFFu, d0.x);
      one((p4 >> 8) & 0xFFu, d0.y);
      one((p4 >> 16) & 0xFFu, d1.x);
      one(p4 >> 24, d1.y);
    }
    if (blockIdx.x == 0)
      for (uint64_t i = n4 * 4 + tid; i < n; i += BLOCK) one(phase[i], dur[i]);
  } else {
    for (uint64_t i = (uint64_t)blockIdx.x * BLOCK + tid; i < n; i += stride) one(phase[i], dur[i]);
  }
  if (__any(bad) && (tid & 63) == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
  // per phase: each wave sums its lanes' rows, one lane per phase then sums
  // the waves and adds the workgroup's total
  const uint32_t wave = tid / 64, lane = tid & 63;
  for (uint32_t p = 0; p < P; ++p) {
    const uint32_t x = p * BLOCK + tid;
    const u128 v = wave_sum_u128(make_u128(s_lo[x], s_wrap[x]));
    uint64_t c = s_n[x];
    for (int d = 32; d >= 1; d >>= 1) c += __shfl_down(c, d, 64);
    if (lane == 0) {
      s_part[wave][p][0] = (uint64_t)v;
      s_part[wave][p][1] = (uint64_t)(v >> 64);
      s_part[wave][p][2] = c;
    }
  }
  __syncthreads();
  if (tid < P) {
    u128 v = 0;
    uint64_t c = 0;
    for (uint32_t w = 0; w < BLOCK / 64; ++w) {
      v += make_u128(s_part[w][tid][0], s_part[w][tid][1]);
      c += s_part[w][tid][2];
    }
    if (c) {
      acc_add_plain(&T[2 * tid], &T[2 * tid + 1], v);
      atomicAdd(&cnt[tid], (unsigned long long)c);
    }
  }
}

// ---------------------------------------------------------------------------
// Exact sums of doubles in [2^-110, 1] as four 48-bit chunks of units of
// 2^-170, and the rounded mean.
struct Chunks {
  uint64_t c[4];
};

__device__ __forceinline__ Chunks to_chunks(double x) {
  Chunks r = {{0, 0, 0, 0}};
  if (!(x > 0.0)) return r;
  const uint64_t b = (uint64_t)__double_as_longlong(x);
  const uint64_t m = (b & (((uint64_t)1 << 52) - 1)) | ((uint64_t)1 << 52);
  const int sh = (int)(b >> 52) - kFixShift;  // >= 8 for x >= 2^-110, <= 118 for x <= 1
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int s = sh - 48 * k;  // chunk k = (m 2^sh) >> 48k, i.e. m shifted by sh - 48k
    const uint64_t v = s >= 0 ? (s < 64 ? m << s : 0) : (-s < 64 ? m >> -s : 0);
    r.c[k] = v & kChunkMask;
  }
  return r;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
  return v;
}

// RN(X 2^-170 / n) for X = sum_k c[k] 2^(48k) (< 2^192) and 1 <= n <= 2^17
// (a count of shapes or operators).  q = floor(X 2^64 / n) by long division
// in 32-bit limbs: each step divides r 2^32 + limb < 2^49 by n, exactly
// representable in fp64, and fixes the fp64 quotient by at most one with the
// exact remainder.  The top 64 bits of q, with a sticky bit for every lower
// bit and the final remainder, round to the same double as the exact
// quotient (q has more than 64 bits whenever X >= 2^60, which holds for every
// nonzero sum here).  All limbs stay in registers (constant indices only).
__device__ double chunks_mean(const Chunks& s, uint64_t n) {
  uint64_t w[4];
  {
    const u128 lo = (u128)s.c[0] + ((u128)s.c[1] << 48);  // chunks 0, 1
    w[0] = (uint64_t)lo;
    u128 acc = (lo >> 64) + ((u128)s.c[2] << 32);         // chunk 2: 2^96 = 2^64 2^32
    w[1] = (uint64_t)acc;
    acc = (acc >> 64) + ((u128)s.c[3] << 16);              // chunk 3: 2^144 = 2^128 2^16
    w[2] = (uint64_t)acc;
    w[3] = (uint64_t)(acc >> 64);
  }
  // numerator X 2^64 as ten 32-bit limbs, least significant first
  const uint32_t num[10] = {0, 0, (uint32_t)w[0], (uint32_t)(w[0] >> 32), (uint32_t)w[1], (uint32_t)(w[1] >> 32),
                            (uint32_t)w[2], (uint32_t)(w[2] >> 32), (uint32_t)w[3], (uint32_t)(w[3] >> 32)};
  const double nd = (double)n;
  uint32_t q[10];
  uint64_t r = 0;
#pragma unroll
  for (int i = 9; i >= 0; --i) {
    const uint64_t cur = (r << 32) | num[i];  // < n 2^32 <= 2^49
    int64_t qi = (int64_t)((double)cur / nd);
    int64_t rem = (int64_t)cur - qi * (int64_t)n;
    if (rem < 0) { --qi; rem += (int64_t)n; }
    if (rem >= (int64_t)n) { ++qi; rem -= (int64_t)n; }
    q[i] = (uint32_t)qi;
    r = (uint64_t)rem;
  }
  // leading limb, and the three limbs from it down (selects, no indexing)
  int top = -1;
#pragma unroll
  for (int i = 0; i < 10; ++i) top = q[i] ? i : top;
  if (top < 0) return 0.0;
  uint32_t l0 = 0, l1 = 0, l2 = 0;
  bool sticky = r != 0;
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    l0 = i == top ? q[i] : l0;
    l1 = i == top - 1 ? q[i] : l1;
    l2 = i == top - 2 ? q[i] : l2;
    sticky |= (i < top - 2) && q[i] != 0;
  }
  const int lz = __clz((int)l0);
  const int bl = 32 * top + 32 - lz;  // bit length of q
  // the 96-bit window l0:l1:l2 aligned so that q's leading one is its bit 95
  const u128 win = (((u128)l0 << 64) | ((u128)l1 << 32) | l2) << lz;
  // (when q has fewer than 64 bits, t is q itself shifted left, exactly)
  uint64_t t = (uint64_t)(win >> 32);
  sticky |= (uint32_t)win != 0;
  t |= sticky ? 1u : 0u;
  const double d = ldexp((double)(uint32_t)(t >> 32), 32) + (double)(uint32_t)t;  // the one rounding
  return ldexp(d, (bl - 64) - 64 - 170);  // t's last bit weighs 2^(bl - 64) units of q
}

// ---------------------------------------------------------------------------
// Heads of the key and operator runs in groups ordered by (key, phase).
__global__ void k_share_heads(const uint32_t* __restrict__ key, uint64_t G, uint32_t* __restrict__ hk,
                              uint32_t* __restrict__ ho) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  const uint32_t k = key[g];
  const bool nk = g == 0 || key[g - 1] != k;
  hk[g] = nk ? 1u : 0u;
  ho[g] = (nk && (g == 0 || (key[g - 1] >> 16) != (k >> 16))) ? 1u : 0u;
}

// One thread per key run: the key's DSL time (phase 1) and total time, its
// share, the operator's first key, and (last group) the key and operator
// counts.  Outputs past the caller's capacities are not written.
__global__ void k_share_keys(SortedGroups g, uint64_t G, const uint32_t* __restrict__ hk,
                             const uint32_t* __restrict__ kidx, const uint32_t* __restrict__ ho,
                             const uint32_t* __restrict__ oidx, ShareOut out, uint64_t kcap, uint64_t ocap,
                             double* __restrict__ share_all, uint32_t* __restrict__ op_first,
                             unsigned long long* __restrict__ words) {
  const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= G) return;
  if (r == G - 1) {
    const uint64_t K = (uint64_t)kidx[r] + hk[r], I = (uint64_t)oidx[r] + ho[r];
    words[0] = K;
    words[1] = I;
    op_first[I] = (uint32_t)K;  // end of the last operator's keys
  }
  if (!hk[r]) return;
  const uint32_t k = g.key[r];
  u128 dsl = 0, tot = 0;
  uint64_t n = 0;
  for (uint64_t x = r; x < G && x < r + 8 && g.key[x] == k; ++x) {  // at most one group per phase
    const u128 w = make_u128(g.wsum[2 * x], g.wsum[2 * x + 1]);
    tot += w;
    if (g.phase[x] == 1) dsl += w;
    n += g.count[x];
  }
  const double sh = tot ? u128_to_f64(dsl) / u128_to_f64(tot) : __builtin_nan("");
  const uint32_t i = kidx[r];
  share_all[i] = sh;
  if (i < kcap) {
    out.key[i] = k;
    out.count[i] = n;
    out.dsl[2 * i] = (uint64_t)dsl;
    out.dsl[2 * i + 1] = (uint64_t)(dsl >> 64);
    out.total[2 * i] = (uint64_t)tot;
    out.total[2 * i + 1] = (uint64_t)(tot >> 64);
    out.share[i] = sh;
  }
  if (ho[r]) {
    const uint32_t o = oidx[r];
    op_first[o] = i;
    if (o < ocap) out.op[o] = k >> 16;
  }
}

// One wave per operator: the exact mean share over its running shapes (keys
// whose share is not NaN), and the operator's term of the overall mean.
__global__ __launch_bounds__(256) void k_share_ops(const double* __restrict__ share_all,
                                                   const uint32_t* __restrict__ op_first, ShareOut out,
                                                   uint64_t ocap, unsigned long long* __restrict__ words) {
  const uint32_t o = blockIdx.x * 4 + threadIdx.x / 64, lane = threadIdx.x & 63;
  const uint64_t I = __hip_atomic_load(&words[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (o >= I) return;  // wave-uniform
  const uint32_t b = op_first[o], e = op_first[o + 1];
  Chunks s = {{0, 0, 0, 0}};
  uint64_t running = 0;
  for (uint32_t i = b + lane; i < e; i += 64) {
    const double x = share_all[i];
    if (x == x) {  // not NaN: the shape ran
      const Chunks c = to_chunks(x);
      for (int k = 0; k < 4; ++k) s.c[k] += c.c[k];
      ++running;
    }
  }
  for (int k = 0; k < 4; ++k) s.c[k] = wave_sum_u64(s.c[k]);
  running = wave_sum_u64(running);
  if (lane == 0) {
    const double mean = running ? chunks_mean(s, running) : __builtin_nan("");
    if (o < ocap) {
      out.op_shapes[o] = (uint32_t)running;
      out.op_share[o] = mean;
    }
    if (running) {
      const Chunks c = to_chunks(mean);
      for (int k = 0; k < 4; ++k) atomicAdd(&words[4 + k], (unsigned long long)c.c[k]);
      atomicAdd(&words[2], 1ull);
    }
  }
}

// The mean over the operators where the share is defined (words[3], NaN when
// none is).
__global__ void k_share_final(unsigned long long* __restrict__ words) {
  if (threadIdx.x != 0) return;
  const uint64_t nd = words[2];
  Chunks s;
  for (int k = 0; k < 4; ++k) s.c[k] = words[4 + k];
  const double a = nd ? chunks_mean(s, nd) : __builtin_nan("");
  words[3] = (unsigned long long)__double_as_longlong(a);
}

}  // namespace

// ---------------------------------------------------------------------------
// Host launchers
void launch_time_totals(hipStream_t s, const EventsDev& ev, uint32_t P, uint32_t nblocks, bool vec,
                        unsigned long long* T, unsigned long long* cnt, uint32_t* err) {
  const size_t smem = (size_t)P * 1024 * 16;
  if (vec)
    hipLaunchKernelGGL((k_time_totals<1024, true>), dim3(nblocks), dim3(1024), smem, s, ev.phase, ev.dur, ev.n, P,
                       T, cnt, err);
  else
    hipLaunchKernelGGL((k_time_totals<1024, false>), dim3(nblocks), dim3(1024), smem, s, ev.phase, ev.dur, ev.n, P,
                       T, cnt, err);
}

void launch_target_share(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t* hk, uint32_t* kidx,
                         uint32_t* ho, uint32_t* oidx, void* scan_tmp, const ShareOut& out, uint64_t kcap,
                         uint64_t ocap, double* share_all, uint32_t* op_first, unsigned long long* words) {
  launch_fill_u64(s, (uint64_t*)words, 8, 0);
  if (G) {
    const uint32_t nb = (uint32_t)((G + 255) / 256);
    hipLaunchKernelGGL(k_share_heads, dim3(nb), dim3(256), 0, s, g.key, G, hk, ho);
    exclusive_scan_u32(s, hk, kidx, G, scan_tmp);
    exclusive_scan_u32(s, ho, oidx, G, scan_tmp);
    hipLaunchKernelGGL(k_share_keys, dim3(nb), dim3(256), 0, s, g, G, hk, kidx, ho, oidx, out, kcap, ocap,
                       share_all, op_first, words);
    // operators: at most min(G, 2^16) (the operator is the key's top 16 bits)
    const uint64_t maxops = G < 65536 ? G : 65536;
    hipLaunchKernelGGL(k_share_ops, dim3((uint32_t)((maxops + 3) / 4)), dim3(256), 0, s, share_all, op_first, out,
                       ocap, words);
  }
  hipLaunchKernelGGL(k_share_final, dim3(1), dim3(64), 0, s, words);
}

hipError_t set_share_smem_limits() {
  const void* fns[] = {(const void*)k_time_totals<1024, true>, (const void*)k_time_totals<1024, false>};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 8 * 1024 * 16);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
