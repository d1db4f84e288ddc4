// kernels_aggregate.hip -- gfx950 kernels for the group-by of §3.4:
//   pass A  (Eq. (2)): T[a,ph] = sum of dur over the invocations of (a, ph)
//   scale   (Eq. (3)): the Q96 factor p_a / T[a,ph] as (m, rho)
//   pass B  (Eq. (2)-(3)): W[k,ph] = sum over invocations of dur * p_a / T[a,ph]
//   compaction of the distinct (key, phase) groups.
// Events are a struct of arrays (key u32, app u32, phase u8, dur i64) read
// with 16-byte nontemporal vector loads, four events per thread per step.
#include <algorithm>

#include "atrex_device.hpp"
#include "atrex_kernels.h"


namespace {

__device__ __forceinline__ void flag_error(uint32_t* err, bool bad, uint32_t bit) {
  // one atomic per wave that saw a bad event
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, bit);
}

// ---------------------------------------------------------------------------
// Pass A, LDS-privatised dense histogram on g = a * P + ph.  Each workgroup
// keeps the low 64 bits of its partial sums in LDS; the (rare) wrap-arounds
// are counted in a global carry table.  Partials go to partial[block][g].
// COUNT: the invocations of each g are counted too (a u32 table after the
// sums; a workgroup sees fewer than 2^31 events), partial counts to
// pcount[block][g].
template <int BLOCK, bool COUNT>
__global__ __launch_bounds__(BLOCK) void k_pass_a_lds(EventsDev ev, uint32_t A, uint32_t P, uint32_t G,
                                                      unsigned long long* __restrict__ partial,
                                                      unsigned long long* __restrict__ carry,
                                                      uint32_t* __restrict__ pcount, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long s_lo[];
  uint32_t* s_n = (uint32_t*)(s_lo + G);  // COUNT only
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) {
    s_lo[g] = 0;
    if (COUNT) s_n[g] = 0;
  }
  __syncthreads();
  const uint64_t n = ev.n, n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * BLOCK;
  bool bad = false;
  auto one = [&](uint32_t a, uint32_t ph, int64_t dd) {
    const bool ok = a < A && ph < P && dd >= 0;
    bad |= !ok;
    if (ok) {
      const uint32_t g = a * P + ph;
      const unsigned long long d = (unsigned long long)dd;
      const unsigned long long old = atomicAdd(&s_lo[g], d);
      if (old + d < old) atomicAdd(&carry[g], 1ull);
      if (COUNT) atomicAdd(&s_n[g], 1u);
    }
  };
  // the next two groups' loads are issued before the current group is added
  uint64_t q = (uint64_t)blockIdx.x * BLOCK + threadIdx.x;
  Ev4 nxt, nxt2;
  if (q < n4) load4<false>(ev.key, ev.app, ev.phase, ev.dur, q * 4, nxt);
  if (q + stride < n4) load4<false>(ev.key, ev.app, ev.phase, ev.dur, (q + stride) * 4, nxt2);
  for (; q < n4; q += stride) {
    const Ev4 e = nxt;
    nxt = nxt2;
    if (q + 2 * stride < n4) load4<false>(ev.key, ev.app, ev.phase, ev.dur, (q + 2 * stride) * 4, nxt2);
#pragma unroll
    for (int j = 0; j < 4; ++j) one(e.app[j], e.ph(j), e.dur[j]);
  }
  if (blockIdx.x == 0)  // tail events
    for (uint64_t i = n4 * 4 + threadIdx.x; i < n; i += BLOCK) one(ev.app[i], ev.phase[i], ev.dur[i]);
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
  __syncthreads();
  unsigned long long* out = partial + (size_t)blockIdx.x * G;
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) {
    out[g] = s_lo[g];
    if (COUNT) pcount[(size_t)blockIdx.x * G + g] = s_n[g];
  }
}

// Pass A with 32-bit LDS accumulators (twice the (app, phase) capacity of the
// 64-bit table).  A wrap of the 32-bit sum and the high half of a duration
// are both counted in ext[g] in units of 2^32 (global atomics, rare: only
// when a workgroup's partial sum of one (app, phase) passes 2^32, or for a
// duration of 2^32 ns or more).  COUNT as in k_pass_a_lds.
template <int BLOCK, bool COUNT>
__global__ __launch_bounds__(BLOCK) void k_pass_a_lds32(EventsDev ev, uint32_t A, uint32_t P, uint32_t G,
                                                        uint32_t* __restrict__ partial,
                                                        unsigned long long* __restrict__ ext,
                                                        uint32_t* __restrict__ pcount, uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s32[];
  uint32_t* s_n = s32 + G;  // COUNT only
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) {
    s32[g] = 0;
    if (COUNT) s_n[g] = 0;
  }
  __syncthreads();
  const uint64_t n = ev.n, n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * BLOCK;
  bool bad = false;
  auto one = [&](uint32_t a, uint32_t ph, int64_t dd) {
    const bool ok = a < A && ph < P && dd >= 0;
    bad |= !ok;
    if (!ok) return;
    const uint32_t g = a * P + ph;
    const uint64_t d = (uint64_t)dd;
    const uint32_t lo = (uint32_t)d;
    const uint32_t old = atomicAdd(&s32[g], lo);
    const uint64_t up = (d >> 32) + ((old + lo < old) ? 1u : 0u);
    if (up) atomicAdd(&ext[g], (unsigned long long)up);
    if (COUNT) atomicAdd(&s_n[g], 1u);
  };
  uint64_t q = (uint64_t)blockIdx.x * BLOCK + threadIdx.x;
  Ev4 nxt;
  if (q < n4) load4<false>(ev.key, ev.app, ev.phase, ev.dur, q * 4, nxt);
  for (; q < n4; q += stride) {
    const Ev4 e = nxt;
    if (q + stride < n4) load4<false>(ev.key, ev.app, ev.phase, ev.dur, (q + stride) * 4, nxt);
#pragma unroll
    for (int j = 0; j < 4; ++j) one(e.app[j], e.ph(j), e.dur[j]);
  }
  if (blockIdx.x == 0)
    for (uint64_t i = n4 * 4 + threadIdx.x; i < n; i += BLOCK) one(ev.app[i], ev.phase[i], ev.dur[i]);
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
  __syncthreads();
  uint32_t* out = partial + (size_t)blockIdx.x * G;
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) {
    out[g] = s32[g];
    if (COUNT) pcount[(size_t)blockIdx.x * G + g] = s_n[g];
  }
}

constexpr int RANGE_DEPTH = 6;  // groups of four events in flight per lane in k_pass_a_range

// Pass A for more (app, phase) pairs than one LDS holds: the pairs are split
// into R ranges of at most GR, the events into `slices`; each workgroup sums
// one (slice, range) in 32-bit LDS counters (wraps and high halves into ext[g]
// as in k_pass_a_lds32).  The R workgroups of a slice are placed on one XCD
// (workgroups go round-robin over the 8 XCDs) and walk the slice in the same
// order with ordinary (L2-allocating) loads, so the slice comes from HBM about
// once and from that XCD's L2 for the others.  Each lane keeps RANGE_DEPTH
// groups of four events in flight.  COUNT: a u32
// count table after the GR counters and their spares.
//
// HIST: workgroup w < hj.nwg also takes the partition histogram of the hot
// scatter's range w (as k_part_hist<true>: the keys outside the seeded image,
// per bucket), one group of four keys per lane after every RANGE_DEPTH groups
// of events, in the time this pass spends waiting on L2.
template <int BLOCK, bool COUNT, bool HIST>
__global__ __launch_bounds__(BLOCK) void k_pass_a_range(EventsDev ev, uint32_t A, uint32_t P, uint32_t G,
                                                        uint32_t GR, uint32_t R, uint32_t slices,
                                                        uint32_t* __restrict__ partial,
                                                        unsigned long long* __restrict__ ext,
                                                        uint32_t* __restrict__ pcount, HistJob hj,
                                                        uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s32[];
  uint32_t* s_n = s32 + GR + 64;  // COUNT only
  // HIST: bucket counters and the image, 16-byte aligned after the tables
  uint32_t* s_h = s32 + (((COUNT ? 2 * GR : GR) + 64 + 3) & ~3u);
  uint32_t* s_img = s_h + (HIST ? (1u << hj.BB) : 0u);
  const uint32_t xcd = blockIdx.x % 8, k = blockIdx.x / 8;
  const uint32_t slice = (k / R) * 8 + xcd, range = k % R;
  const bool sums = slice < slices;                 // uniform over the workgroup
  const bool hist = HIST && blockIdx.x < hj.nwg;    // uniform
  if (!sums && !hist) return;
  const uint32_t g0 = range * GR, g1 = sums ? min(G, g0 + GR) : g0;
  for (uint32_t g = threadIdx.x; g < g1 - g0; g += BLOCK) {
    s32[g] = 0;
    if (COUNT) s_n[g] = 0;
  }
  if (hist) {
    for (uint32_t i = threadIdx.x; i < (1u << hj.BB); i += BLOCK) s_h[i] = 0;
    for (uint32_t i = threadIdx.x; i < hj.S; i += BLOCK) s_img[i] = hj.seed[i];
  }
  __syncthreads();
  // the histogram's range [hb, he) and its groups of four keys
  const uint64_t hb = hist ? min(hj.n, (uint64_t)blockIdx.x * hj.per) : 0;
  const uint64_t he = hist ? min(hj.n, hb + hj.per) : 0;
  const uint64_t hng = (he - hb) / 4, hiters = (hng + BLOCK - 1) / BLOCK;
  const uint32_t hsh = 32 - hj.BB;
  uint64_t hi = 0;
  v4u hk = {0, 0, 0, 0};
  auto hload = [&](uint64_t j) {
    const uint64_t gi = j * BLOCK + threadIdx.x;
    if (gi < hng) hk = __builtin_nontemporal_load((const v4u*)(hj.key + hb + 4 * gi));
  };
  // plain no-return LDS atomics: the keys outside the image are the colder
  // ones, spread over the buckets (the hot keys are the image's)
  auto hstep = [&]() {  // uniform: every lane of the workgroup calls it
    const bool v = hi * BLOCK + threadIdx.x < hng;
    const v4u kk = hk;
    if (hi + 1 < hiters) hload(hi + 1);
    const uint32_t kv[4] = {kk.x, kk.y, kk.z, kk.w};
    bool cold[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cold[j] = v && image_slot(s_img, hj.S, kv[j]) == ATREX_NO_SLOT;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (cold[j]) atomicAdd(&s_h[hash32(kv[j]) >> hsh], 1u);
    ++hi;
  };
  if (HIST && hiters) hload(0);
  const uint64_t n = ev.n;
  const uint64_t per = ((n + slices - 1) / slices + 3) / 4 * 4;
  const uint64_t b = sums ? min(n, (uint64_t)slice * per) : 0, e = sums ? min(n, b + per) : 0;
  bool bad = false;
  auto one = [&](uint32_t a, uint32_t ph, int64_t dd) {
    const bool ok = a < A && ph < P && dd >= 0;
    bad |= !ok;
    const uint32_t g = a * P + ph;
    if (!ok || g < g0 || g >= g1) return;
    const uint64_t d = (uint64_t)dd;
    const uint32_t lo = (uint32_t)d;
    const uint32_t old = atomicAdd(&s32[g - g0], lo);
    const uint64_t up = (d >> 32) + ((old + lo < old) ? 1u : 0u);
    if (up) atomicAdd(&ext[g], (unsigned long long)up);
    if (COUNT) atomicAdd(&s_n[g - g0], 1u);
  };
  // groups of four events of the slice: iteration `it` covers groups
  // it * BLOCK + [0, BLOCK); the trip count is uniform over the workgroup
  const uint64_t ng = (e - b) / 4;
  const uint64_t iters = (ng + BLOCK - 1) / BLOCK;
  struct G4 {
    v4u a;
    uint32_t p;
    v2l d0, d1;
  };
  auto load = [&](uint64_t it, G4& x) {
    const uint64_t gi = it * BLOCK + threadIdx.x;
    if (gi < ng) {
      const uint64_t i = b + 4 * gi;
      x.a = *(const v4u*)(ev.app + i);
      x.p = *(const uint32_t*)(ev.phase + i);
      x.d0 = *(const v2l*)(ev.dur + i);
      x.d1 = *(const v2l*)(ev.dur + i + 2);
    }
  };
  // Four events without branches.  An event outside the range adds to a
  // per-lane spare counter past the range, so the four LDS atomics issue back
  // to back and are waited for once (an atomic masked to the lanes in range
  // would be waited for before the next one is issued).  When every lane's four
  // events are valid (the usual case, checked for the group at once: largest
  // app, the phase bytes, the sign of the durations) the counter's byte offset
  // and the range test need no per-event validity; otherwise the wave takes the
  // per-event checks.  The high words and wrap-arounds go to ext[g] only when
  // present.  COUNT: the counts are added with no-return atomics, in range only.
  const uint32_t gn = g1 - g0, lane = threadIdx.x & 63;
  const uint32_t spare4 = 4 * (GR + lane), gn4 = 4 * gn, P4 = 4 * P, g04 = 4 * g0;
  const uint32_t pbytes = P * 0x01010101u;  // P in every byte (P <= 128)
  auto process = [&](uint64_t it, const G4& x) {
    if (it * BLOCK + threadIdx.x >= ng) return;
    const uint32_t av[4] = {x.a.x, x.a.y, x.a.z, x.a.w};
    const int64_t dv[4] = {x.d0.x, x.d0.y, x.d1.x, x.d1.y};
    uint32_t dhi[4], old[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) dhi[j] = (uint32_t)((uint64_t)dv[j] >> 32);
    // byte b of `pbad` has its top bit set iff phase byte b >= P (or >= 128)
    const uint32_t pbad = (x.p | ((x.p | 0x80808080u) - pbytes)) & 0x80808080u;
    const uint32_t amax = max(max(av[0], av[1]), max(av[2], av[3]));
    const uint32_t hor = dhi[0] | dhi[1] | dhi[2] | dhi[3];
    const bool valid = (amax < A) & (pbad == 0) & ((int32_t)hor >= 0);
    if (__all(valid)) {
      uint32_t rb[4];
      bool in[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // 4 (a P + ph - g0): a < A < 2^24 and 4 A P < 2^32
        rb[j] = __umul24(av[j], P4) + ((((x.p >> (8 * j)) & 0xFFu) << 2) - g04);
        in[j] = rb[j] < gn4;
        rb[j] = in[j] ? rb[j] : spare4;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) old[j] = atomicAdd((uint32_t*)((char*)s32 + rb[j]), (uint32_t)dv[j]);
      if (COUNT) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (in[j]) atomicAdd((uint32_t*)((char*)s_n + rb[j]), 1u);
      }
      bool cy = false;
#pragma unroll
      for (int j = 0; j < 4; ++j) cy |= in[j] & (old[j] + (uint32_t)dv[j] < old[j]);
      if (__any(cy | (hor != 0)))
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t up = dhi[j] + ((old[j] + (uint32_t)dv[j] < old[j]) ? 1u : 0u);  // < 2^31 + 1
          if (in[j] && up) atomicAdd(&ext[g0 + rb[j] / 4], (unsigned long long)up);
        }
      return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) one(av[j], (x.p >> (8 * j)) & 0xFFu, dv[j]);
  };
  // a ring of DEPTH groups per lane: group it is processed while the loads of
  // the next DEPTH - 1 are in flight (the loads come from L2 with a long
  // latency under the R-fold re-reads; the waves would otherwise wait on them)
  G4 x[RANGE_DEPTH];
#pragma unroll
  for (int k = 0; k < RANGE_DEPTH; ++k)
    if ((uint64_t)k < iters) load(k, x[k]);
  for (uint64_t it = 0; it < iters; it += RANGE_DEPTH) {
#pragma unroll
    for (int k = 0; k < RANGE_DEPTH; ++k) {
      if (it + k >= iters) break;
      process(it + k, x[k]);
      if (it + k + RANGE_DEPTH < iters) load(it + k + RANGE_DEPTH, x[k]);
    }
    if (HIST && hi < hiters) hstep();
  }
  for (uint64_t i = b + 4 * ng + threadIdx.x; i < e; i += BLOCK) one(ev.app[i], ev.phase[i], ev.dur[i]);
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
  if (HIST) {
    while (hi < hiters) hstep();
    for (uint64_t i = hb + 4 * hng + threadIdx.x; i < he; i += BLOCK) {  // the range's last keys
      const uint32_t kk = hj.key[i];
      if (image_slot(s_img, hj.S, kk) == ATREX_NO_SLOT) atomicAdd(&s_h[hash32(kk) >> hsh], 1u);
    }
  }
  __syncthreads();
  if (sums) {
    uint32_t* out = partial + (size_t)slice * G;
    for (uint32_t g = threadIdx.x; g < g1 - g0; g += BLOCK) {
      out[g0 + g] = s32[g];
      if (COUNT) pcount[(size_t)slice * G + g0 + g] = s_n[g];
    }
  }
  if (hist)
    for (uint32_t i = threadIdx.x; i < (1u << hj.BB); i += BLOCK) hj.H[(size_t)i * hj.nwg + blockIdx.x] = s_h[i];
}

// Pass A straight into global 128-bit accumulators (any number of (a, ph));
// COUNT: invocation counts into cnt[g] (u64, global atomics).
template <int BLOCK, bool COUNT>
__global__ __launch_bounds__(BLOCK) void k_pass_a_global(EventsDev ev, uint32_t A, uint32_t P,
                                                         unsigned long long* __restrict__ T,
                                                         unsigned long long* __restrict__ cnt,
                                                         uint32_t* __restrict__ err) {
  const uint64_t n = ev.n;
  bool bad = false;
  for (uint64_t i = (uint64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (uint64_t)gridDim.x * BLOCK) {
    const uint32_t a = ev.app[i], ph = ev.phase[i];
    const int64_t d = ev.dur[i];
    const bool ok = a < A && ph < P && d >= 0;
    bad |= !ok;
    if (ok) {
      const size_t g = (size_t)a * P + ph;
      acc_add_plain(&T[2 * g], &T[2 * g + 1], (u128)(uint64_t)d);
      if (COUNT) atomicAdd(&cnt[g], 1ull);
    }
  }
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
}

// ---------------------------------------------------------------------------
// Scale, Eq. (3): for each (a, ph) with T > 0 and c_a > 0,
//   r = 2^96 c_a / (C T), rho = floor(log2 r), m = floor(r 2^(55 - rho)).
// With Y = C T, bc = bitlen(c_a), by = bitlen(Y) and r0 = 96 + bc - by, r lies
// in (2^(r0-1), 2^(r0+1)), so q = floor(c_a 2^e / Y) with e = 56 - bc + by
// lies in [2^55, 2^57): if q >= 2^56 then rho = r0 and m = floor(q / 2), else
// rho = r0 - 1 and m = q.  q comes from an fp64 estimate (off by at most a few
// tens), an exact 256-bit remainder R = c_a 2^e - q Y, a second fp64 step
// q += rint(R / Y) that leaves |R| < Y, and a final -1 when R < 0.

// value of a signed 256-bit two's-complement number (4 little-endian limbs),
// rounded to fp64 (exactness is not needed: it feeds an estimate)
__device__ __forceinline__ double s256_to_f64(const uint64_t w[4]) {
  const bool neg = (int64_t)w[3] < 0;
  uint64_t a[4];
  uint64_t br = neg ? 1 : 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // |x| = ~x + 1 when negative
    const uint64_t x = neg ? ~w[i] : w[i];
    a[i] = x + br;
    br = (br && a[i] == 0) ? 1 : 0;
  }
  const double v = ldexp((double)a[3], 192) + ldexp((double)a[2], 128) + ldexp((double)a[1], 64) + (double)a[0];
  return neg ? -v : v;
}

// w -= s * Y (s >= 0 or s < 0, |s| < 2^63), Y = (y0, y1, y2), 256-bit wrap-around
__device__ __forceinline__ void s256_sub_mul(uint64_t w[4], int64_t s, uint64_t y0, uint64_t y1, uint64_t y2) {
  const bool neg = s < 0;
  const uint64_t q = neg ? (uint64_t)(-s) : (uint64_t)s;
  const u128 p0 = (u128)q * y0;
  const u128 p1 = (u128)q * y1 + (uint64_t)(p0 >> 64);
  const u128 p2 = (u128)q * y2 + (uint64_t)(p1 >> 64);
  const uint64_t m[4] = {(uint64_t)p0, (uint64_t)p1, (uint64_t)p2, (uint64_t)(p2 >> 64)};
  uint64_t c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (neg) {  // w += q * Y
      const u128 t = (u128)w[i] + m[i] + c;
      w[i] = (uint64_t)t;
      c = (uint64_t)(t >> 64);
    } else {    // w -= q * Y
      const uint64_t x = w[i];
      const uint64_t d = x - m[i] - c;
      c = (x < m[i] || (x - m[i]) < c) ? 1 : 0;
      w[i] = d;
    }
  }
}

// Scale words of one (app, phase): T > 0 (< 2^94), c_a > 0, C = sum of c (< 2^64).
__device__ __forceinline__ void scale_words(u128 t, uint32_t ca, uint64_t C, uint64_t& sw, uint64_t& bsw) {
  // Y = C * T < 2^158
  const u128 p0 = (u128)C * (uint64_t)t;
  const u128 p1 = (u128)C * (uint64_t)(t >> 64) + (uint64_t)(p0 >> 64);
  const uint64_t y0 = (uint64_t)p0, y1 = (uint64_t)p1, y2 = (uint64_t)(p1 >> 64);
  const int by = y2 ? 192 - __clzll(y2) : y1 ? 128 - __clzll(y1) : 64 - __clzll(y0);
  const int bc = 32 - __clz(ca);
  const int r0 = 96 + bc - by;
  const int e = 56 - bc + by;  // in [25, 213]
  const double yd = ldexp((double)y2, 128) + ldexp((double)y1, 64) + (double)y0;
  double qd = floor(ldexp((double)ca, e) / yd);
  qd = fmin(fmax(qd, 0.0), 0x1p58);
  int64_t q = (int64_t)qd;
  // R = c_a 2^e - q Y
  uint64_t R[4] = {0, 0, 0, 0};
  {
    const int L = e >> 6, b = e & 63;
    const uint64_t lo = (uint64_t)ca << b;
    const uint64_t hi = b ? ((uint64_t)ca >> (64 - b)) : 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) R[i] = (i == L) ? lo : (i == L + 1) ? hi : 0;
  }
  s256_sub_mul(R, q, y0, y1, y2);
  const int64_t dq = (int64_t)rint(s256_to_f64(R) / yd);
  q += dq;
  s256_sub_mul(R, dq, y0, y1, y2);
  if ((int64_t)R[3] < 0) q -= 1;
  const uint64_t uq = (uint64_t)q;
  int rho;
  uint64_t m;
  if (uq >> 56) {
    rho = r0;
    m = uq >> 1;
  } else {
    rho = r0 - 1;
    m = uq;
  }
  sw = scale_pack(m, rho);
  bsw = bscale_pack(m, rho);
}

__device__ __forceinline__ void write_scale(uint32_t g, u128 t, const uint32_t* __restrict__ c, uint64_t C,
                                            uint32_t P, uint64_t* __restrict__ scale, uint64_t* __restrict__ bscale) {
  const uint32_t ca = c[g / P];
  uint64_t sw = 0, bsw = 0;
  if (t != 0 && ca != 0) scale_words(t, ca, C, sw, bsw);
  scale[g] = sw;
  bscale[g] = bsw;
}

__global__ void k_scale(const uint64_t* __restrict__ T, const uint32_t* __restrict__ c,
                        const uint64_t* __restrict__ Csum, uint32_t A, uint32_t P,
                        uint64_t* __restrict__ scale, uint64_t* __restrict__ bscale) {
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= A * P) return;
  write_scale(g, make_u128(T[2 * g], T[2 * g + 1]), c, *Csum, P, scale, bscale);
}

// T[g] = sum over blocks of partial[b][g] + ext[g] * 2^ext_shift, and the
// scale words of g (Eq. (3)) from it; with pcount, n[g] = sum over blocks of
// pcount[b][g].  Block = 64 consecutive g x 16 strides over the partial rows.
template <typename PT>
__global__ __launch_bounds__(1024) void k_pass_a_reduce(const PT* __restrict__ partial, uint32_t nb, uint32_t G,
                                                        unsigned long long* __restrict__ ext, int ext_shift,
                                                        uint64_t* __restrict__ T, const uint32_t* __restrict__ c,
                                                        const uint64_t* __restrict__ Csum, uint32_t P,
                                                        uint64_t* __restrict__ scale, uint64_t* __restrict__ bscale,
                                                        const uint32_t* __restrict__ pcount,
                                                        uint64_t* __restrict__ cnt) {
  __shared__ uint64_t s_lo[16][64], s_hi[16][64], s_n[16][64];
  const uint32_t gl = threadIdx.x & 63, r = threadIdx.x >> 6;
  const uint32_t g = blockIdx.x * 64 + gl;
  u128 acc = 0;
  uint64_t na = 0;
  if (g < G) {
#pragma unroll 8
    for (uint32_t b = r; b < nb; b += 16) acc += (uint64_t)partial[(size_t)b * G + g];
    if (pcount)
#pragma unroll 8
      for (uint32_t b = r; b < nb; b += 16) na += pcount[(size_t)b * G + g];
  }
  s_lo[r][gl] = (uint64_t)acc;
  s_hi[r][gl] = (uint64_t)(acc >> 64);
  s_n[r][gl] = na;
  __syncthreads();
  if (r == 0 && g < G) {
    u128 t = (u128)ext[g] << ext_shift;
    ext[g] = 0;  // left clear for the next pass A (the only reader of ext is this kernel)
    uint64_t nt = 0;
    for (int i = 0; i < 16; ++i) {
      t += make_u128(s_lo[i][gl], s_hi[i][gl]);
      nt += s_n[i][gl];
    }
    T[2 * g] = (uint64_t)t;
    T[2 * g + 1] = (uint64_t)(t >> 64);
    if (pcount) cnt[g] = nt;
    write_scale(g, t, c, *Csum, P, scale, bscale);  // Eq. (3) scale of this (app, phase)
  }
}

// ---------------------------------------------------------------------------
// Global key dictionary: open addressing over 64-bit slots holding key + 1
// (0 = free).  A key's slot index never changes once claimed.
__device__ __forceinline__ int64_t dict_slot(unsigned long long* __restrict__ dict, uint32_t mask, uint32_t key,
                                             uint32_t* __restrict__ err) {
  const unsigned long long tag = (unsigned long long)key + 1ull;
  uint32_t h = hash32(key) & mask;
  for (uint32_t probe = 0; probe <= mask; ++probe) {
    unsigned long long cur = __hip_atomic_load(&dict[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (cur == tag) return h;
    if (cur == 0) {
      cur = atomicCAS(&dict[h], 0ull, tag);
      if (cur == 0 || cur == tag) return h;
    }
    h = (h + 1) & mask;
  }
  atomicOr(err, ATREX_ERRBIT_CAPACITY);
  return -1;
}

template <bool RAW>
__device__ __forceinline__ void global_accumulate(const GroupTables& gt, uint32_t P, uint32_t key, uint32_t ph,
                                                  uint64_t d, u128 v, uint32_t* err) {
  const int64_t j = dict_slot(gt.dict, gt.dict_mask, key, err);
  if (j < 0) return;
  const size_t gi = (size_t)j * P + ph;
  acc_add(&gt.acc[2 * gi], &gt.acc[2 * gi + 1], v);
  if (RAW) acc_add_plain(&gt.raw[2 * gi], &gt.raw[2 * gi + 1], (u128)d);
}

// Pass B through the global dictionary and global atomics only.  NO_APP:
// the events carry no application (every event is application 0).
template <int BLOCK, bool RAW, bool NO_APP = false>
__global__ __launch_bounds__(BLOCK) void k_pass_b_global(EventsDev ev, uint32_t A, uint32_t P,
                                                         const uint64_t* __restrict__ scale, GroupTables gt,
                                                         uint32_t* __restrict__ err) {
  const uint64_t n = ev.n;
  bool bad = false;
  for (uint64_t i = (uint64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (uint64_t)gridDim.x * BLOCK) {
    const uint32_t k = ev.key[i], a = app_at<NO_APP>(ev.app, i), ph = ev.phase[i];
    const int64_t d = ev.dur[i];
    const bool ok = a < A && ph < P && d >= 0;
    bad |= !ok;
    if (!ok) continue;
    const u128 v = event_share((uint64_t)d, scale[(size_t)a * P + ph]);
    global_accumulate<RAW>(gt, P, k, ph, (uint64_t)d, v, err);
  }
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
}

// ---------------------------------------------------------------------------
// Pass B with a per-workgroup LDS hash table (the low/medium-cardinality
// engine).  LDS holds S slots in buckets of four (S sized to the LDS budget,
// not a power of two): a key tag and, per phase, a two-word accumulator.  A
// key's home bucket is one of the first S / 4 - 1 buckets; its window is the
// home bucket and the next one.  Per event the window's eight tags are read
// with two 16-byte LDS loads and matched without branches.  A key outside its
// window is looked up by probing on from the home bucket and inserted into the
// first free slot (at most MAXPROBE buckets); an event whose key finds no slot
// (or the reserved tag value) is appended to a spill list and handled after
// the kernel, so that no wave waits on device-wide atomics.  Before the LDS atomics, lanes of a wave that hit the
// same (slot, phase) as the wave's first active lane are summed with shuffles
// and added once (hot keys).  At the end each workgroup writes its table into
// 256 owner regions (owner = top byte of the key hash); k_owner_finish sums
// each owner's regions.
constexpr uint32_t MAXPROBE = 8;  // buckets
constexpr uint32_t INVALID_GI = 0xFFFFFFFFu;


struct SpillList {
  uint32_t* key;             // spilled events as records: workgroup w owns [w * cap, (w + 1) * cap)
  uint64_t* val;             // (share lo, share hi | phase << 40)
  uint64_t* raw;             // durations (RAW)
  uint32_t* count;           // [nwg] records written by each workgroup
  uint32_t cap;
};

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63; }

// Wave-aggregated append of this lane's event as a record when `spill` is
// set, to this workgroup's region of the spill list (counter in LDS).  A
// region that fills up raises ATREX_ERRBIT_SPILL (the caller then runs the
// partition engine on all events instead).
__device__ __forceinline__ void spill_append(const SpillList& sp, uint32_t* s_count, bool spill, uint32_t key,
                                             u128 v, uint32_t ph, uint64_t d, uint32_t* err) {
  const uint64_t bm = __ballot(spill);
  if (bm == 0) return;
  const uint32_t leader = __ffsll((unsigned long long)bm) - 1;
  uint32_t base = 0;
  if (lane_id() == leader) base = atomicAdd(s_count, (uint32_t)__popcll(bm));
  base = __shfl(base, leader, 64);
  if (!spill) return;
  const uint32_t r = base + __popcll(bm & ((1ull << lane_id()) - 1ull));
  if (r >= sp.cap) {
    atomicOr(err, ATREX_ERRBIT_SPILL);
    return;
  }
  const size_t i = (size_t)blockIdx.x * sp.cap + r;
  sp.key[i] = key;
  sp.val[2 * i] = (uint64_t)v;
  sp.val[2 * i + 1] = (uint64_t)(v >> 64) | ((uint64_t)ph << 40);
  if (sp.raw) sp.raw[i] = d;
}

// Wave-aggregated append of one row per lane with `want` set.
__device__ __forceinline__ void row_push(const Rows& R, bool want, uint64_t rk, uint64_t lo, uint64_t hi,
                                         uint64_t rlo, uint64_t rhi, uint32_t* err) {
  const uint64_t bm = __ballot(want);
  if (bm == 0) return;
  const uint32_t leader = __ffsll((unsigned long long)bm) - 1;
  unsigned long long base = 0;
  if (lane_id() == leader) base = atomicAdd(R.count, (unsigned long long)__popcll(bm));
  base = __shfl(base, leader, 64);
  if (!want) return;
  const uint64_t pos = base + __popcll(bm & ((1ull << lane_id()) - 1ull));
  if (pos >= R.cap) {
    atomicOr(err, ATREX_ERRBIT_CAPACITY);
    return;
  }
  R.rk[pos] = rk;
  R.lo[pos] = lo;
  R.hi[pos] = hi;
  if (R.rlo) {
    R.rlo[pos] = rlo;
    R.rhi[pos] = rhi;
  }
}

// Events of one group of four per lane, once their scale words have been
// requested: everything the accumulation step needs.
struct StagedEv4 {
  uint32_t key[4], gi[4];  // keys, LDS entries found in the windows (or INVALID_GI)
  uint32_t ph4;        // the four phases, one byte each
  int64_t dur[4];
  uint64_t sw[4];      // pass-B scale words
};

// seed (nullable): a tag table image of S slots that every workgroup starts
// from (the workload's hottest keys, each inside its window); the table is
// then closed: an event whose key is not in its window is spilled at once.
template <int BLOCK, bool RAW, bool NO_APP = false, bool SEEDED = false>
__global__ __launch_bounds__(BLOCK) void k_pass_b_lds(EventsDev ev, uint32_t P, const uint64_t* __restrict__ scale,
                                                      const uint64_t* __restrict__ bscale, uint32_t S,
                                                      OwnerRegions orr, SpillList sp, Rows rows,
                                                      const uint32_t* __restrict__ seed, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  const uint32_t SP = S * P;
  // low and high words of the [S * P] accumulators as two arrays (8-byte
  // stride: twice the LDS banks of interleaved pairs for the random 64-bit
  // atomics), each followed by 64 per-lane dummy entries that take the atomics
  // of lanes with nothing to add (never read); RAW: the same again
  const uint32_t NE = SP + 64;
  unsigned long long* s_lo = smem;
  unsigned long long* s_hi = smem + NE;
  unsigned long long* s_rlo = smem + 2 * NE;  // RAW only
  unsigned long long* s_rhi = smem + 3 * NE;
  uint32_t* s_tag = (uint32_t*)(smem + (RAW ? 4 : 2) * NE);
  uint32_t* s_ocnt = s_tag + S;                 // [ATREX_OWNERS]
  uint32_t& s_spills = s_ocnt[ATREX_OWNERS];    // dynamic LDS: static LDS would not fit beside 160 KB
  uint32_t& s_next = s_ocnt[ATREX_OWNERS + 1];  // next unclaimed block of this workgroup's range
  // Pass A has validated every event (app < A, phase < P, dur >= 0) and the
  // call fails on a range error, so the loop below takes the fields as valid;
  // after a range error this kernel only publishes empty regions.
  const bool range_error = (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) &
                            ATREX_ERRBIT_RANGE) != 0;
  if (range_error) {
    for (uint32_t o = threadIdx.x; o < ATREX_OWNERS; o += BLOCK) orr.count[(size_t)blockIdx.x * ATREX_OWNERS + o] = 0;
    if (threadIdx.x == 0) sp.count[blockIdx.x] = 0;
    return;
  }
  const uint64_t n = ev.n, n4 = n / 4;
  // blocks of 64 groups of four events (one group per lane): this
  // workgroup's contiguous share [blk_lo, blk_hi)
  const uint32_t NBLK = (uint32_t)((n4 + 63) / 64), FULLBLK = (uint32_t)(n4 / 64);
  const uint32_t blk_lo = (uint32_t)((uint64_t)blockIdx.x * NBLK / gridDim.x);
  const uint32_t blk_hi = (uint32_t)((uint64_t)(blockIdx.x + 1) * NBLK / gridDim.x);
  if (threadIdx.x == 0) {
    s_spills = 0;
    s_next = blk_lo;
  }
  for (uint32_t i = threadIdx.x; i < SP; i += BLOCK) {
    s_lo[i] = 0;
    s_hi[i] = 0;
    if (RAW) { s_rlo[i] = 0; s_rhi[i] = 0; }
  }
  const uint32_t dummy = SP + (threadIdx.x & 63);  // this lane's dummy entry
  for (uint32_t i = threadIdx.x; i < S; i += BLOCK) s_tag[i] = SEEDED ? seed[i] : ATREX_EMPTY_KEY;
  for (uint32_t i = threadIdx.x; i < ATREX_OWNERS; i += BLOCK) s_ocnt[i] = 0;
  __syncthreads();
  const uint32_t lane = lane_id();
  const uint32_t NB = S / 4;         // buckets; S is a multiple of 4, S >= 8
  const uint32_t NH8 = (NB - 1) << 8;  // home bucket = floor((hash >> 8) * (NB - 1) / 2^24), NB < 2^16
  auto bucket_tags = [&](uint32_t b) -> uint4 { return *(const uint4*)&s_tag[4 * b]; };
  // Slot of key k from its home bucket b (tags tv already read): the key's
  // slot in this or a following bucket, else the first free slot claimed for
  // it; INVALID_GI when not placed within MAXPROBE buckets.  Two lanes may
  // claim two slots for one key in a race; both then accumulate and the owner
  // merge adds them up.  The rare path: a plain loop, at most 4 retries per
  // bucket (each failed claim fills a slot).
  auto find_slot = [&](uint32_t k, uint32_t b, uint4 tv) -> uint32_t {
    uint32_t probe = 0;
#pragma unroll 1
    for (uint32_t step = 0; step < 8 * MAXPROBE; ++step) {
      if (tv.x == k) return 4 * b;
      if (tv.y == k) return 4 * b + 1;
      if (tv.z == k) return 4 * b + 2;
      if (tv.w == k) return 4 * b + 3;
      const uint32_t e = tv.x == ATREX_EMPTY_KEY ? 0u : tv.y == ATREX_EMPTY_KEY ? 1u
                       : tv.z == ATREX_EMPTY_KEY ? 2u : tv.w == ATREX_EMPTY_KEY ? 3u : 4u;
      if (e < 4) {
        const uint32_t t = atomicCAS(&s_tag[4 * b + e], ATREX_EMPTY_KEY, k);
        if (t == ATREX_EMPTY_KEY || t == k) return 4 * b + e;
      } else {
        if (++probe == MAXPROBE) return INVALID_GI;
        b = (b + 1 == NB) ? 0 : b + 1;
      }
      tv = bucket_tags(b);
    }
    return INVALID_GI;
  };
  // stage(): request the scale words of a loaded group and find its events'
  // slots in their windows (a chain of selects over the eight tags, last slot
  // first, gives the first slot holding the key).  The host takes this engine
  // only when A * P < 2^24, so the scale word index is one 24-bit multiply-add.
  auto home_bucket = [&](uint32_t k) -> uint32_t {
    return (uint32_t)(((uint64_t)(hash_mul(k) >> 8) * (NH8 & 0xFFFFFFu)) >> 32);  // = lds_home_bucket(k, NB)
  };
  auto stage = [&](const Ev4& e, StagedEv4& g) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      g.sw[j] = bscale[__umul24(e.app[j], P) + e.ph(j)];
      g.key[j] = e.key[j];
      g.dur[j] = e.dur[j];
    }
    g.ph4 = e.ph4;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t k = e.key[j], b = home_bucket(k);
      const uint4 t0 = bucket_tags(b), t1 = bucket_tags(b + 1);
      uint32_t w = INVALID_GI;
      w = t1.w == k ? 7u : w;
      w = t1.z == k ? 6u : w;
      w = t1.y == k ? 5u : w;
      w = t1.x == k ? 4u : w;
      w = t0.w == k ? 3u : w;
      w = t0.z == k ? 2u : w;
      w = t0.y == k ? 1u : w;
      w = t0.x == k ? 0u : w;
      const bool hit = w != INVALID_GI && k != ATREX_EMPTY_KEY;
      g.gi[j] = hit ? __umul24(4 * b + w, P) + e.ph(j) : INVALID_GI;
    }
  };
  // The waves of the workgroup claim the blocks of its share one at a time
  // from a counter in LDS, so that waves the SIMD favours take more blocks and
  // all finish together (with a fixed split the last ones would run with ever
  // fewer waves beside them).
  constexpr uint32_t END = ~0u, TAIL = ~0u - 1;  // TAIL: the n % 4 tail events (one per lane, first wave)
  auto next_blk = [&]() -> uint32_t {
    uint32_t bk = 0;
    if (lane == 0) bk = atomicAdd(&s_next, 1u);
    bk = __builtin_amdgcn_readfirstlane(bk);
    return bk < blk_hi ? bk : END;
  };
  // events of this lane's group that exist, and the index of its event 0:
  // wanted only on the rare paths
  auto nvalid_of = [&](uint32_t bk) -> uint32_t {
    if (bk == TAIL) return n4 * 4 + lane < n ? 1u : 0u;
    return (bk < FULLBLK || 64 * (uint64_t)bk + lane < n4) ? 4u : 0u;
  };
  auto first_of = [&](uint32_t bk) -> uint64_t {
    return bk == TAIL ? n4 * 4 + lane : (64 * (uint64_t)bk + lane) * 4;
  };
  // process(): shares, slots, accumulation of a staged group.  Events past
  // the end carry the reserved key, so they miss the window.
  auto process = [&](const StagedEv4& g, uint32_t bk) {
    uint32_t ph[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) ph[j] = (g.ph4 >> (8 * j)) & 0xFFu;
    uint64_t vlo[4], vhi[4];
    uint32_t slow = 0, wide = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      slow |= (uint32_t)(g.sw[j] >> 32);
      wide |= (uint32_t)((uint64_t)g.dur[j] >> 32);
    }
    if (__builtin_expect(__any((slow >> 31) != 0), 0)) {  // rho outside [-8, 63]: the general scale word
      const uint32_t nvalid = nvalid_of(bk);
      const uint64_t first = first_of(bk);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool valid = (uint32_t)j < nvalid;
        const uint64_t i = valid ? first + j : 0;
        const u128 v = event_share((uint64_t)g.dur[j], valid ? scale[app_at<NO_APP>(ev.app, i) * P + ph[j]] : 0);
        vlo[j] = (uint64_t)v;
        vhi[j] = (uint64_t)(v >> 64);
      }
    } else if (__builtin_expect(__any(wide != 0), 0)) {  // a duration of 2^32 ns or more
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bscale_share64((uint64_t)g.dur[j], (uint32_t)g.sw[j], (uint32_t)(g.sw[j] >> 32), vlo[j], vhi[j]);
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint32_t hi32;
        bscale_share32((uint32_t)g.dur[j], (uint32_t)g.sw[j], (uint32_t)(g.sw[j] >> 32), vlo[j], hi32);
        vhi[j] = hi32;
      }
    }
    uint32_t gi[4];
    bool miss = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      gi[j] = g.gi[j];
      miss |= gi[j] == INVALID_GI;
    }
    if (__builtin_expect(__any(miss), 0)) {
      // first occurrence of a key, a key placed past its window, the reserved
      // key, or events past the end: probe on (not in a seeded table), then
      // spill what is unplaced
      const uint32_t nvalid = nvalid_of(bk);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool valid = (uint32_t)j < nvalid;
        if (!SEEDED && valid && gi[j] == INVALID_GI && g.key[j] != ATREX_EMPTY_KEY) {
          const uint32_t b = home_bucket(g.key[j]);
          const uint32_t sl = find_slot(g.key[j], b, bucket_tags(b));
          if (sl != INVALID_GI) gi[j] = __umul24(sl, P) + ph[j];
        }
        spill_append(sp, &s_spills, valid && gi[j] == INVALID_GI, g.key[j], make_u128(vlo[j], vhi[j]), ph[j],
                     (uint64_t)g.dur[j], err);
      }
    }
    // hot groups: when at least half the lanes share the first lane's (slot,
    // phase) in the first event slot, up to two groups are taken off the
    // atomics: each lane sums its own events of the group, the wave sums the
    // lanes, and one lane adds the total once (a hot key split over two
    // phases would otherwise put half the wave on one LDS address).  A
    // milder skew costs less as LDS atomic conflicts.
    bool hot = false;
    {
      const uint64_t act = __ballot(gi[0] != INVALID_GI);
      if (act) {
        const uint32_t fl = __ffsll((unsigned long long)act) - 1;
        const uint32_t lead = __builtin_amdgcn_readlane(gi[0], fl);
        hot = __popcll(__ballot(gi[0] == lead)) >= 32;
      }
    }
    if (hot) {
#pragma unroll 1
      for (int r = 0; r < 2; ++r) {
        // the group of the first lane's first remaining event (in the first
        // round, the one that made the wave hot)
        const uint32_t first = gi[0] != INVALID_GI ? gi[0]
                             : gi[1] != INVALID_GI ? gi[1]
                             : gi[2] != INVALID_GI ? gi[2] : gi[3];
        const uint64_t act = __ballot(first != INVALID_GI);
        if (act == 0) break;
        const uint32_t lead = __builtin_amdgcn_readlane(first, __ffsll((unsigned long long)act) - 1);
        uint32_t cnt = 0;
        u128 sv = 0, sr = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool m = gi[j] == lead;
          cnt += (uint32_t)__popcll(__ballot(m));
          sv += m ? make_u128(vlo[j], vhi[j]) : (u128)0;
          if (RAW) sr += m ? (u128)(uint64_t)g.dur[j] : (u128)0;
        }
        if (cnt < 32) break;  // wave-uniform
        const u128 tot = wave_total_u98(sv);  // sv < 2^98: four shares of at most 2^96
        u128 rtot = 0;
        if (RAW) rtot = wave_sum_u128(sr);
        if (lane == 0) {
          acc_add_n(&s_lo[lead], &s_hi[lead], tot, cnt);
          if (RAW) acc_add_plain(&s_rlo[lead], &s_rhi[lead], rtot);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (gi[j] == lead) gi[j] = INVALID_GI;
      }
    }
    // accumulate without branches: a lane with nothing to add for an event
    // adds into its own dummy entry.  The four low-word atomics go first (their
    // returned values give the carries), then the high words with the count.
    uint32_t at[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) at[j] = gi[j] != INVALID_GI ? gi[j] : dummy;
    unsigned long long old[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) old[j] = atomicAdd(&s_lo[at[j]], (unsigned long long)vlo[j]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const unsigned long long carry = (old[j] + vlo[j] < old[j]) ? 1ull : 0ull;
      atomicAdd(&s_hi[at[j]], (unsigned long long)vhi[j] + carry + (1ull << ATREX_COUNT_SHIFT));
    }
    if (RAW) {
#pragma unroll
      for (int j = 0; j < 4; ++j) old[j] = atomicAdd(&s_rlo[at[j]], (unsigned long long)g.dur[j]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (old[j] + (uint64_t)g.dur[j] < old[j]) atomicAdd(&s_rhi[at[j]], 1ull);
    }
  };
  // A three-stage pipeline: while one block is accumulated, the scale words
  // of the next and the loads of the one after are in flight.  Full blocks
  // load through the wave's scalar base address; the one partial block clamps
  // its indices and gives the events past the end the reserved key.
  {
    auto load_blk = [&](uint32_t bk, Ev4& e) {
      const uint64_t g0 = 64 * (uint64_t)bk;
      if (bk < FULLBLK) {
        load4_lane<NO_APP>(ev.key, ev.app, ev.phase, ev.dur, g0 * 4, lane, e);
      } else {
        const uint64_t q = g0 + lane;
        load4<true, NO_APP>(ev.key, ev.app, ev.phase, ev.dur, min(q, n4 - 1) * 4, e);
        if (q >= n4) {
#pragma unroll
          for (int j = 0; j < 4; ++j) e.key[j] = ATREX_EMPTY_KEY;
        }
      }
    };
    uint32_t bA = next_blk();
    if (bA != END) {
      Ev4 raw;
      StagedEv4 gA, gB;
      load_blk(bA, raw);
      stage(raw, gA);
      uint32_t bB = next_blk();
      if (bB != END) load_blk(bB, raw);
      for (;;) {  // gA holds block bA, raw block bB (when it exists)
        uint32_t bC = END;
        if (bB != END) {
          stage(raw, gB);
          bC = next_blk();
          if (bC != END) load_blk(bC, raw);
        }
        process(gA, bA);
        if (bB == END) break;
        uint32_t bD = END;
        if (bC != END) {
          stage(raw, gA);
          bD = next_blk();
          if (bD != END) load_blk(bD, raw);
        }
        process(gB, bB);
        if (bC == END) break;
        bA = bC;
        bB = bD;
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < 64) {  // n % 4 tail events, one wave
    const uint64_t i = n4 * 4 + lane;
    Ev4 e;
#pragma unroll
    for (int j = 0; j < 4; ++j) { e.key[j] = ATREX_EMPTY_KEY; e.app[j] = 0; e.dur[j] = 0; }
    e.ph4 = 0;
    if (i < n) {
      e.key[0] = ev.key[i]; e.app[0] = app_at<NO_APP>(ev.app, i); e.ph4 = ev.phase[i]; e.dur[0] = ev.dur[i];
    }
    StagedEv4 g;
    stage(e, g);
    process(g, TAIL);
  }
  __syncthreads();
  // this workgroup's table -> owner regions (owner = top byte of the key hash);
  // a region that is full sends its rows straight to the row list
  for (uint32_t s0 = 0; s0 < S; s0 += BLOCK) {
    const uint32_t sl = s0 + threadIdx.x;
    const uint32_t t = sl < S ? s_tag[sl] : ATREX_EMPTY_KEY;
    bool spill_rows = false;
    if (t != ATREX_EMPTY_KEY) {
      const uint32_t o = hash32(t) >> 24;
      const uint32_t r = atomicAdd(&s_ocnt[o], 1u);
      if (r < orr.capo) {
        const size_t rec = ((size_t)blockIdx.x * ATREX_OWNERS + o) * orr.capo + r;
        orr.key[rec] = t;
        for (uint32_t ph = 0; ph < P; ++ph) {
          orr.acc[(rec * P + ph) * 2] = s_lo[sl * P + ph];
          orr.acc[(rec * P + ph) * 2 + 1] = s_hi[sl * P + ph];
          if (RAW) {
            orr.raw[(rec * P + ph) * 2] = s_rlo[sl * P + ph];
            orr.raw[(rec * P + ph) * 2 + 1] = s_rhi[sl * P + ph];
          }
        }
      } else {
        spill_rows = true;
      }
    }
    for (uint32_t ph = 0; ph < P; ++ph) {
      const size_t gi = (size_t)sl * P + ph;
      const uint64_t hi = spill_rows ? s_hi[gi] : 0;
      const bool want = spill_rows && (hi >> ATREX_COUNT_SHIFT) != 0;
      row_push(rows, want, ((uint64_t)t << 3) | ph, want ? s_lo[gi] : 0, hi,
               (RAW && want) ? s_rlo[gi] : 0, (RAW && want) ? s_rhi[gi] : 0, err);
    }
  }
  __syncthreads();
  for (uint32_t o = threadIdx.x; o < ATREX_OWNERS; o += BLOCK)
    orr.count[(size_t)blockIdx.x * ATREX_OWNERS + o] = min(s_ocnt[o], orr.capo);
  if (threadIdx.x == 0) sp.count[blockIdx.x] = min(s_spills, sp.cap);
}

// ---------------------------------------------------------------------------
// Global-hash engine output: every (dictionary slot, phase) with at least one
// invocation becomes a row.
__global__ void k_compact_rows(GroupTables gt, uint32_t P, Rows rows, uint32_t* __restrict__ err) {
  const uint64_t total = (uint64_t)(gt.dict_mask + 1) * P;
  for (uint64_t base = (uint64_t)blockIdx.x * blockDim.x; base < total; base += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t gi = base + threadIdx.x;
    bool live = false;
    uint64_t rk = 0, lo = 0, hi = 0, rl = 0, rh = 0;
    if (gi < total) {
      const unsigned long long tag = gt.dict[gi / P];
      hi = gt.acc[2 * gi + 1];
      live = tag != 0 && (hi >> ATREX_COUNT_SHIFT) != 0;
      rk = ((uint64_t)(uint32_t)(tag - 1) << 3) | (gi % P);
      lo = gt.acc[2 * gi];
      if (gt.raw) { rl = gt.raw[2 * gi]; rh = gt.raw[2 * gi + 1]; }
    }
    row_push(rows, live, rk, lo, hi, rl, rh, err);
  }
}

// Scale words -> (m, rho) for inspection.
__global__ void k_unpack_scale(const uint64_t* __restrict__ sw, uint64_t G, uint64_t* __restrict__ mant,
                               int32_t* __restrict__ rho) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  const uint64_t w = sw[g];
  if (mant) mant[g] = w ? ((w & (((uint64_t)1 << 55) - 1)) | ((uint64_t)1 << 55)) : 0;
  if (rho) rho[g] = w ? (int32_t)(w >> 56) - 64 : 0;
}

// ---------------------------------------------------------------------------
// Seeding the LDS engine with the hottest keys.  A sample of NS events at a
// fixed stride counts its keys in a global table (open addressing, key + 1,
// 0 = free; each workgroup's share counted in LDS first); the occupied
// entries become sort keys (the inverted count: ascending = hottest first,
// ties in table order); one workgroup then places the hottest 2S keys, 1024
// at a time in that order, into a tag image of S slots, each in the first
// free slot of its window (home bucket and the next, or its own bucket only;
// a key whose window is full is left out), and counts the sampled events the
// placed keys cover.  Which keys are seeded changes only which events spill,
// never a result.
constexpr uint32_t kSeedCountBits = 19, kSeedCountMask = (1u << kSeedCountBits) - 1;

// Each workgroup counts kSeedPerWG sampled events in an LDS table (the lanes
// of a wave sharing the wave's first key add once), then adds each distinct
// key to the global table once, with its count: a key that dominates the
// events costs one global atomic per workgroup instead of one per sample
// (atomics on one address serialise).
constexpr uint32_t kSeedPerWG = 2048, kSeedLdsSlots = 4096;

__global__ __launch_bounds__(1024) void k_seed_count(const uint32_t* __restrict__ key, uint64_t n, uint32_t NS,
                                                     unsigned long long* __restrict__ tab, uint32_t mask,
                                                     uint32_t* __restrict__ cnt) {
  __shared__ uint32_t s_key[kSeedLdsSlots], s_cnt[kSeedLdsSlots];
  const uint32_t tid = threadIdx.x, lane = tid & 63;
  for (uint32_t i = tid; i < kSeedLdsSlots; i += 1024) {
    s_key[i] = ATREX_EMPTY_KEY;
    s_cnt[i] = 0;
  }
  constexpr uint32_t PER = kSeedPerWG / 1024;
  uint32_t kk[PER];
#pragma unroll
  for (uint32_t j = 0; j < PER; ++j) {
    const uint32_t s = blockIdx.x * kSeedPerWG + j * 1024 + tid;
    kk[j] = s < NS ? key[(uint64_t)s * n / NS] : ATREX_EMPTY_KEY;
  }
  __syncthreads();
#pragma unroll
  for (uint32_t j = 0; j < PER; ++j) {
    const uint32_t k = kk[j];
    const bool live = k != ATREX_EMPTY_KEY;  // the reserved tag is never seeded
    const uint64_t act = __ballot(live);
    if (act == 0) continue;  // wave-uniform
    const uint32_t lead = (uint32_t)__ffsll((unsigned long long)act) - 1;
    const uint32_t k0 = __builtin_amdgcn_readlane(k, lead);
    const uint64_t same = __ballot(live && k == k0);
    if (live && (k != k0 || lane == lead)) {
      const uint32_t add = k == k0 ? (uint32_t)__popcll(same) : 1u;
      uint32_t h = hash32(k) & (kSeedLdsSlots - 1);
      for (uint32_t probe = 0; probe < kSeedLdsSlots; ++probe) {  // at most kSeedPerWG of the slots are taken
        const uint32_t prev = atomicCAS(&s_key[h], ATREX_EMPTY_KEY, k);
        if (prev == ATREX_EMPTY_KEY || prev == k) {
          atomicAdd(&s_cnt[h], add);
          break;
        }
        h = (h + 1) & (kSeedLdsSlots - 1);
      }
    }
  }
  __syncthreads();
  for (uint32_t i = tid; i < kSeedLdsSlots; i += 1024) {
    const uint32_t k = s_key[i];
    if (k == ATREX_EMPTY_KEY) continue;
    uint32_t h = hash32(k) & mask;
    for (uint32_t probe = 0; probe <= mask; ++probe) {  // the table has at least twice NS slots
      const unsigned long long prev = atomicCAS(&tab[h], 0ull, (unsigned long long)k + 1);
      if (prev == 0 || prev == (unsigned long long)k + 1) {
        atomicAdd(&cnt[h], s_cnt[i]);
        break;
      }
      h = (h + 1) & mask;
    }
  }
}

__global__ void k_seed_list(const unsigned long long* __restrict__ tab, const uint32_t* __restrict__ cnt,
                            uint32_t cap, uint64_t* __restrict__ list, uint32_t* __restrict__ idx) {
  const uint32_t h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= cap) return;
  // (key << 32 | 2^19 - 1 - count): the sort takes the low 19 bits only
  // (counts are at most NS <= 2^18; free slots, with count 0, sort last)
  list[h] = tab[h] ? ((uint64_t)(uint32_t)(tab[h] - 1) << 32) | (kSeedCountMask - cnt[h]) : kSeedCountMask;
  idx[h] = h;
}

// window 2: a key may sit in its home bucket or the next (lds_home_bucket,
// the LDS engine's lookup); window 1: in its own bucket only (lds_only_bucket).
__global__ __launch_bounds__(1024) void k_seed_build(const uint64_t* __restrict__ list, uint32_t L, uint32_t S,
                                                     uint32_t window, uint32_t* __restrict__ seed,
                                                     unsigned long long* __restrict__ covered) {
  extern __shared__ uint32_t s_img[];  // [S]
  __shared__ unsigned long long s_cov;
  for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) s_img[i] = ATREX_EMPTY_KEY;
  if (threadIdx.x == 0) s_cov = 0;
  __syncthreads();
  // candidates in chunks of 1024, hottest chunk first; within a chunk each
  // thread claims the first free slot of its key's window
  const uint32_t NB = S / 4;
  for (uint32_t c0 = 0; c0 < L; c0 += 1024) {
    const uint32_t c = c0 + threadIdx.x;
    const uint64_t e = c < L ? list[c] : kSeedCountMask;
    const uint32_t count = kSeedCountMask - (uint32_t)(e & kSeedCountMask);
    if (count) {
      const uint32_t k = (uint32_t)(e >> 32);
      const uint32_t b = window == 2 ? lds_home_bucket(k, NB) : lds_only_bucket(k, NB);
      for (uint32_t t = 4 * b; t < 4 * b + 4 * window; ++t) {
        if (atomicCAS(&s_img[t], ATREX_EMPTY_KEY, k) == ATREX_EMPTY_KEY) {
          atomicAdd(&s_cov, (unsigned long long)count);
          break;
        }
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *covered = s_cov;
  for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) seed[i] = s_img[i];
}

// ---------------------------------------------------------------------------
// Incremental refresh (an append-only event log): the per-(app, phase) totals
// of the events folded so far (run) plus those of the new events (T, n, as
// pass A left them) become the totals of the whole log, in T and n.  Skipped
// after a range error in the new events, so that a failed refresh leaves
// every total as it was.
__global__ void k_fold_totals(uint64_t* __restrict__ T, uint64_t* __restrict__ cnt,
                              const uint64_t* __restrict__ T_run, const uint64_t* __restrict__ n_run, uint64_t G,
                              const uint32_t* __restrict__ err) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G || (__hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & ATREX_ERRBIT_RANGE)) return;
  const u128 t = make_u128(T[2 * g], T[2 * g + 1]) + make_u128(T_run[2 * g], T_run[2 * g + 1]);
  T[2 * g] = (uint64_t)t;
  T[2 * g + 1] = (uint64_t)(t >> 64);
  cnt[g] += n_run[g];
}

__global__ void k_copy_u64(uint64_t* __restrict__ dst, const uint64_t* __restrict__ src, uint64_t n) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

}  // namespace

// ---------------------------------------------------------------------------
// Host launchers
void launch_seed(hipStream_t s, const uint32_t* key, uint64_t n, uint32_t NS, uint64_t* tab, uint32_t tab_cap,
                 uint32_t* cnt, uint64_t* list, uint32_t* idx, uint64_t* list2, uint32_t* idx2, void* sort_tmp,
                 uint32_t S, uint32_t* seed, unsigned long long* covered) {
  launch_fill_u64(s, tab, tab_cap, 0);
  launch_fill_u32(s, cnt, tab_cap, 0);
  hipLaunchKernelGGL(k_seed_count, dim3((NS + kSeedPerWG - 1) / kSeedPerWG), dim3(1024), 0, s, key, n, NS,
                     (unsigned long long*)tab, tab_cap - 1, cnt);
  hipLaunchKernelGGL(k_seed_list, dim3((tab_cap + 255) / 256), dim3(256), 0, s, (const unsigned long long*)tab, cnt,
                     tab_cap, list, idx);
  radix_sort_pairs(s, list, idx, list2, idx2, tab_cap, kSeedCountBits, sort_tmp);  // hottest first, free last
  launch_seed_image(s, list, tab_cap, S, 2, seed, covered);
}

void launch_seed_image(hipStream_t s, const uint64_t* list, uint32_t tab_cap, uint32_t S, uint32_t window,
                       uint32_t* seed, unsigned long long* covered) {
  // candidates: the hottest 2S keys (colder ones rarely find a free slot in their window)
  hipLaunchKernelGGL(k_seed_build, dim3(1), dim3(1024), (size_t)S * 4, s, list, std::min<uint32_t>(tab_cap, 2 * S), S,
                     window, seed, covered);
}

void launch_fold_totals(hipStream_t s, uint64_t* T, uint64_t* cnt, const uint64_t* T_run, const uint64_t* n_run,
                        uint64_t G, const uint32_t* err) {
  if (G) hipLaunchKernelGGL(k_fold_totals, dim3((uint32_t)((G + 255) / 256)), dim3(256), 0, s, T, cnt, T_run, n_run, G, err);
}

void launch_copy_u64(hipStream_t s, uint64_t* dst, const uint64_t* src, uint64_t n) {
  if (!n) return;
  const uint64_t nb = std::min<uint64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_copy_u64, dim3((uint32_t)nb), dim3(256), 0, s, dst, src, n);
}

void launch_unpack_scale(hipStream_t s, const uint64_t* sw, uint64_t G, uint64_t* mant, int32_t* rho) {
  if (G) hipLaunchKernelGGL(k_unpack_scale, dim3((uint32_t)((G + 255) / 256)), dim3(256), 0, s, sw, G, mant, rho);
}

void launch_pass_a_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                       unsigned long long* partial, unsigned long long* carry, uint32_t* pcount, uint32_t* err) {
  const uint32_t G = A * P;
  if (pcount)
    hipLaunchKernelGGL((k_pass_a_lds<1024, true>), dim3(nblocks), dim3(1024), (size_t)G * 12, s, ev, A, P, G, partial,
                       carry, pcount, err);
  else
    hipLaunchKernelGGL((k_pass_a_lds<1024, false>), dim3(nblocks), dim3(1024), (size_t)G * 8, s, ev, A, P, G, partial,
                       carry, pcount, err);
}

void launch_pass_a_reduce(hipStream_t s, const unsigned long long* partial, uint32_t nb, uint32_t G,
                          unsigned long long* carry, uint64_t* T, const uint32_t* c, const uint64_t* Csum,
                          uint32_t P, uint64_t* scale, void* bscale, const uint32_t* pcount, uint64_t* cnt) {
  hipLaunchKernelGGL(k_pass_a_reduce<unsigned long long>, dim3((G + 63) / 64), dim3(1024), 0, s, partial, nb, G, carry,
                     64, T, c, Csum, P, scale, (uint64_t*)bscale, pcount, cnt);
}

void launch_pass_a_lds32(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                         uint32_t* partial, unsigned long long* ext, uint32_t* pcount, uint32_t* err) {
  const uint32_t G = A * P;
  if (pcount)
    hipLaunchKernelGGL((k_pass_a_lds32<1024, true>), dim3(nblocks), dim3(1024), (size_t)G * 8, s, ev, A, P, G,
                       partial, ext, pcount, err);
  else
    hipLaunchKernelGGL((k_pass_a_lds32<1024, false>), dim3(nblocks), dim3(1024), (size_t)G * 4, s, ev, A, P, G,
                       partial, ext, pcount, err);
}

void launch_pass_a_reduce32(hipStream_t s, const uint32_t* partial, uint32_t nb, uint32_t G,
                            unsigned long long* ext, uint64_t* T, const uint32_t* c, const uint64_t* Csum,
                            uint32_t P, uint64_t* scale, void* bscale, const uint32_t* pcount, uint64_t* cnt) {
  hipLaunchKernelGGL(k_pass_a_reduce<uint32_t>, dim3((G + 63) / 64), dim3(1024), 0, s, partial, nb, G, ext, 32, T, c,
                     Csum, P, scale, (uint64_t*)bscale, pcount, cnt);
}

void launch_pass_a_range(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t GR, uint32_t R,
                         uint32_t slices, uint32_t* partial, unsigned long long* ext, uint32_t* pcount,
                         const HistJob* hj, uint32_t* err) {
  const uint32_t G = A * P;
  const uint32_t nblocks = ((slices + 7) / 8) * 8 * R;
  const size_t tables = ((((size_t)(pcount ? 2 * GR : GR) + 64 + 3) & ~(size_t)3)) * 4;
  const HistJob none{};
#define ATREX_RANGE(C, H)                                                                                    \
  hipLaunchKernelGGL((k_pass_a_range<1024, C, H>), dim3(std::max(nblocks, H ? hj->nwg : 0u)), dim3(1024),  \
                     tables + (H ? pass_a_hist_bytes(*hj) : 0), s, ev, A, P, G, GR, R, slices, partial, ext,  \
                     pcount, H ? *hj : none, err)
  if (hj) {
    if (pcount) ATREX_RANGE(true, true); else ATREX_RANGE(false, true);
  } else {
    if (pcount) ATREX_RANGE(true, false); else ATREX_RANGE(false, false);
  }
#undef ATREX_RANGE
}

size_t pass_a_hist_bytes(const HistJob& hj) { return ((size_t)4 << hj.BB) + (size_t)4 * hj.S; }

void launch_pass_a_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                          unsigned long long* T, unsigned long long* cnt, uint32_t* err) {
  if (cnt)
    hipLaunchKernelGGL((k_pass_a_global<256, true>), dim3(nblocks), dim3(256), 0, s, ev, A, P, T, cnt, err);
  else
    hipLaunchKernelGGL((k_pass_a_global<256, false>), dim3(nblocks), dim3(256), 0, s, ev, A, P, T, cnt, err);
}

void launch_scale(hipStream_t s, const uint64_t* T, const uint32_t* c, const uint64_t* Csum, uint32_t A,
                  uint32_t P, uint64_t* scale, void* bscale) {
  const uint32_t G = A * P;
  hipLaunchKernelGGL(k_scale, dim3((G + 255) / 256), dim3(256), 0, s, T, c, Csum, A, P, scale, (uint64_t*)bscale);
}

void launch_pass_b_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                          const GroupTables& gt, bool raw, uint32_t nblocks, uint32_t* err) {
  if (!ev.app)  // events without applications (the host takes no raw time then)
    hipLaunchKernelGGL((k_pass_b_global<256, false, true>), dim3(nblocks), dim3(256), 0, s, ev, A, P, scale, gt, err);
  else if (raw)
    hipLaunchKernelGGL((k_pass_b_global<256, true>), dim3(nblocks), dim3(256), 0, s, ev, A, P, scale, gt, err);
  else
    hipLaunchKernelGGL((k_pass_b_global<256, false>), dim3(nblocks), dim3(256), 0, s, ev, A, P, scale, gt, err);
}

uint32_t pass_b_lds_slots(uint32_t P, bool raw, size_t lds_bytes) {
  const size_t per_slot = 4 + (size_t)16 * P * (raw ? 2 : 1);
  const size_t fixed = ATREX_OWNERS * 4 + 256 + (size_t)64 * 16 * (raw ? 2 : 1);
  size_t S = (lds_bytes - fixed) / per_slot;
  if (S > 8 * 1024) S = 8 * 1024;  // the bucket hash needs S / 4 < 2^16
  return (uint32_t)(S & ~(size_t)3);  // whole buckets of four
}

size_t pass_b_lds_smem(uint32_t P, bool raw, uint32_t S) {
  return ((size_t)S * P * 16 + 64 * 16) * (raw ? 2 : 1) + (size_t)S * 4 + ATREX_OWNERS * 4 + 8;
}

// a workgroup sees about n / nwg events (its share of the 64-group blocks,
// and the tail); its spill region holds five eighths of that (a table seeded
// with the hottest keys is taken when they cover at least half of a sample)
uint32_t spill_cap(uint64_t n, uint32_t nwg) { return (uint32_t)((n + nwg - 1) / nwg * 5 / 8 + 8 * 1024); }

uint32_t owner_cap(uint32_t S) { return 2 * ((S + ATREX_OWNERS - 1) / ATREX_OWNERS) + 32; }

void launch_pass_b_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                       const void* bscale_v, bool raw, uint32_t S, uint32_t nblocks, const OwnerRegions& orr, uint32_t* spill_key,
                       uint64_t* spill_val, uint64_t* spill_raw, uint32_t* spill_count, uint32_t scap,
                       const Rows& rows, const uint32_t* seed, uint32_t* err) {
  const size_t smem = pass_b_lds_smem(P, raw, S);
  SpillList sp{spill_key, spill_val, spill_raw, spill_count, scap};
  const uint64_t* bscale = (const uint64_t*)bscale_v;
  (void)A;
  if (!ev.app)  // events without applications (the host takes no raw time then, nor seeds)
    hipLaunchKernelGGL((k_pass_b_lds<1024, false, true>), dim3(nblocks), dim3(1024), smem, s, ev, P, scale, bscale, S,
                       orr, sp, rows, seed, err);
  else if (seed && raw)
    hipLaunchKernelGGL((k_pass_b_lds<1024, true, false, true>), dim3(nblocks), dim3(1024), smem, s, ev, P, scale,
                       bscale, S, orr, sp, rows, seed, err);
  else if (seed)
    hipLaunchKernelGGL((k_pass_b_lds<1024, false, false, true>), dim3(nblocks), dim3(1024), smem, s, ev, P, scale,
                       bscale, S, orr, sp, rows, seed, err);
  else if (raw)
    hipLaunchKernelGGL((k_pass_b_lds<1024, true>), dim3(nblocks), dim3(1024), smem, s, ev, P, scale, bscale, S, orr,
                       sp, rows, seed, err);
  else
    hipLaunchKernelGGL((k_pass_b_lds<1024, false>), dim3(nblocks), dim3(1024), smem, s, ev, P, scale, bscale, S, orr,
                       sp, rows, seed, err);
}

void launch_compact_rows(hipStream_t s, const GroupTables& gt, uint32_t P, const Rows& rows, uint32_t* err) {
  const uint64_t total = (uint64_t)(gt.dict_mask + 1) * P;
  uint64_t nb = (total + 255) / 256;
  if (nb > 4096) nb = 4096;
  hipLaunchKernelGGL(k_compact_rows, dim3((uint32_t)nb), dim3(256), 0, s, gt, P, rows, err);
}

hipError_t set_kernel_smem_limits() {
  const void* pass_a[] = {(const void*)k_pass_a_lds<1024, false>,   (const void*)k_pass_a_lds<1024, true>,
                          (const void*)k_pass_a_lds32<1024, false>, (const void*)k_pass_a_lds32<1024, true>,
                          (const void*)k_pass_a_range<1024, false, false>, (const void*)k_pass_a_range<1024, true, false>,
                          (const void*)k_pass_a_range<1024, false, true>, (const void*)k_pass_a_range<1024, true, true>};
  hipError_t e = hipSuccess;
  for (const void* f : pass_a) {
    e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
  }
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, false, true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, true, false, true>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, false, false, true>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e != hipSuccess) return e;
  e = set_score_smem_limits();
  if (e != hipSuccess) return e;
  e = set_share_smem_limits();
  if (e != hipSuccess) return e;
  e = set_stats_smem_limits();
  if (e != hipSuccess) return e;
  e = set_units_smem_limits();
  if (e != hipSuccess) return e;
  e = set_normalize_smem_limits();
  if (e != hipSuccess) return e;
  e = set_join_smem_limits();
  if (e != hipSuccess) return e;
  return set_rows_smem_limits();
}
