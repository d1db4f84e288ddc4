// kernels_small.hip -- single-workgroup versions of the ordering, per-phase
// normalisation (§3.4) and score (§3.6, Eq. (4)-(6)) steps for small sizes
// (at most SMALL_N rows / groups / scored units).  Each is one launch that
// reads its sizes from device memory, so a call needs no intermediate host
// synchronisation; sizes above SMALL_N leave a "not done" flag and the caller
// uses the multi-kernel path.  Sorting is a bitonic network in LDS; unit sums
// are a block-wide segmented scan.
#include <math.h>

#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t SMALL_N = 8192;       // groups / scored units
constexpr uint32_t ROWS_N = 16384;       // rows
constexpr uint32_t NT = 1024;            // threads
constexpr uint32_t PER = SMALL_N / NT;   // items per thread (blocked)
constexpr uint32_t RPER = ROWS_N / NT;
constexpr uint32_t NW = NT / 64;

__device__ __forceinline__ uint32_t pow2_at_least(uint32_t n) {
  uint32_t p = 1;
  while (p < n) p <<= 1;
  return p;
}

// Ascending bitonic sort of a[0..N), N a power of two, all threads.
__device__ void bitonic_u64(uint64_t* a, uint32_t N) {
  for (uint32_t k = 2; k <= N; k <<= 1)
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < N; i += NT) {
        const uint32_t p = i ^ j;
        if (p > i) {
          const uint64_t x = a[i], y = a[p];
          if ((x > y) == ((i & k) == 0)) { a[i] = y; a[p] = x; }
        }
      }
      __syncthreads();
    }
}

// Exclusive block scan of one u32 per thread; returns the block total too.
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

// ---------------------------------------------------------------- rows -> groups
// Sort rows by key (rk << 14 | row index), sum runs of equal rk.
__global__ __launch_bounds__(NT) void k_small_rows(Rows rows, SortedGroups out, unsigned long long* __restrict__ G_out,
                                                   uint32_t* __restrict__ done) {
  __shared__ uint64_t s_a[ROWS_N];
  __shared__ uint32_t s_w[NW];
  const uint64_t R = *rows.count;
  if (R > ROWS_N) {
    if (threadIdx.x == 0) *done = 0;
    return;
  }
  const uint32_t n = (uint32_t)R, N = pow2_at_least(n < 2 ? 2 : n);
  for (uint32_t i = threadIdx.x; i < N; i += NT) s_a[i] = i < n ? ((rows.rk[i] << 14) | i) : ~0ull;
  __syncthreads();
  bitonic_u64(s_a, N);
  auto is_head = [&](uint32_t i) { return i < n && (i == 0 || (s_a[i - 1] >> 14) != (s_a[i] >> 14)); };
  uint32_t heads = 0;
  for (uint32_t t = 0; t < RPER; ++t) heads += is_head(threadIdx.x * RPER + t) ? 1u : 0u;
  uint32_t total;
  uint32_t g = block_exscan(heads, s_w, total);
  for (uint32_t t = 0; t < RPER; ++t) {
    const uint32_t i = threadIdx.x * RPER + t;
    if (!is_head(i)) continue;
    const uint64_t rk = s_a[i] >> 14;
    u128 x = 0, r = 0;
    for (uint32_t e = i; e < n && (s_a[e] >> 14) == rk; ++e) {
      const uint32_t j = (uint32_t)(s_a[e] & (ROWS_N - 1));
      x += make_u128(rows.lo[j], rows.hi[j]);
      if (out.raw) r += make_u128(rows.rlo[j], rows.rhi[j]);
    }
    out.key[g] = (uint32_t)(rk >> 3);
    out.phase[g] = (uint8_t)(rk & 7);
    out.count[g] = (uint64_t)(x >> (64 + ATREX_COUNT_SHIFT));
    const u128 W = x & (((u128)1 << (64 + ATREX_COUNT_SHIFT)) - 1);
    out.wsum[2 * g] = (uint64_t)W;
    out.wsum[2 * g + 1] = (uint64_t)(W >> 64);
    if (out.raw) {
      out.raw[2 * g] = (uint64_t)r;
      out.raw[2 * g + 1] = (uint64_t)(r >> 64);
    }
    ++g;
  }
  if (threadIdx.x == 0) {
    *G_out = total;
    *done = 1;
  }
}

// ---------------------------------------------------------------- normalisation
// Per-phase totals S, weights RN(W)/RN(S), and Eq. (3) units for operators
// (key >> 16) and keys: U = (L / |Phi|) * sum W, w = RN(U) / RN(sum U).  The
// first row of each unit sums the unit's rows.
__global__ __launch_bounds__(NT) void k_small_normalize(SortedGroups g, uint64_t G, uint32_t P, uint64_t L,
                                                        uint64_t* __restrict__ S_out, uint32_t* __restrict__ okey,
                                                        uint8_t* __restrict__ oph, uint64_t* __restrict__ ocount,
                                                        uint64_t* __restrict__ owsum, uint64_t* __restrict__ oraw,
                                                        double* __restrict__ oweight, uint64_t* __restrict__ oS,
                                                        UnitTable ops, UnitTable keys,
                                                        unsigned long long* __restrict__ counts,
                                                        uint32_t* __restrict__ done) {
  __shared__ uint64_t s_lo[NW * 8], s_hi[NW * 8];
  __shared__ uint32_t s_w[NW];
  __shared__ uint64_t s_S[16];
  __shared__ uint64_t s_tot[2];
  if (G > SMALL_N) {
    if (threadIdx.x == 0) *done = 0;
    return;
  }
  const uint32_t n = (uint32_t)G;
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // per-phase totals: strided rows, one u128 per phase per thread
  for (uint32_t p = 0; p < P; ++p) {
    u128 acc = 0;
    for (uint32_t i = threadIdx.x; i < n; i += NT)
      if (g.phase[i] == p) acc += make_u128(g.wsum[2 * i], g.wsum[2 * i + 1]);
    acc = wave_sum_u128(acc);
    if (lane == 0) { s_lo[wave * 8 + p] = (uint64_t)acc; s_hi[wave * 8 + p] = (uint64_t)(acc >> 64); }
  }
  __syncthreads();
  if (threadIdx.x < P) {
    u128 t = 0;
    for (uint32_t v = 0; v < NW; ++v) t += make_u128(s_lo[v * 8 + threadIdx.x], s_hi[v * 8 + threadIdx.x]);
    s_S[2 * threadIdx.x] = (uint64_t)t;
    s_S[2 * threadIdx.x + 1] = (uint64_t)(t >> 64);
    S_out[2 * threadIdx.x] = oS[2 * threadIdx.x] = (uint64_t)t;
    S_out[2 * threadIdx.x + 1] = oS[2 * threadIdx.x + 1] = (uint64_t)(t >> 64);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < n; i += NT) {
    const uint32_t ph = g.phase[i];
    const u128 w = make_u128(g.wsum[2 * i], g.wsum[2 * i + 1]);
    const u128 Sp = make_u128(s_S[2 * ph], s_S[2 * ph + 1]);
    okey[i] = g.key[i];
    oph[i] = (uint8_t)ph;
    ocount[i] = g.count[i];
    owsum[2 * i] = g.wsum[2 * i];
    owsum[2 * i + 1] = g.wsum[2 * i + 1];
    if (oraw) { oraw[2 * i] = g.raw[2 * i]; oraw[2 * i + 1] = g.raw[2 * i + 1]; }
    oweight[i] = Sp == 0 ? 0.0 : u128_to_f64(w) / u128_to_f64(Sp);
  }
  // Eq. (3) units: u = 0 operators, u = 1 keys
  for (int u = 0; u < 2; ++u) {
    const int shift = u == 0 ? 16 : 0;
    const UnitTable tab = u == 0 ? ops : keys;
    auto is_head = [&](uint32_t i) { return i < n && (i == 0 || (g.key[i - 1] >> shift) != (g.key[i] >> shift)); };
    uint32_t nheads = 0;
    for (uint32_t t = 0; t < PER; ++t) nheads += is_head(threadIdx.x * PER + t) ? 1u : 0u;
    uint32_t nunits;
    uint32_t k = block_exscan(nheads, s_w, nunits);
    u128 myU = 0;
    for (uint32_t t = 0; t < PER; ++t) {
      const uint32_t i = threadIdx.x * PER + t;
      if (!is_head(i)) continue;
      const uint32_t id = g.key[i] >> shift;
      u128 sum = 0;
      uint32_t mask = 0;
      for (uint32_t e = i; e < n && (g.key[e] >> shift) == id; ++e) {
        sum += make_u128(g.wsum[2 * e], g.wsum[2 * e + 1]);
        mask |= 1u << g.phase[e];
      }
      const uint32_t nph = __popc(mask);
      const u128 U = nph ? (u128)(L / nph) * sum : (u128)0;
      tab.id[k] = id;
      tab.U[2 * k] = (uint64_t)U;
      tab.U[2 * k + 1] = (uint64_t)(U >> 64);
      myU += U;
      ++k;
    }
    const u128 tot = wave_sum_u128(myU);
    if (lane == 0) { s_lo[wave] = (uint64_t)tot; s_hi[wave] = (uint64_t)(tot >> 64); }
    __syncthreads();
    if (threadIdx.x == 0) {
      u128 T = 0;
      for (uint32_t v = 0; v < NW; ++v) T += make_u128(s_lo[v], s_hi[v]);
      s_tot[0] = (uint64_t)T;
      s_tot[1] = (uint64_t)(T >> 64);
      counts[u] = nunits;
    }
    __syncthreads();
    const u128 T = make_u128(s_tot[0], s_tot[1]);
    const double dT = u128_to_f64(T);
    for (uint32_t q = threadIdx.x; q < nunits; q += NT)
      tab.w[q] = T == 0 ? 0.0 : u128_to_f64(make_u128(tab.U[2 * q], tab.U[2 * q + 1])) / dT;
    __syncthreads();
  }
  if (threadIdx.x == 0) *done = 1;
}

// ---------------------------------------------------------------- score
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

// Ascending bitonic sort of (k, v) pairs by k, N a power of two, all threads.
__device__ void bitonic_pairs(uint64_t* k, uint32_t* v, uint32_t N) {
  for (uint32_t kk = 2; kk <= N; kk <<= 1)
    for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < N; i += NT) {
        const uint32_t p = i ^ j;
        if (p > i) {
          const uint64_t x = k[i], y = k[p];
          if ((x > y) == ((i & kk) == 0)) {
            k[i] = y;
            k[p] = x;
            const uint32_t t = v[i];
            v[i] = v[p];
            v[p] = t;
          }
        }
      }
      __syncthreads();
    }
}

// Eq. (4) validation, duplicate check, Eq. (5) medians, Eq. (6) weighted sum.
// Order within an operator: the S values sorted by their top 46 bits, runs of
// equal prefixes then sorted exactly by the head of the run (NaN last).
__global__ __launch_bounds__(NT) void k_small_score(const uint32_t* __restrict__ score_key,
                                                    const double* __restrict__ S, uint64_t n64, UnitTable opt,
                                                    uint64_t nops_trace, uint32_t* __restrict__ op_out,
                                                    double* __restrict__ w_out, double* __restrict__ s_out,
                                                    double* __restrict__ s_agg, uint64_t* __restrict__ totU,
                                                    unsigned long long* __restrict__ nret, uint64_t* __restrict__ rU,
                                                    uint32_t* __restrict__ err) {
  constexpr uint32_t HS = 2 * SMALL_N;  // duplicate-check hash set
  constexpr uint64_t NAN_KEY = ((uint64_t)1 << 46) - 1;
  __shared__ uint64_t s_k[SMALL_N];
  __shared__ uint32_t s_i[SMALL_N];
  __shared__ uint32_t s_w[NW];
  __shared__ uint32_t s_full;  // occurrences of the key equal to the free-slot marker
  __shared__ uint64_t s_u[NW * 2];
  uint32_t* s_h = (uint32_t*)s_k;       // duplicate check, before the sort keys are built
  double* s_cs = (double*)s_i;          // compensated sums, after the medians
  double* s_cc = (double*)s_i + NT;
  const uint32_t n = (uint32_t)n64;
  const uint32_t N = pow2_at_least(n < 2 ? 2 : n);
  // Eq. (4): S_j in (0, 1]; NaN = not correct
  bool bad = false;
  for (uint32_t j = threadIdx.x; j < n; j += NT) {
    const double v = S[j];
    bad |= !isnan(v) && !(v > 0.0 && v <= 1.0);
  }
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
  // duplicate keys: insert every key into an LDS hash set
  for (uint32_t i = threadIdx.x; i < HS; i += NT) s_h[i] = 0xFFFFFFFFu;
  if (threadIdx.x == 0) s_full = 0;
  __syncthreads();
  bool dup = false;
  for (uint32_t j = threadIdx.x; j < n; j += NT) {
    const uint32_t key = score_key[j];
    if (key == 0xFFFFFFFFu) {
      dup |= atomicAdd(&s_full, 1u) > 0;
      continue;
    }
    uint32_t h = (key * 0x9E3779B1u) >> (32 - 14);  // HS = 2^14
    for (;;) {
      const uint32_t cur = atomicCAS(&s_h[h], 0xFFFFFFFFu, key);
      if (cur == 0xFFFFFFFFu) break;
      if (cur == key) { dup = true; break; }
      h = (h + 1) & (HS - 1);
    }
  }
  if (__any(dup) && (threadIdx.x & 63) == 0) atomicOr(err, ATREX_ERRBIT_DUP);
  __syncthreads();
  // order by (operator, S prefix)
  for (uint32_t i = threadIdx.x; i < N; i += NT) {
    uint64_t k = ~0ull;
    if (i < n) {
      const double v = S[i];
      const uint64_t pre = isnan(v) ? NAN_KEY : (((uint64_t)__double_as_longlong(v) >> 16) & NAN_KEY);
      k = ((uint64_t)(score_key[i] >> 16) << 46) | pre;
    }
    s_k[i] = k;
    s_i[i] = i;
  }
  __syncthreads();
  bitonic_pairs(s_k, s_i, N);
  // exact order inside runs of equal (operator, prefix)
  for (uint32_t t = 0; t < PER; ++t) {
    const uint32_t i = threadIdx.x * PER + t;
    if (i >= n || (i > 0 && s_k[i - 1] == s_k[i])) continue;
    uint32_t e = i + 1;
    while (e < n && s_k[e] == s_k[i]) ++e;
    for (uint32_t a = i + 1; a < e; ++a) {  // insertion sort by full S bits
      const uint32_t x = s_i[a];
      const uint64_t xb = (uint64_t)__double_as_longlong(S[x]);
      uint32_t b = a;
      while (b > i && (uint64_t)__double_as_longlong(S[s_i[b - 1]]) > xb) {
        s_i[b] = s_i[b - 1];
        --b;
      }
      s_i[b] = x;
    }
  }
  __syncthreads();
  // operator segments: medians (Eq. (5)) and U of the retained operators
  auto is_head = [&](uint32_t i) { return i < n && (i == 0 || (s_k[i - 1] >> 46) != (s_k[i] >> 46)); };
  uint32_t ops_here = 0;
  for (uint32_t t = 0; t < PER; ++t) ops_here += is_head(threadIdx.x * PER + t) ? 1u : 0u;
  uint32_t nops;
  uint32_t ob = block_exscan(ops_here, s_w, nops);
  u128 myU = 0;
  for (uint32_t t = 0; t < PER; ++t) {
    const uint32_t i = threadIdx.x * PER + t;
    if (!is_head(i)) continue;
    const uint32_t op = (uint32_t)(s_k[i] >> 46);
    uint32_t e = i, c = 0;
    while (e < n && (s_k[e] >> 46) == op) {
      if ((s_k[e] & NAN_KEY) != NAN_KEY || !isnan(S[s_i[e]])) ++c;
      ++e;
    }
    double Si = 0.0;
    if (c) {
      const uint32_t h = c / 2;
      Si = (c & 1) ? S[s_i[i + h]] : (S[s_i[i + h - 1]] + S[s_i[i + h]]) / 2.0;
    }
    uint64_t lo = 0, hi = nops_trace;
    while (lo < hi) {
      const uint64_t mid = (lo + hi) / 2;
      if (opt.id[mid] < op) lo = mid + 1; else hi = mid;
    }
    u128 U = 0;
    if (lo < nops_trace && opt.id[lo] == op) U = make_u128(opt.U[2 * lo], opt.U[2 * lo + 1]);
    myU += U;
    op_out[ob] = op;
    s_out[ob] = Si;
    rU[2 * ob] = (uint64_t)U;
    rU[2 * ob + 1] = (uint64_t)(U >> 64);
    ++ob;
  }
  const u128 tu = wave_sum_u128(myU);
  if ((threadIdx.x & 63) == 0) { s_u[2 * (threadIdx.x >> 6)] = (uint64_t)tu; s_u[2 * (threadIdx.x >> 6) + 1] = (uint64_t)(tu >> 64); }
  __syncthreads();
  u128 T = 0;
  for (uint32_t v = 0; v < NW; ++v) T += make_u128(s_u[2 * v], s_u[2 * v + 1]);
  if (threadIdx.x == 0) {
    totU[0] = (uint64_t)T;
    totU[1] = (uint64_t)(T >> 64);
    *nret = nops;
  }
  const double dT = u128_to_f64(T);
  __syncthreads();  // s_i is reused below
  // Eq. (6): compensated sum over contiguous runs, then a TwoSum tree
  const uint32_t per = (nops + NT - 1) / NT;
  const uint32_t b = threadIdx.x * per, e = min(b + per, nops);
  Comp accs{0.0, 0.0};
  for (uint32_t k = b; k < e; ++k) {
    const double wk = T == 0 ? 0.0 : u128_to_f64(make_u128(rU[2 * k], rU[2 * k + 1])) / dT;
    w_out[k] = wk;
    accs = comp_add(accs, __dmul_rn(wk, s_out[k]));
  }
  s_cs[threadIdx.x] = accs.s;
  s_cc[threadIdx.x] = accs.c;
  __syncthreads();
  for (uint32_t d = NT / 2; d >= 1; d >>= 1) {
    if (threadIdx.x < d) {
      const Comp m = comp_merge(Comp{s_cs[threadIdx.x], s_cc[threadIdx.x]}, Comp{s_cs[threadIdx.x + d], s_cc[threadIdx.x + d]});
      s_cs[threadIdx.x] = m.s;
      s_cc[threadIdx.x] = m.c;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *s_agg = s_cs[0] + s_cc[0];
}

}  // namespace

uint32_t small_n() { return SMALL_N; }
uint32_t small_rows_n() { return ROWS_N; }

void launch_small_rows(hipStream_t s, const Rows& rows, const SortedGroups& out, unsigned long long* G_out,
                       uint32_t* done) {
  hipLaunchKernelGGL(k_small_rows, dim3(1), dim3(NT), 0, s, rows, out, G_out, done);
}

void launch_small_normalize(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t L, uint64_t* S_out,
                            uint32_t* okey, uint8_t* oph, uint64_t* ocount, uint64_t* owsum, uint64_t* oraw,
                            double* oweight, uint64_t* oS, UnitTable ops, UnitTable keys,
                            unsigned long long* counts, uint32_t* done) {
  hipLaunchKernelGGL(k_small_normalize, dim3(1), dim3(NT), 0, s, g, G, P, L, S_out, okey, oph, ocount, owsum, oraw,
                     oweight, oS, ops, keys, counts, done);
}

void launch_small_score(hipStream_t s, const uint32_t* score_key, const double* S, uint64_t n, UnitTable opt,
                        uint64_t nops_trace, uint32_t* op_out, double* w_out, double* s_out, double* s_agg,
                        uint64_t* totU, unsigned long long* nret, uint64_t* rU, uint32_t* err) {
  hipLaunchKernelGGL(k_small_score, dim3(1), dim3(NT), 0, s, score_key, S, n, opt, nops_trace, op_out, w_out, s_out,
                     s_agg, totU, nret, rU, err);
}
