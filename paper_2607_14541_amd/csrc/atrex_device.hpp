// atrex_device.hpp -- device helpers shared by the gfx950 kernels.
//
// Fixed-point conventions (see include/atrex.h):
//   scale word per (app, phase): 0 = no share, else
//     bits 56..63 = rho + 64 (rho in [-63, 96]), bits 0..54 = m - 2^55,
//     m in [2^55, 2^56) the truncated mantissa of r = 2^96 c_a / (C T).
//   per-event share v = floor(dur * m * 2^(rho - 55)) <= 2^96  (Eq. (3) term
//   p_a * d / D_a^phi in Q96).
//   A (key, phase) accumulator is two 64-bit words:
//     lo = (sum v) mod 2^64,
//     hi = floor(sum v / 2^64) + count * 2^33   (floor(...) <= 2^32 because the
//          shares of one phase sum to at most 2^96; count < 2^31).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef unsigned __int128 u128;

#define ATREX_EMPTY_KEY 0xFFFFFFFFu  // LDS tag of a free slot
#define ATREX_COUNT_SHIFT 33
#define ATREX_MANT_BITS 56

// --- scale word -----------------------------------------------------------
__device__ __forceinline__ uint64_t scale_pack(uint64_t m, int rho) {
  return ((uint64_t)(rho + 64) << 56) | (m - ((uint64_t)1 << (ATREX_MANT_BITS - 1)));
}

// v = floor(d * m * 2^(rho - 55)); exact because the product fits in 119 bits
// and the true value is at most 2^96.
__device__ __forceinline__ u128 event_share(uint64_t d, uint64_t sw) {
  if (sw == 0) return 0;
  const uint64_t m = (sw & (((uint64_t)1 << 55) - 1)) | ((uint64_t)1 << 55);
  const int sh = (int)(sw >> 56) - 64 - (ATREX_MANT_BITS - 1);
  const u128 p = (u128)d * m;
  return sh >= 0 ? (p << sh) : (p >> (-sh));
}

// Right-shift amount of the share when rho <= 55 and 55 - rho < 64 (the
// common case: every (app, phase) whose share of a single invocation is below
// 2^55 in Q96), else -1.
__device__ __forceinline__ int share_rshift(uint64_t sw) {
  const int s = 55 + 64 - (int)(sw >> 56);
  return (s >= 0 && s < 64) ? s : -1;
}

// event_share for a scale word with share_rshift(sw) = s in [0, 63]:
// (d * m) >> s with 64-bit halves (sw = 0 gives 0 since m is then masked to 0).
__device__ __forceinline__ void event_share_rs(uint64_t d, uint64_t sw, int s, uint64_t& vlo, uint64_t& vhi) {
  const uint64_t m = sw ? ((sw & (((uint64_t)1 << 55) - 1)) | ((uint64_t)1 << 55)) : 0;
  const uint64_t lo = d * m;
  const uint64_t hi = __umul64hi(d, m);
  vlo = s ? ((lo >> s) | (hi << (64 - s))) : lo;
  vhi = hi >> s;
}

// --- pass-B scale word ------------------------------------------------------
// bits 0..55 = m, bits 56..63 = u = 63 - rho for rho in [-8, 63] (u in [0, 71]),
// so that v = floor(d * (m * 2^8) / 2^u); u = 255 marks the rare rho outside
// [-8, 63], which takes the general scale word.  0 = no share.
#define ATREX_BSCALE_SLOW 255u
__device__ __forceinline__ uint64_t bscale_pack(uint64_t m, int rho) {
  const uint64_t u = (rho >= -8 && rho <= 63) ? (uint64_t)(63 - rho) : (uint64_t)ATREX_BSCALE_SLOW;
  return (u << 56) | m;
}

// Share of an event with d < 2^32 from a pass-B word (u <= 71), given as its
// two 32-bit halves: Y = d * (m * 2^8) < 2^96 in three words from two
// 32 x 32 -> 64-bit products, then v = Y >> u (< 2^96) by selecting words on
// bits 5 and 6 of u and funnel-shifting by u mod 32.
__device__ __forceinline__ void bscale_share32(uint32_t d, uint32_t elo, uint32_t ehi, uint64_t& vlo,
                                               uint32_t& vhi) {
  const uint32_t u = ehi >> 24;
  const uint32_t M0 = elo << 8, M1 = __builtin_amdgcn_alignbit(ehi & 0xFFFFFFu, elo, 24u);
  const uint64_t p0 = (uint64_t)d * M0;
  const uint64_t p1 = (uint64_t)d * M1 + (p0 >> 32);
  const uint32_t y0 = (uint32_t)p0, y1 = (uint32_t)p1, y2 = (uint32_t)(p1 >> 32);
  const bool b1 = (u & 32u) != 0, b2 = (u & 64u) != 0;
  const uint32_t g0 = b1 ? y1 : y0, g1 = b1 ? y2 : y1, g2 = b1 ? 0u : y2;
  const uint32_t f0 = b2 ? g2 : g0, f1 = b2 ? 0u : g1, f2 = b2 ? 0u : g2;
  vlo = ((uint64_t)__builtin_amdgcn_alignbit(f2, f1, u) << 32) | __builtin_amdgcn_alignbit(f1, f0, u);
  vhi = f2 >> (u & 31u);
}

// The same for any duration d < 2^63 (u <= 71): Y = d * (m * 2^8) < 2^127 in
// four words from four 32 x 32 -> 64-bit products, v = Y >> u (<= 2^96).
__device__ __forceinline__ void bscale_share64(uint64_t d, uint32_t elo, uint32_t ehi, uint64_t& vlo, uint64_t& vhi) {
  const uint32_t u = ehi >> 24;
  const uint32_t M0 = elo << 8, M1 = __builtin_amdgcn_alignbit(ehi & 0xFFFFFFu, elo, 24u);
  const uint32_t d0 = (uint32_t)d, d1 = (uint32_t)(d >> 32);
  const uint64_t p00 = (uint64_t)d0 * M0;
  const uint64_t t1 = (uint64_t)d0 * M1 + (p00 >> 32);
  const uint64_t t2 = (uint64_t)d1 * M0 + (uint32_t)t1;
  const uint64_t t3 = (uint64_t)d1 * M1 + ((t1 >> 32) + (t2 >> 32));
  const uint32_t y0 = (uint32_t)p00, y1 = (uint32_t)t2, y2 = (uint32_t)t3, y3 = (uint32_t)(t3 >> 32);
  const bool b1 = (u & 32u) != 0, b2 = (u & 64u) != 0;
  const uint32_t g0 = b1 ? y1 : y0, g1 = b1 ? y2 : y1, g2 = b1 ? y3 : y2, g3 = b1 ? 0u : y3;
  const uint32_t f0 = b2 ? g2 : g0, f1 = b2 ? g3 : g1, f2 = b2 ? 0u : g2, f3 = b2 ? 0u : g3;
  vlo = ((uint64_t)__builtin_amdgcn_alignbit(f2, f1, u) << 32) | __builtin_amdgcn_alignbit(f1, f0, u);
  vhi = ((uint64_t)(f3 >> (u & 31u)) << 32) | __builtin_amdgcn_alignbit(f3, f2, u);
}

// --- u128 -> fp64, round to nearest, ties to even (IEEE 754 conversion) -----
// The top 64 bits from the leading one on, with a sticky bit for any nonzero
// bit below them, round to the same double as x; that u64 is converted as
// (high word) 2^32 + (low word): both terms are exact, so the one addition is
// the only rounding.  The power-of-two scaling is exact.
__device__ __forceinline__ double u128_to_f64(u128 x) {
  const uint64_t hi = (uint64_t)(x >> 64), lo = (uint64_t)x;
  const int s = hi ? __clzll(hi) : 0;
  const uint64_t top = s ? (hi << s) | (lo >> (64 - s)) : hi;
  const uint64_t below = s ? lo << s : lo;
  const uint64_t t = hi ? top | (below != 0 ? 1u : 0u) : lo;
  const double r = ldexp((double)(uint32_t)(t >> 32), 32) + (double)(uint32_t)t;
  return hi ? ldexp(r, 64 - s) : r;
}

// --- global -> LDS staging by one workgroup -------------------------------------
// dst[j] = f(src[j]) for j < n, by the NT threads of the workgroup; each
// thread issues its KL loads of a round before the first store, so a round
// costs one memory latency instead of KL.
template <uint32_t NT, int KL, typename D, typename T, typename F>
__device__ __forceinline__ void lds_stage(D* dst, const T* __restrict__ src, uint32_t n, F f) {
  for (uint32_t j0 = 0; j0 < n; j0 += KL * NT) {
    T v[KL];
#pragma unroll
    for (int k = 0; k < KL; ++k) {
      const uint32_t j = j0 + (uint32_t)k * NT + threadIdx.x;
      v[k] = j < n ? src[j] : T();
    }
#pragma unroll
    for (int k = 0; k < KL; ++k) {
      const uint32_t j = j0 + (uint32_t)k * NT + threadIdx.x;
      if (j < n) dst[j] = f(v[k]);
    }
  }
}

// --- hashing ----------------------------------------------------------------
// Multiplicative (Fibonacci) hash; the slot is taken from the high bits.  The
// multiplier is the odd integer nearest 2^32 / phi (golden ratio), Knuth's
// multiplicative hashing (TAOCP vol. 3, §6.4).
__device__ __forceinline__ uint32_t hash_mul(uint32_t k) { return k * 0x9E3779B1u; }

// Home bucket of key k in an LDS table of NB buckets of four slots (NB <
// 2^16): floor((hash >> 8) * (NB - 1) / 2^24), always below NB - 1, so the
// key's window (its home bucket and the next) lies inside the table.
__device__ __forceinline__ uint32_t lds_home_bucket(uint32_t k, uint32_t NB) {
  return (uint32_t)(((uint64_t)(hash_mul(k) >> 8) * ((NB - 1) << 8)) >> 32);
}

// Bucket of key k in a table of NB four-slot buckets whose keys sit in their
// bucket only (no window): floor(hash * NB / 2^32).
__device__ __forceinline__ uint32_t lds_only_bucket(uint32_t k, uint32_t NB) {
  return (uint32_t)(((uint64_t)hash_mul(k) * NB) >> 32);
}

// Wave-aggregated LDS counter increment: lanes whose bucket equals the first
// active lane's add once together (a hot bucket costs one atomic per wave);
// returns each lane's rank among the increments of its counter.
__device__ __forceinline__ uint32_t count_in(uint32_t* cnt, uint32_t b, bool active) {
  const uint64_t act = __ballot(active);
  if (act == 0) return 0;
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t lead = __builtin_amdgcn_readlane(b, __ffsll((unsigned long long)act) - 1);
  const uint64_t same = __ballot(active && b == lead);
  uint32_t base = 0;
  if (lane == (uint32_t)(__ffsll((unsigned long long)act) - 1)) base = atomicAdd(&cnt[lead], (uint32_t)__popcll(same));
  base = __builtin_amdgcn_readlane(base, __ffsll((unsigned long long)act) - 1);
  if (active && b == lead) return base + (uint32_t)__popcll(same & ((1ull << lane) - 1ull));
  return active ? atomicAdd(&cnt[b], 1u) : 0u;
}

#define ATREX_NO_SLOT 0xFFFFFFFFu

// Key `k` is in a seeded table image of S slots whose keys sit in their own
// four-slot bucket (lds_only_bucket): its slot, else ATREX_NO_SLOT.  The
// reserved key is never in the image (it marks free slots).
__device__ __forceinline__ uint32_t image_slot(const uint32_t* s_img, uint32_t S, uint32_t k) {
  const uint32_t b = lds_only_bucket(k, S / 4);
  const uint4 t = *(const uint4*)&s_img[4 * b];
  uint32_t x = ATREX_NO_SLOT;
  x = t.w == k ? 4 * b + 3 : x;
  x = t.z == k ? 4 * b + 2 : x;
  x = t.y == k ? 4 * b + 1 : x;
  x = t.x == k ? 4 * b : x;
  return k == ATREX_EMPTY_KEY ? ATREX_NO_SLOT : x;
}

// An invertible 32-bit mixer of xorshift-multiply rounds (shifts 16, 15, 16):
// the "lowbias32" function found by C. Wellons' hash-prospector search
// (published 2018, public domain).  Every round is a bijection, so the key can
// be recovered from the hash (the inverse is unmix32 in kernels_rows.hip).
__device__ __forceinline__ uint32_t hash32(uint32_t k) {
  k ^= k >> 16;
  k *= 0x7feb352dU;
  k ^= k >> 15;
  k *= 0x846ca68bU;
  k ^= k >> 16;
  return k;
}

// --- wave helpers (wave64) -------------------------------------------------------
__device__ __forceinline__ uint64_t u128_lo(u128 x) { return (uint64_t)x; }
__device__ __forceinline__ uint64_t u128_hi(u128 x) { return (uint64_t)(x >> 64); }
__device__ __forceinline__ u128 make_u128(uint64_t lo, uint64_t hi) {
  return ((u128)hi << 64) | lo;
}

__device__ __forceinline__ u128 shfl_down_u128(u128 v, int d) {
  const uint64_t lo = __shfl_down((unsigned long long)(uint64_t)v, d, 64);
  const uint64_t hi = __shfl_down((unsigned long long)(uint64_t)(v >> 64), d, 64);
  return make_u128(lo, hi);
}

__device__ __forceinline__ u128 shfl_up_u128(u128 v, int d) {
  const uint64_t lo = __shfl_up((unsigned long long)(uint64_t)v, d, 64);
  const uint64_t hi = __shfl_up((unsigned long long)(uint64_t)(v >> 64), d, 64);
  return make_u128(lo, hi);
}

__device__ __forceinline__ u128 wave_sum_u128(u128 v) {
  for (int d = 32; d >= 1; d >>= 1) v += shfl_down_u128(v, d);
  return v;  // valid in lane 0
}

// Inclusive scan over the 64 lanes of a wave (lane i gets x_0 + ... + x_i)
// by DPP: row shifts by 1, 2, 4 and 8 lanes within each row of 16, then the
// broadcasts of lane 15 into rows 1 and 3 and of lane 31 into rows 2 and 3.
// Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Sum over the 64 lanes of a wave of a u32 whose total fits in 32 bits,
// returned in every lane (lane 63 of the inclusive scan).
__device__ __forceinline__ uint32_t wave_total_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan_u32(x), 63);
}

// Wave total of a u128 below 2^98 per lane, in every lane: four 26-bit limbs,
// whose sums over 64 lanes stay below 2^32, summed with wave_total_u32.
__device__ __forceinline__ u128 wave_total_u98(u128 v) {
  const uint32_t M = (1u << 26) - 1;
  const uint64_t lo = (uint64_t)v, hi = (uint64_t)(v >> 64);
  const uint32_t l0 = wave_total_u32((uint32_t)lo & M);
  const uint32_t l1 = wave_total_u32((uint32_t)(lo >> 26) & M);
  const uint32_t l2 = wave_total_u32((uint32_t)((lo >> 52) | (hi << 12)) & M);
  const uint32_t l3 = wave_total_u32((uint32_t)(hi >> 14));
  return (u128)l0 + ((u128)l1 << 26) + ((u128)l2 << 52) + ((u128)l3 << 78);
}

// Accumulate a share into a two-word accumulator (global or LDS) with
// 64-bit atomics: the low word's carry is detected from the returned value.
template <typename Ptr>
__device__ __forceinline__ void acc_add(Ptr lo, Ptr hi, u128 v) {
  const unsigned long long vlo = (unsigned long long)(uint64_t)v;
  const unsigned long long old = atomicAdd(lo, vlo);
  const unsigned long long carry = (old + vlo < old) ? 1ull : 0ull;
  atomicAdd(hi, (unsigned long long)(uint64_t)(v >> 64) + carry + (1ull << ATREX_COUNT_SHIFT));
}

// The same for a pre-summed share of `count` invocations.
template <typename Ptr>
__device__ __forceinline__ void acc_add_n(Ptr lo, Ptr hi, u128 v, uint32_t count) {
  const unsigned long long vlo = (unsigned long long)(uint64_t)v;
  const unsigned long long old = atomicAdd(lo, vlo);
  const unsigned long long carry = (old + vlo < old) ? 1ull : 0ull;
  atomicAdd(hi, (unsigned long long)(uint64_t)(v >> 64) + carry +
                    ((unsigned long long)count << ATREX_COUNT_SHIFT));
}

// Plain (count-free) 128-bit accumulation, e.g. raw device time.
template <typename Ptr>
__device__ __forceinline__ void acc_add_plain(Ptr lo, Ptr hi, u128 v) {
  const unsigned long long vlo = (unsigned long long)(uint64_t)v;
  const unsigned long long old = atomicAdd(lo, vlo);
  const unsigned long long carry = (old + vlo < old) ? 1ull : 0ull;
  const unsigned long long vhi = (unsigned long long)(uint64_t)(v >> 64) + carry;
  if (vhi) atomicAdd(hi, vhi);
}

// --- hot entries in registers --------------------------------------------------
// Up to two accumulator entries (a slot and phase of an LDS table) that most
// lanes of a wave hit, chosen once from the wave's first step (at least
// `min_lanes` of its 64 lanes on one entry).  A record of a hot entry is added
// to per-lane registers instead of by two LDS atomics; flush() sums the lanes
// once and hands each entry's total to the caller in lane 0.
template <bool RAW>
struct HotPair {
  static constexpr uint32_t NONE = 0xFFFFFFFFu;
  uint32_t ga, gb;  // wave-uniform entries (NONE: unused)
  u128 va, vb;      // share sums
  u128 ra, rb;      // raw time sums (RAW)
  uint32_t ca, cb;  // invocation counts
  __device__ __forceinline__ void reset() {
    ga = gb = NONE;
    va = vb = ra = rb = 0;
    ca = cb = 0;
  }
  __device__ __forceinline__ void choose(uint32_t gi, uint32_t min_lanes) {
    const uint64_t act = __ballot(gi != NONE);
    if (act == 0) return;
    const uint32_t l1 = __builtin_amdgcn_readlane(gi, __ffsll((unsigned long long)act) - 1);
    const uint64_t s1 = __ballot(gi == l1);
    uint32_t a = NONE, b = NONE;
    if ((uint32_t)__popcll(s1) >= min_lanes) a = l1;
    const uint64_t rest = act & ~s1;
    if (rest) {
      const uint32_t l2 = __builtin_amdgcn_readlane(gi, __ffsll((unsigned long long)rest) - 1);
      if ((uint32_t)__popcll(__ballot(gi == l2)) >= min_lanes) {
        if (a == NONE) a = l2; else b = l2;
      }
    }
    ga = __builtin_amdgcn_readfirstlane(a);
    gb = __builtin_amdgcn_readfirstlane(b);
  }
  // adds the record and returns true when gi is a hot entry
  __device__ __forceinline__ bool take(uint32_t gi, uint64_t lo, uint64_t hi, uint64_t d) {
    if (ga == NONE) return false;  // wave-uniform
    const bool a = gi == ga, b = gb != NONE && gi == gb;
    const u128 v = make_u128(lo, hi);
    va += a ? v : (u128)0;
    vb += b ? v : (u128)0;
    ca += a ? 1u : 0u;
    cb += b ? 1u : 0u;
    if (RAW) {
      ra += a ? (u128)d : (u128)0;
      rb += b ? (u128)d : (u128)0;
    }
    return a || b;
  }
  // add(entry, share total, count, raw total) is called in lane 0 per used entry
  template <class F>
  __device__ __forceinline__ void flush(F add) {
    if (ga == NONE) return;  // wave-uniform
    for (int e = 0; e < 2; ++e) {
      const uint32_t g = e ? gb : ga;
      if (g == NONE) continue;
      const u128 tv = wave_sum_u128(e ? vb : va);
      const u128 tr = RAW ? wave_sum_u128(e ? rb : ra) : (u128)0;
      uint32_t c = e ? cb : ca;
      for (int d = 32; d >= 1; d >>= 1) c += __shfl_down(c, d, 64);
      if ((threadIdx.x & 63) == 0 && c) add(g, tv, c, tr);
    }
  }
};

// --- streaming event loads ----------------------------------------------------
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef long long v2l __attribute__((ext_vector_type(2)));

// Four consecutive events starting at a multiple of 4 (16-byte aligned SoA),
// with 16-byte non-temporal vector loads.
// The four phases stay packed, one byte each, until used: unpacking them
// right after the load would wait for it, and (loads completing in order)
// for every load issued before it.
struct Ev4 {
  uint32_t key[4], app[4];
  uint32_t ph4;
  int64_t dur[4];
  __device__ __forceinline__ uint32_t ph(int j) const { return (ph4 >> (8 * j)) & 0xFFu; }
};

// NO_APP: the events carry no application (plain device-time group-by);
// every event belongs to application 0 and the app array is not read.
template <bool WITH_KEY, bool NO_APP = false>
__device__ __forceinline__ void load4(const uint32_t* __restrict__ key, const uint32_t* __restrict__ app,
                                      const uint8_t* __restrict__ phase, const int64_t* __restrict__ dur,
                                      uint64_t i, Ev4& e) {
  if (WITH_KEY) {
    const v4u k = __builtin_nontemporal_load((const v4u*)(key + i));
    e.key[0] = k.x; e.key[1] = k.y; e.key[2] = k.z; e.key[3] = k.w;
  }
  const v4u a = NO_APP ? v4u{0u, 0u, 0u, 0u} : __builtin_nontemporal_load((const v4u*)(app + i));
  const uint32_t p = __builtin_nontemporal_load((const uint32_t*)(phase + i));
  const v2l d0 = __builtin_nontemporal_load((const v2l*)(dur + i));
  const v2l d1 = __builtin_nontemporal_load((const v2l*)(dur + i + 2));
  e.app[0] = a.x; e.app[1] = a.y; e.app[2] = a.z; e.app[3] = a.w;
  e.ph4 = p;
  e.dur[0] = d0.x; e.dur[1] = d0.y; e.dur[2] = d1.x; e.dur[3] = d1.y;
}

// The same for a wave whose 64 groups of four all exist: event index e0 of
// lane 0 is wave-uniform, so each load takes a scalar base address and a
// 32-bit lane offset.
template <bool NO_APP = false>
__device__ __forceinline__ void load4_lane(const uint32_t* __restrict__ key, const uint32_t* __restrict__ app,
                                           const uint8_t* __restrict__ phase, const int64_t* __restrict__ dur,
                                           uint64_t e0, uint32_t lane, Ev4& e) {
  const v4u k = __builtin_nontemporal_load((const v4u*)(key + e0) + lane);
  const v4u a = NO_APP ? v4u{0u, 0u, 0u, 0u} : __builtin_nontemporal_load((const v4u*)(app + e0) + lane);
  const uint32_t p = __builtin_nontemporal_load((const uint32_t*)(phase + e0) + lane);
  const v2l d0 = __builtin_nontemporal_load((const v2l*)(dur + e0) + 2 * lane);
  const v2l d1 = __builtin_nontemporal_load((const v2l*)(dur + e0) + 2 * lane + 1);
  e.key[0] = k.x; e.key[1] = k.y; e.key[2] = k.z; e.key[3] = k.w;
  e.app[0] = a.x; e.app[1] = a.y; e.app[2] = a.z; e.app[3] = a.w;
  e.ph4 = p;
  e.dur[0] = d0.x; e.dur[1] = d0.y; e.dur[2] = d1.x; e.dur[3] = d1.y;
}

// Application of event i (0 for events that carry none).
template <bool NO_APP>
__device__ __forceinline__ uint32_t app_at(const uint32_t* __restrict__ app, uint64_t i) {
  return NO_APP ? 0u : app[i];
}

// Error bits of the device error word.
#define ATREX_ERRBIT_RANGE 1u
#define ATREX_ERRBIT_CAPACITY 2u
#define ATREX_ERRBIT_DUP 4u
#define ATREX_ERRBIT_SPILL 8u
