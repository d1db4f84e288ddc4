// kernels_aggregate.hip -- gfx950 kernels for the group-by of §3.4:
//   pass A  (Eq. (2)): T[a,ph] = sum of dur over the invocations of (a, ph)
//   scale   (Eq. (3)): the Q96 factor p_a / T[a,ph] as (m, rho)
//   pass B  (Eq. (2)-(3)): W[k,ph] = sum over invocations of dur * p_a / T[a,ph]
//   compaction of the distinct (key, phase) groups.
// Events are a struct of arrays (key u32, app u32, phase u8, dur i64) read
// with 16-byte nontemporal vector loads, four events per thread per step.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef long long v2l __attribute__((ext_vector_type(2)));

namespace {

// ---------------------------------------------------------------------------
// Streaming event loads: four consecutive events starting at a multiple of 4.
struct Ev4 {
  uint32_t key[4], app[4];
  uint32_t ph[4];
  int64_t dur[4];
};

template <bool WITH_KEY>
__device__ __forceinline__ void load4(const uint32_t* __restrict__ key, const uint32_t* __restrict__ app,
                                      const uint8_t* __restrict__ phase, const int64_t* __restrict__ dur,
                                      uint64_t i, Ev4& e) {
  if (WITH_KEY) {
    const v4u k = __builtin_nontemporal_load((const v4u*)(key + i));
    e.key[0] = k.x; e.key[1] = k.y; e.key[2] = k.z; e.key[3] = k.w;
  }
  const v4u a = __builtin_nontemporal_load((const v4u*)(app + i));
  const uint32_t p = __builtin_nontemporal_load((const uint32_t*)(phase + i));
  const v2l d0 = __builtin_nontemporal_load((const v2l*)(dur + i));
  const v2l d1 = __builtin_nontemporal_load((const v2l*)(dur + i + 2));
  e.app[0] = a.x; e.app[1] = a.y; e.app[2] = a.z; e.app[3] = a.w;
  e.ph[0] = p & 0xFF; e.ph[1] = (p >> 8) & 0xFF; e.ph[2] = (p >> 16) & 0xFF; e.ph[3] = p >> 24;
  e.dur[0] = d0.x; e.dur[1] = d0.y; e.dur[2] = d1.x; e.dur[3] = d1.y;
}

__device__ __forceinline__ void flag_error(uint32_t* err, bool bad, uint32_t bit) {
  // one atomic per wave that saw a bad event
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, bit);
}

// ---------------------------------------------------------------------------
// Pass A, LDS-privatised dense histogram on g = a * P + ph.  Each workgroup
// keeps the low 64 bits of its partial sums in LDS; the (rare) wrap-arounds
// are counted in a global carry table.  Partials go to partial[block][g].
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_pass_a_lds(EventsDev ev, uint32_t A, uint32_t P, uint32_t G,
                                                      unsigned long long* __restrict__ partial,
                                                      unsigned long long* __restrict__ carry,
                                                      uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long s_lo[];
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) s_lo[g] = 0;
  __syncthreads();
  const uint64_t n = ev.n, n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * BLOCK;
  bool bad = false;
  for (uint64_t q = (uint64_t)blockIdx.x * BLOCK + threadIdx.x; q < n4; q += stride) {
    Ev4 e;
    load4<false>(ev.key, ev.app, ev.phase, ev.dur, q * 4, e);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = e.app[j] < A && e.ph[j] < P && e.dur[j] >= 0;
      bad |= !ok;
      if (ok) {
        const uint32_t g = e.app[j] * P + e.ph[j];
        const unsigned long long d = (unsigned long long)e.dur[j];
        const unsigned long long old = atomicAdd(&s_lo[g], d);
        if (old + d < old) atomicAdd(&carry[g], 1ull);
      }
    }
  }
  if (blockIdx.x == 0) {  // tail events
    for (uint64_t i = n4 * 4 + threadIdx.x; i < n; i += BLOCK) {
      const uint32_t a = ev.app[i], ph = ev.phase[i];
      const int64_t dd = ev.dur[i];
      const bool ok = a < A && ph < P && dd >= 0;
      bad |= !ok;
      if (ok) {
        const uint32_t g = a * P + ph;
        const unsigned long long old = atomicAdd(&s_lo[g], (unsigned long long)dd);
        if (old + (unsigned long long)dd < old) atomicAdd(&carry[g], 1ull);
      }
    }
  }
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
  __syncthreads();
  unsigned long long* out = partial + (size_t)blockIdx.x * G;
  for (uint32_t g = threadIdx.x; g < G; g += BLOCK) out[g] = s_lo[g];
}

// T[g] = sum over blocks of partial[b][g] + carry[g] * 2^64.
__global__ void k_pass_a_reduce(const unsigned long long* __restrict__ partial, uint32_t nb, uint32_t G,
                                const unsigned long long* __restrict__ carry, uint64_t* __restrict__ T) {
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  u128 s = (u128)carry[g] << 64;
  for (uint32_t b = 0; b < nb; ++b) s += partial[(size_t)b * G + g];
  T[2 * g] = (uint64_t)s;
  T[2 * g + 1] = (uint64_t)(s >> 64);
}

// Pass A straight into global 128-bit accumulators (any number of (a, ph)).
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_pass_a_global(EventsDev ev, uint32_t A, uint32_t P,
                                                         unsigned long long* __restrict__ T,
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
    }
  }
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
}

// ---------------------------------------------------------------------------
// Scale, Eq. (3): for each (a, ph) with T > 0 and c_a > 0,
//   r = 2^96 c_a / (C T), rho = floor(log2 r), m = floor(r 2^(55 - rho)).
// With r0 = bitlen(2^96 c_a) - bitlen(C T), r lies in (2^(r0-1), 2^(r0+1)), so
// q = floor(2^96 c_a 2^(56 - r0) / (C T)) lies in [2^55, 2^57): if q >= 2^56
// then rho = r0 and m = floor(q / 2), else rho = r0 - 1 and m = q.  q is found
// by 57 steps of shift-and-subtract long division on 4 x 64-bit limbs.
struct W256 {
  uint64_t w[4];
};

__device__ __forceinline__ int w256_bitlen(const W256& a) {
#pragma unroll
  for (int i = 3; i >= 0; --i)
    if (a.w[i]) return 64 * i + 64 - __clzll(a.w[i]);
  return 0;
}

__device__ __forceinline__ W256 w256_shl(const W256& a, int s) {  // 0 <= s < 256
  W256 r;
  const int L = s >> 6, b = s & 63;
#pragma unroll
  for (int i = 3; i >= 0; --i) {
    const int j = i - L;
    uint64_t v = 0;
    if (j >= 0) {
      v = a.w[j] << b;
      if (b && j >= 1) v |= a.w[j - 1] >> (64 - b);
    }
    r.w[i] = v;
  }
  return r;
}

__device__ __forceinline__ bool w256_ge(const W256& a, const W256& b) {
#pragma unroll
  for (int i = 3; i >= 0; --i)
    if (a.w[i] != b.w[i]) return a.w[i] > b.w[i];
  return true;
}

__device__ __forceinline__ void w256_sub_inplace(W256& a, const W256& b) {
  uint64_t br = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint64_t x = a.w[i], y = b.w[i];
    const uint64_t d = x - y - br;
    br = (x < y) || (x - y < br) ? 1 : 0;
    a.w[i] = d;
  }
}

__global__ void k_scale(const uint64_t* __restrict__ T, const uint32_t* __restrict__ c,
                        const uint64_t* __restrict__ Csum, uint32_t A, uint32_t P,
                        uint64_t* __restrict__ scale) {
  const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= A * P) return;
  const u128 t = make_u128(T[2 * g], T[2 * g + 1]);
  const uint32_t ca = c[g / P];
  if (t == 0 || ca == 0) {
    scale[g] = 0;
    return;
  }
  const uint64_t C = *Csum;
  // Y = C * T (at most 159 bits)
  const u128 p0 = (u128)C * (uint64_t)t;
  const u128 p1 = (u128)C * (uint64_t)(t >> 64);
  W256 Y;
  Y.w[0] = (uint64_t)p0;
  const u128 mid = (p0 >> 64) + (uint64_t)p1;
  Y.w[1] = (uint64_t)mid;
  Y.w[2] = (uint64_t)((p1 >> 64) + (mid >> 64));
  Y.w[3] = 0;
  const int bx = 96 + 32 - __clz(ca);  // bitlen(2^96 c_a)
  const int r0 = bx - w256_bitlen(Y);
  // numerator 2^(96 + s1) c_a, denominator Y 2^s2, quotient < 2^57
  const int s1 = r0 < 56 ? 56 - r0 : 0;
  const int s2 = r0 > 56 ? r0 - 56 : 0;
  const W256 den = w256_shl(Y, s2);
  W256 rem;  // numerator >> 57; the numerator's low 57 bits are zero
  rem.w[0] = ca; rem.w[1] = rem.w[2] = rem.w[3] = 0;
  rem = w256_shl(rem, 96 + s1 - 57);
  uint64_t q = 0;
  for (int i = 56; i >= 0; --i) {
    rem = w256_shl(rem, 1);
    q <<= 1;
    if (w256_ge(rem, den)) {
      w256_sub_inplace(rem, den);
      q |= 1;
    }
  }
  int rho;
  uint64_t m;
  if (q >> 56) {
    rho = r0;
    m = q >> 1;
  } else {
    rho = r0 - 1;
    m = q;
  }
  scale[g] = scale_pack(m, rho);
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

// Pass B through the global dictionary and global atomics only.
template <int BLOCK, bool RAW>
__global__ __launch_bounds__(BLOCK) void k_pass_b_global(EventsDev ev, uint32_t A, uint32_t P,
                                                         const uint64_t* __restrict__ scale, GroupTables gt,
                                                         uint32_t* __restrict__ err) {
  const uint64_t n = ev.n;
  bool bad = false;
  for (uint64_t i = (uint64_t)blockIdx.x * BLOCK + threadIdx.x; i < n; i += (uint64_t)gridDim.x * BLOCK) {
    const uint32_t k = ev.key[i], a = ev.app[i], ph = ev.phase[i];
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
// Pass B with a per-workgroup LDS hash table: slot s holds a key tag and, per
// phase, a two-word accumulator.  Keys that cannot be placed within MAXPROBE
// probes (or the reserved tag value) go straight to the global tables.  At the
// end each workgroup adds its table into the global tables.
template <int BLOCK, bool RAW>
__global__ __launch_bounds__(BLOCK) void k_pass_b_lds(EventsDev ev, uint32_t A, uint32_t P,
                                                      const uint64_t* __restrict__ scale, GroupTables gt,
                                                      uint32_t slots_log2, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  const uint32_t S = 1u << slots_log2, SP = S * P;
  unsigned long long* s_lo = smem;
  unsigned long long* s_hi = smem + SP;
  unsigned long long* r_lo = smem + 2 * SP;               // RAW only
  unsigned long long* r_hi = smem + 3 * SP;               // RAW only
  uint32_t* s_tag = (uint32_t*)(smem + (RAW ? 4 : 2) * SP);
  for (uint32_t i = threadIdx.x; i < SP; i += BLOCK) {
    s_lo[i] = 0;
    s_hi[i] = 0;
    if (RAW) { r_lo[i] = 0; r_hi[i] = 0; }
  }
  for (uint32_t i = threadIdx.x; i < S; i += BLOCK) s_tag[i] = ATREX_EMPTY_KEY;
  __syncthreads();
  const uint32_t mask = S - 1;
  const uint32_t shift = 32 - slots_log2;
  constexpr uint32_t MAXPROBE = 64;
  const uint64_t n = ev.n, n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * BLOCK;
  bool bad = false;
  auto one = [&](uint32_t k, uint32_t a, uint32_t ph, int64_t d) {
    const bool ok = a < A && ph < P && d >= 0;
    bad |= !ok;
    if (!ok) return;
    const u128 v = event_share((uint64_t)d, scale[(size_t)a * P + ph]);
    int32_t slot = -1;
    if (k != ATREX_EMPTY_KEY) {
      uint32_t h = (hash32(k) >> shift) & mask;  // slots_log2 >= 1
      for (uint32_t probe = 0; probe < MAXPROBE; ++probe) {
        uint32_t t = s_tag[h];
        if (t == ATREX_EMPTY_KEY) t = atomicCAS(&s_tag[h], ATREX_EMPTY_KEY, k);
        if (t == k || t == ATREX_EMPTY_KEY) {
          slot = (int32_t)h;
          break;
        }
        h = (h + 1) & mask;
      }
    }
    if (slot >= 0) {
      const uint32_t gi = (uint32_t)slot * P + ph;
      acc_add(&s_lo[gi], &s_hi[gi], v);
      if (RAW) acc_add_plain(&r_lo[gi], &r_hi[gi], (u128)(uint64_t)d);
    } else {
      global_accumulate<RAW>(gt, P, k, ph, (uint64_t)d, v, err);
    }
  };
  for (uint64_t q = (uint64_t)blockIdx.x * BLOCK + threadIdx.x; q < n4; q += stride) {
    Ev4 e;
    load4<true>(ev.key, ev.app, ev.phase, ev.dur, q * 4, e);
#pragma unroll
    for (int j = 0; j < 4; ++j) one(e.key[j], e.app[j], e.ph[j], e.dur[j]);
  }
  if (blockIdx.x == 0)
    for (uint64_t i = n4 * 4 + threadIdx.x; i < n; i += BLOCK) one(ev.key[i], ev.app[i], ev.phase[i], ev.dur[i]);
  flag_error(err, bad, ATREX_ERRBIT_RANGE);
  __syncthreads();
  // merge this workgroup's table into the global tables
  for (uint32_t s = threadIdx.x; s < S; s += BLOCK) {
    const uint32_t k = s_tag[s];
    if (k == ATREX_EMPTY_KEY) continue;
    const int64_t j = dict_slot(gt.dict, gt.dict_mask, k, err);
    if (j < 0) continue;
    for (uint32_t ph = 0; ph < P; ++ph) {
      const uint32_t li = s * P + ph;
      const unsigned long long hi = s_hi[li], lo = s_lo[li];
      if ((hi >> ATREX_COUNT_SHIFT) == 0) continue;  // no invocation in this phase
      const size_t gi = (size_t)j * P + ph;
      const unsigned long long old = atomicAdd(&gt.acc[2 * gi], lo);
      atomicAdd(&gt.acc[2 * gi + 1], hi + ((old + lo < old) ? 1ull : 0ull));
      if (RAW) acc_add_plain(&gt.raw[2 * gi], &gt.raw[2 * gi + 1], make_u128(r_lo[li], r_hi[li]));
    }
  }
}

// ---------------------------------------------------------------------------
// Compaction: every (dictionary slot, phase) with at least one invocation
// becomes a group row (sort key = key << 3 | phase, source index).
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_compact(GroupTables gt, uint32_t P, uint64_t max_groups,
                                                   uint64_t* __restrict__ sk, uint32_t* __restrict__ src,
                                                   unsigned long long* __restrict__ counter,
                                                   uint32_t* __restrict__ err) {
  __shared__ uint32_t s_base;
  __shared__ uint32_t s_wcnt[BLOCK / 64];
  const uint64_t total = (uint64_t)(gt.dict_mask + 1) * P;
  for (uint64_t base = (uint64_t)blockIdx.x * BLOCK; base < total; base += (uint64_t)gridDim.x * BLOCK) {
    const uint64_t gi = base + threadIdx.x;
    bool live = false;
    uint32_t key = 0;
    if (gi < total) {
      const uint64_t j = gi / P;
      const unsigned long long tag = gt.dict[j];
      live = tag != 0 && (gt.acc[2 * gi + 1] >> ATREX_COUNT_SHIFT) != 0;
      key = (uint32_t)(tag - 1);
    }
    const uint64_t bal = __ballot(live);
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t before = __popcll(bal & ((1ull << lane) - 1));
    if (lane == 0) s_wcnt[wave] = __popcll(bal);
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t tot = 0;
      for (int w = 0; w < BLOCK / 64; ++w) {
        const uint32_t c = s_wcnt[w];
        s_wcnt[w] = tot;
        tot += c;
      }
      s_base = tot ? (uint32_t)atomicAdd(counter, (unsigned long long)tot) : 0;
    }
    __syncthreads();
    if (live) {
      const uint64_t pos = (uint64_t)s_base + s_wcnt[wave] + before;
      if (pos < max_groups) {
        sk[pos] = ((uint64_t)key << 3) | (uint64_t)(gi % P);
        src[pos] = (uint32_t)gi;
      } else {
        atomicOr(err, ATREX_ERRBIT_CAPACITY);
      }
    }
    __syncthreads();
  }
}

// Sorted rows -> group arrays.
__global__ void k_gather_groups(const uint64_t* __restrict__ sk, const uint32_t* __restrict__ src, uint64_t G,
                                GroupTables gt, bool raw, SortedGroups out) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= G) return;
  const uint64_t gi = src[i];
  const uint64_t hi = gt.acc[2 * gi + 1];
  out.key[i] = (uint32_t)(sk[i] >> 3);
  out.phase[i] = (uint8_t)(sk[i] & 7);
  out.count[i] = hi >> ATREX_COUNT_SHIFT;
  out.wsum[2 * i] = gt.acc[2 * gi];
  out.wsum[2 * i + 1] = hi & ((1ull << ATREX_COUNT_SHIFT) - 1);
  if (raw) {
    out.raw[2 * i] = gt.raw[2 * gi];
    out.raw[2 * i + 1] = gt.raw[2 * gi + 1];
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

}  // namespace

// ---------------------------------------------------------------------------
// Host launchers
void launch_unpack_scale(hipStream_t s, const uint64_t* sw, uint64_t G, uint64_t* mant, int32_t* rho) {
  if (G) hipLaunchKernelGGL(k_unpack_scale, dim3((uint32_t)((G + 255) / 256)), dim3(256), 0, s, sw, G, mant, rho);
}

void launch_pass_a_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                       unsigned long long* partial, unsigned long long* carry, uint32_t* err) {
  const uint32_t G = A * P;
  const size_t smem = (size_t)G * 8;
  hipLaunchKernelGGL((k_pass_a_lds<512>), dim3(nblocks), dim3(512), smem, s, ev, A, P, G, partial, carry, err);
}

void launch_pass_a_reduce(hipStream_t s, const unsigned long long* partial, uint32_t nb, uint32_t G,
                          const unsigned long long* carry, uint64_t* T) {
  hipLaunchKernelGGL(k_pass_a_reduce, dim3((G + 255) / 256), dim3(256), 0, s, partial, nb, G, carry, T);
}

void launch_pass_a_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                          unsigned long long* T, uint32_t* err) {
  hipLaunchKernelGGL((k_pass_a_global<256>), dim3(nblocks), dim3(256), 0, s, ev, A, P, T, err);
}

void launch_scale(hipStream_t s, const uint64_t* T, const uint32_t* c, const uint64_t* Csum, uint32_t A,
                  uint32_t P, uint64_t* scale) {
  const uint32_t G = A * P;
  hipLaunchKernelGGL(k_scale, dim3((G + 255) / 256), dim3(256), 0, s, T, c, Csum, A, P, scale);
}

void launch_pass_b_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                          const GroupTables& gt, bool raw, uint32_t nblocks, uint32_t* err) {
  if (raw)
    hipLaunchKernelGGL((k_pass_b_global<256, true>), dim3(nblocks), dim3(256), 0, s, ev, A, P, scale, gt, err);
  else
    hipLaunchKernelGGL((k_pass_b_global<256, false>), dim3(nblocks), dim3(256), 0, s, ev, A, P, scale, gt, err);
}

size_t pass_b_lds_smem(uint32_t P, bool raw, uint32_t slots_log2) {
  const size_t S = (size_t)1 << slots_log2;
  return S * P * 8 * (raw ? 4 : 2) + S * 4;
}

void launch_pass_b_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                       const GroupTables& gt, bool raw, uint32_t slots_log2, uint32_t nblocks, uint32_t* err) {
  const size_t smem = pass_b_lds_smem(P, raw, slots_log2);
  if (raw)
    hipLaunchKernelGGL((k_pass_b_lds<1024, true>), dim3(nblocks), dim3(1024), smem, s, ev, A, P, scale, gt,
                       slots_log2, err);
  else
    hipLaunchKernelGGL((k_pass_b_lds<1024, false>), dim3(nblocks), dim3(1024), smem, s, ev, A, P, scale, gt,
                       slots_log2, err);
}

void launch_compact(hipStream_t s, const GroupTables& gt, uint32_t P, uint64_t max_groups, uint64_t* sk,
                    uint32_t* src, unsigned long long* counter, uint32_t* err) {
  const uint64_t total = (uint64_t)(gt.dict_mask + 1) * P;
  uint64_t nb = (total + 255) / 256;
  if (nb > 4096) nb = 4096;
  hipLaunchKernelGGL((k_compact<256>), dim3((uint32_t)nb), dim3(256), 0, s, gt, P, max_groups, sk, src, counter,
                     err);
}

void launch_gather_groups(hipStream_t s, const uint64_t* sk, const uint32_t* src, uint64_t G, const GroupTables& gt,
                          bool raw, const SortedGroups& out) {
  if (G == 0) return;
  hipLaunchKernelGGL(k_gather_groups, dim3((uint32_t)((G + 255) / 256)), dim3(256), 0, s, sk, src, G, gt, raw, out);
}

hipError_t set_kernel_smem_limits() {
  hipError_t e = hipFuncSetAttribute((const void*)k_pass_a_lds<512>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     160 * 1024);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)k_pass_b_lds<1024, true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                          160 * 1024);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void*)k_pass_b_lds<1024, false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             160 * 1024);
}
