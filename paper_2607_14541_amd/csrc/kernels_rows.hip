// kernels_rows.hip -- group rows and the radix-partition engine (gfx950).
//
// Every pass-B engine emits rows (sort key = key << 3 | phase, two-word
// accumulator X = W + count * 2^97, optional raw time); a radix sort on the
// sort key and a segmented sum turn the rows into the ordered groups.
//
//  * owner merge: the LDS engine leaves, per workgroup, its table split into
//    256 owner regions (owner = top byte of an invertible hash of the key);
//    one workgroup per owner sums the regions in an LDS table and writes a
//    sorted list; the lists are put in global order by ranking each row in
//    every list (no sort), or become rows when that cannot be done.
//  * radix-partition engine (high key cardinality, and the LDS engine's
//    spilled events): per-workgroup bucket histograms of the top BB bits of the
//    key hash, one scan, a scatter of 16-byte records (Q96 share, phase, the
//    low 32 - BB hash bits), then per bucket chunk an LDS group-by that emits
//    rows; the key is recovered by inverting the hash.
#include <algorithm>

#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t MAXPROBE_R = 32;
constexpr uint32_t EMPTY_TAG = 0xFFFFFFFFu;

// Inverse of hash32 (atrex_device.hpp, the "lowbias32" mixer of C. Wellons'
// hash-prospector): its rounds undone in reverse order.  x ^= x >> 16 is its
// own inverse on 32 bits; x ^= x >> 15 is undone by x ^= (x >> 15) ^ (x >> 30);
// each multiplier is replaced by its inverse modulo 2^32 (checked: the
// products 0x846ca68b * 0x43021123 and 0x7feb352d * 0x1d69e2a5 are 1 mod 2^32).
__device__ __forceinline__ uint32_t unmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x43021123u;  // inverse of 0x846ca68b mod 2^32
  h ^= (h >> 15) ^ (h >> 30);
  h *= 0x1d69e2a5u;  // inverse of 0x7feb352d mod 2^32
  h ^= h >> 16;
  return h;
}

__device__ __forceinline__ uint32_t lane_of() { return threadIdx.x & 63; }

// Wave-aggregated append of one row per lane with `want` set.
__device__ __forceinline__ void row_append(const Rows& R, bool want, uint64_t rk, uint64_t lo, uint64_t hi,
                                           uint64_t rlo, uint64_t rhi, uint32_t* err) {
  const uint64_t bm = __ballot(want);
  if (bm == 0) return;
  const uint32_t leader = __ffsll((unsigned long long)bm) - 1;
  unsigned long long base = 0;
  if (lane_of() == leader) base = atomicAdd(R.count, (unsigned long long)__popcll(bm));
  base = __shfl(base, leader, 64);
  if (!want) return;
  const uint64_t pos = base + __popcll(bm & ((1ull << lane_of()) - 1ull));
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

// Add a two-word accumulator value (lo, hi) into LDS words with carry.
__device__ __forceinline__ void lds_add2(unsigned long long* plo, unsigned long long* phi, uint64_t lo, uint64_t hi) {
  const unsigned long long old = atomicAdd(plo, (unsigned long long)lo);
  const unsigned long long c = (old + lo < old) ? 1ull : 0ull;
  if (hi + c) atomicAdd(phi, (unsigned long long)(hi + c));
}

// LDS group table shared by the owner merge and the bucket aggregation:
// S slots of (tag, P two-word accumulators [, P raw accumulators]).
template <bool RAW>
struct LdsTable {
  unsigned long long *lo, *hi, *rlo, *rhi;
  uint32_t* tag;
  uint32_t S, P;
  __device__ void init(unsigned long long* smem, uint32_t S_, uint32_t P_) {
    S = S_;
    P = P_;
    const uint32_t SP = S * P;
    lo = smem;
    hi = smem + SP;
    rlo = smem + 2 * SP;
    rhi = smem + 3 * SP;
    tag = (uint32_t*)(smem + (RAW ? 4 : 2) * SP);
  }
  __device__ void clear() {
    const uint32_t SP = S * P;
    for (uint32_t i = threadIdx.x; i < SP; i += blockDim.x) {
      lo[i] = 0;
      hi[i] = 0;
      if (RAW) { rlo[i] = 0; rhi[i] = 0; }
    }
    for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) tag[i] = EMPTY_TAG;
  }
  // slot of tag t (t != EMPTY_TAG), or -1 when not placed within the probe limit
  __device__ int32_t slot(uint32_t t) {
    if (t == EMPTY_TAG) return -1;  // the free-slot marker is never a tag
    uint32_t h = __umulhi(t * 0x9E3779B1u, S);
#pragma unroll 1
    for (uint32_t probe = 0; probe < MAXPROBE_R; ++probe) {
      uint32_t cur = tag[h];
      if (cur == EMPTY_TAG) cur = atomicCAS(&tag[h], EMPTY_TAG, t);
      if (cur == t || cur == EMPTY_TAG) return (int32_t)h;
      h = (h + 1 == S) ? 0 : h + 1;
    }
    return -1;
  }
};

// ---------------------------------------------------------------- owner lists
// One workgroup per owner: sum the owner's regions (and, when the spill total
// is at most sp.inline_max, the spill records whose key belongs to this owner)
// in a small LDS table, then sort the owner's (key, phase) rows in LDS and
// write them as a list with the per-phase partial sums of W.  Keys the table
// cannot place go to the row list.
constexpr uint32_t MAXPROBE_O = 64;
constexpr uint32_t kRegionMap = 24 * 1024;  // records per owner mapped to their region by a byte table

__device__ __forceinline__ uint32_t owner_of(uint32_t key) { return hash32(key) >> 24; }

// Exclusive prefix of n <= 256 values into pre[0..n] (pre[n] = total): thread
// t < n passes its value v (its own load, so all loads are in flight at
// once), every thread of the workgroup calls; ends with a barrier.
__device__ __forceinline__ void prefix256(uint32_t n, uint32_t v, uint32_t* pre, uint32_t* s_w4) {
  const uint32_t t = threadIdx.x, lane = t & 63, w = t >> 6;
  const uint32_t x = t < n ? v : 0u;
  uint32_t inc = x;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d, 64);
    if (lane >= (uint32_t)d) inc += y;
  }
  if (w < 4 && lane == 63) s_w4[w] = inc;
  __syncthreads();
  if (t < 256) {
    uint32_t off = 0;
    for (uint32_t q = 0; q < w; ++q) off += s_w4[q];
    if (t < n) pre[t] = off + inc - x;
    if (t == 255) pre[n] = off + inc;
  }
  __syncthreads();
}

// last w with pre[w] <= idx (pre ascending, pre[0] = 0, idx < pre[n])
__device__ __forceinline__ uint32_t upper_index(const uint32_t* pre, uint32_t n, uint32_t idx) {
  uint32_t lo = 0, hi = n;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (pre[mid] <= idx) lo = mid; else hi = mid;
  }
  return lo;
}

template <bool RAW>
__global__ __launch_bounds__(1024) void k_owner_finish(OwnerRegions orr, uint32_t nwg, uint32_t P, uint32_t So,
                                                       SpillIn sp, OwnerLists ol, Rows rows,
                                                       uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  __shared__ uint32_t s_pre[257], s_spre[257], s_w4[4];
  __shared__ uint32_t s_cnt, s_dbase;
  __shared__ unsigned long long s_plo[16], s_phi[16];
  const uint32_t SoP = So * P;
  unsigned long long* acc = smem;                    // [So * P] x (lo, hi)
  unsigned long long* racc = smem + 2 * SoP;         // RAW only
  uint64_t* skey = (uint64_t*)(smem + (RAW ? 4 : 2) * SoP);  // [pow2 >= So * P] sort keys
  uint32_t SoP2 = 1;
  while (SoP2 < SoP) SoP2 <<= 1;
  uint32_t* tag = (uint32_t*)(skey + SoP2);          // [So]
  uint8_t* s_wid = (uint8_t*)(tag + So);             // [kRegionMap] region (workgroup) of each record
  const uint32_t o = blockIdx.x, tid = threadIdx.x;
  // region sizes and spill-region sizes, loaded together (nwg, sp.nwg <= 256)
  // while the table is cleared
  const uint32_t rc = tid < nwg ? orr.count[(size_t)tid * ATREX_OWNERS + o] : 0u;
  const uint32_t sc = tid < sp.nwg ? sp.count[tid] : 0u;
  for (uint32_t i = tid; i < 2 * SoP; i += 1024) {
    acc[i] = 0;
    if (RAW) racc[i] = 0;
  }
  for (uint32_t i = tid; i < So; i += 1024) tag[i] = EMPTY_TAG;
  if (tid < 16) { s_plo[tid] = 0; s_phi[tid] = 0; }
  if (tid == 0) s_cnt = 0;
  prefix256(nwg, rc, s_pre, s_w4);
  prefix256(sp.nwg, sc, s_spre, s_w4);
  const uint32_t total = s_pre[nwg];
  const bool mapped = total <= kRegionMap;  // record -> region by table, else by binary search
  if (mapped && tid < nwg)
    for (uint32_t r = s_pre[tid]; r < s_pre[tid + 1]; ++r) s_wid[r] = (uint8_t)tid;
  __syncthreads();
  auto slot_of = [&](uint32_t key) -> int32_t {
    if (key == EMPTY_TAG) return -1;  // the free-slot marker is never a tag
    uint32_t h = hash32(key) & (So - 1);
#pragma unroll 1
    for (uint32_t probe = 0; probe < MAXPROBE_O; ++probe) {
      uint32_t cur = tag[h];
      if (cur == EMPTY_TAG) cur = atomicCAS(&tag[h], EMPTY_TAG, key);
      if (cur == key || cur == EMPTY_TAG) return (int32_t)h;
      h = (h + 1) & (So - 1);
    }
    return -1;
  };
  // the owner's regions, one (record, phase) item per thread and round: the
  // loads of a round's K items are issued before any is used
  constexpr int K = RAW ? 8 : 16;
  const uint32_t items = total * P;
  for (uint32_t base = 0; base < items; base += K * 1024) {  // uniform trip count (row_append)
    uint32_t key[K];
    uint64_t lo[K], hi[K], rl[K], rh[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const uint32_t it = base + (uint32_t)k * 1024 + tid;
      key[k] = EMPTY_TAG;
      lo[k] = hi[k] = rl[k] = rh[k] = 0;
      if (it < items) {
        const uint32_t idx = it / P, ph = it - idx * P;
        const uint32_t w = mapped ? s_wid[idx] : upper_index(s_pre, nwg, idx);
        const size_t rec = ((size_t)w * ATREX_OWNERS + o) * orr.capo + (idx - s_pre[w]);
        key[k] = orr.key[rec];
        lo[k] = orr.acc[(rec * P + ph) * 2];
        hi[k] = orr.acc[(rec * P + ph) * 2 + 1];
        if (RAW) { rl[k] = orr.raw[(rec * P + ph) * 2]; rh[k] = orr.raw[(rec * P + ph) * 2 + 1]; }
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const uint32_t it = base + (uint32_t)k * 1024 + tid;
      const uint32_t ph = it % P;
      const bool present = it < items && (hi[k] >> ATREX_COUNT_SHIFT) != 0;
      const int32_t sl = present ? slot_of(key[k]) : -1;
      if (present && sl >= 0) {
        lds_add2(&acc[2 * (sl * P + ph)], &acc[2 * (sl * P + ph) + 1], lo[k], hi[k]);
        if (RAW) lds_add2(&racc[2 * (sl * P + ph)], &racc[2 * (sl * P + ph) + 1], rl[k], rh[k]);
      }
      row_append(rows, present && sl < 0, ((uint64_t)key[k] << 3) | ph, lo[k], hi[k], rl[k], rh[k], err);
    }
  }
  // the spill records of this owner, when they are few
  const uint32_t stotal = s_spre[sp.nwg];
  if (stotal <= sp.inline_max) {
    for (uint32_t base = 0; base < stotal; base += 1024) {
      const uint32_t idx = base + tid;
      bool mine = false;
      uint32_t key = 0, ph = 0;
      uint64_t lo = 0, hi = 0, d = 0;
      int32_t sl = -1;
      if (idx < stotal) {
        const uint32_t w = upper_index(s_spre, sp.nwg, idx);
        const size_t r = (size_t)w * sp.cap + (idx - s_spre[w]);
        key = sp.key[r];
        mine = owner_of(key) == o;
        if (mine) {
          lo = sp.val[2 * r];
          const uint64_t w1 = sp.val[2 * r + 1];
          hi = (w1 & (((uint64_t)1 << 40) - 1)) + ((uint64_t)1 << ATREX_COUNT_SHIFT);
          ph = (uint32_t)(w1 >> 40);
          if (RAW) d = sp.raw[r];
          sl = slot_of(key);
          if (sl >= 0) {
            lds_add2(&acc[2 * (sl * P + ph)], &acc[2 * (sl * P + ph) + 1], lo, hi);
            if (RAW) lds_add2(&racc[2 * (sl * P + ph)], &racc[2 * (sl * P + ph) + 1], d, 0);
          }
        }
      }
      row_append(rows, mine && sl < 0, ((uint64_t)key << 3) | ph, lo, hi, d, 0, err);
    }
  }
  __syncthreads();
  // present (slot, phase) pairs -> sort keys rk << 20 | (slot * P + phase)
  for (uint32_t i = tid; i < SoP; i += 1024) {
    const uint32_t t = tag[i / P];
    if (t != EMPTY_TAG && (acc[2 * i + 1] >> ATREX_COUNT_SHIFT) != 0) {
      const uint32_t at = atomicAdd(&s_cnt, 1u);
      skey[at] = ((((uint64_t)t << 3) | (i % P)) << 20) | i;
    }
  }
  __syncthreads();
  const uint32_t cnt = s_cnt;
  if (cnt <= 64) {  // ascending bitonic sort in one wave's registers
    if (tid < 64) {
      uint64_t v = tid < cnt ? skey[tid] : ~0ull;
      for (uint32_t k = 2; k <= 64; k <<= 1)
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
          const uint64_t w = __shfl_xor((unsigned long long)v, (int)j, 64);
          const bool up = (tid & k) == 0, lower = (tid & j) == 0;
          v = (lower == up) ? (v < w ? v : w) : (v < w ? w : v);
        }
      if (tid < cnt) skey[tid] = v;
    }
    __syncthreads();
  } else {
    uint32_t N = 1;
    while (N < cnt) N <<= 1;
    for (uint32_t i = cnt + tid; i < N; i += 1024) skey[i] = ~0ull;
    __syncthreads();
    for (uint32_t k = 2; k <= N; k <<= 1)  // ascending bitonic sort in LDS, N <= So * P
      for (uint32_t j = k >> 1; j > 0; j >>= 1) {
        for (uint32_t i = tid; i < N; i += 1024) {
          const uint32_t q = i ^ j;
          if (q > i) {
            const uint64_t x = skey[i], y = skey[q];
            if ((x > y) == ((i & k) == 0)) { skey[i] = y; skey[q] = x; }
          }
        }
        __syncthreads();
      }
  }
  // the list, its keys in the dense key array, and the per-phase partial sums of W
  if (tid == 0) s_dbase = cnt ? (uint32_t)atomicAdd(ol.dcount, (unsigned long long)cnt) : 0u;
  __syncthreads();
  const size_t base = (size_t)o * ol.cap, dbase = s_dbase;
  for (uint32_t i = tid; i < cnt; i += 1024) {
    const uint64_t sk = skey[i];
    const uint32_t e = (uint32_t)(sk & 0xFFFFF);
    const uint64_t lo = acc[2 * e], hi = acc[2 * e + 1];
    ol.rk[base + i] = sk >> 20;
    ol.dkey[dbase + i] = (uint32_t)(sk >> 23);
    ol.lo[base + i] = lo;
    ol.hi[base + i] = hi;
    if (RAW) { ol.rlo[base + i] = racc[2 * e]; ol.rhi[base + i] = racc[2 * e + 1]; }
    const uint32_t ph = e % P;
    const unsigned long long wh = hi & (((uint64_t)1 << ATREX_COUNT_SHIFT) - 1);
    const unsigned long long old = atomicAdd(&s_plo[ph], (unsigned long long)lo);
    atomicAdd(&s_phi[ph], wh + ((old + lo < old) ? 1ull : 0ull));
  }
  __syncthreads();
  if (tid < P) {
    ol.part[((size_t)o * P + tid) * 2] = s_plo[tid];
    ol.part[((size_t)o * P + tid) * 2 + 1] = s_phi[tid];
  }
  if (tid == 0) ol.count[o] = cnt;
}

// Global order of the owner lists' rows.  A key's rows all sit in one list,
// adjacent and ordered by phase, so a row's position is the number of rows
// with a smaller key (over all lists) plus its place among its key's rows.
// Each owner's workgroup stages every row key (the dense key array the owner
// merge appends to) in LDS and counts, for each of its distinct keys, the
// smaller ones: wave ballots, no search.  Done only when no row went to the
// row list, the spill records were merged and the rows fit in LDS (kRankMax,
// fewer when the owner lists are long); workgroup 0 also writes S[ph].
__global__ __launch_bounds__(1024) void k_rank_groups(OwnerLists ol, uint32_t P, SpillIn sp, Rows rows,
                                                      const uint32_t* __restrict__ err, SortedGroups out,
                                                      uint64_t* __restrict__ S_out, unsigned long long* __restrict__ G_out,
                                                      uint32_t* __restrict__ done, uint32_t rmax) {
  extern __shared__ unsigned long long smem[];
  __shared__ uint32_t s_w4[4], s_nh, s_stot, s_wc[16 * 16];
  __shared__ unsigned long long s_plo[8], s_phi[8];
  uint32_t* s_key = (uint32_t*)smem;              // [rmax <= kRankMax] every row key
  uint32_t* s_own = s_key + rmax;                 // [ol.cap] this owner's row keys
  uint32_t* s_pos = s_own + ol.cap;               // [ol.cap] positions of this owner's key heads (by row)
  uint32_t* s_head = s_pos + ol.cap;              // [ol.cap] this owner's key heads (rows)
  uint32_t* s_hkey = s_head + ol.cap;             // [ol.cap] their keys
  const uint32_t o = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  // sizes and status words, loaded together
  const uint32_t co = ol.count[o];
  const uint32_t R = (uint32_t)*ol.dcount;
  const uint32_t sc = tid < sp.nwg ? sp.count[tid] : 0u;
  const unsigned long long nrows = *rows.count;
  const uint32_t e0 = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid < 8) { s_plo[tid] = 0; s_phi[tid] = 0; }
  if (tid == 0) { s_nh = 0; s_stot = 0; }
  __syncthreads();
  {
    uint32_t t = sc;
    for (int d = 32; d >= 1; d >>= 1) t += __shfl_xor(t, d, 64);
    if (lane == 0 && t) atomicAdd(&s_stot, t);
  }
  __syncthreads();
  const uint32_t stot = s_stot;
  const bool ok = nrows == 0 && stot <= sp.inline_max && R <= rmax &&
                  (e0 & (ATREX_ERRBIT_RANGE | ATREX_ERRBIT_CAPACITY | ATREX_ERRBIT_SPILL)) == 0;
  if (o == 0 && tid == 0) G_out[2] = stot;  // spill records, for the host's fallback
  if (!ok) {
    if (o == 0 && tid == 0) *done = 0;
    return;
  }
  // every row key and this owner's row keys into LDS: loads first
  constexpr int K = kRankMax / 1024;
  uint32_t v[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const uint32_t idx = (uint32_t)k * 1024 + tid;
    v[k] = idx < R ? ol.dkey[idx] : 0u;
  }
  const size_t base = (size_t)o * ol.cap;
  for (uint32_t i = tid; i < co; i += 1024) s_own[i] = (uint32_t)(ol.rk[base + i] >> 3);
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const uint32_t idx = (uint32_t)k * 1024 + tid;
    if (idx < R) s_key[idx] = v[k];
  }
  // workgroup 0: S[ph] from the owners' partial sums, one (owner, phase) per thread
  if (o == 0) {
    for (uint32_t q = tid; q < ATREX_OWNERS * P; q += 1024) {
      const uint64_t lo = ol.part[2 * (size_t)q], hi = ol.part[2 * (size_t)q + 1];
      const uint32_t ph = q % P;
      const unsigned long long old = atomicAdd(&s_plo[ph], (unsigned long long)lo);
      atomicAdd(&s_phi[ph], (unsigned long long)hi + ((old + lo < old) ? 1ull : 0ull));
    }
  }
  __syncthreads();
  // this owner's distinct keys (first row of each key) and each row's head
  for (uint32_t i = tid; i < co; i += 1024) {
    const uint32_t k = s_own[i];
    if (i == 0 || s_own[i - 1] != k) {
      const uint32_t h = atomicAdd(&s_nh, 1u);
      s_hkey[h] = k;
      s_head[h] = i;
    }
  }
  // this wave's share of the staged keys, in registers
  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint32_t y[K];
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const uint32_t idx = (uint32_t)k * 1024 + wave * 64 + lane;
    y[k] = idx < R ? s_key[idx] : 0xFFFFFFFFu;
  }
  __syncthreads();
  // rows with a smaller key, HB heads at a time: each wave counts its keys
  // below each head's key with ballots; the 16 waves' counts are summed
  constexpr int HB = 16;
  const uint32_t nh = s_nh;
  for (uint32_t h0 = 0; h0 < nh; h0 += HB) {
    uint32_t xk[HB];
#pragma unroll
    for (int j = 0; j < HB; ++j) xk[j] = s_hkey[min(h0 + (uint32_t)j, nh - 1)];
#pragma unroll
    for (int j = 0; j < HB; ++j) {
      uint32_t c = 0;
#pragma unroll
      for (int k = 0; k < K; ++k) c += (uint32_t)__popcll(__ballot(y[k] < xk[j]));
      if (lane == 0) s_wc[wave * HB + j] = c;
    }
    __syncthreads();
    if (tid < HB && h0 + tid < nh) {
      uint32_t c = 0;
      for (uint32_t w = 0; w < 16; ++w) c += s_wc[w * HB + tid];
      s_pos[s_head[h0 + tid]] = c;
    }
    __syncthreads();
  }
  // a row's position: its key's count plus its place among its key's rows
  for (uint32_t i = tid; i < co; i += 1024) {
    uint32_t hb = i;  // the key's first row: at most P - 1 rows back
    while (hb > 0 && s_own[hb - 1] == s_own[i]) --hb;
    const uint32_t g = s_pos[hb] + (i - hb);
    const uint64_t rk = ol.rk[base + i];
    const uint64_t hi = ol.hi[base + i];
    out.key[g] = (uint32_t)(rk >> 3);
    out.phase[g] = (uint8_t)(rk & 7);
    out.count[g] = hi >> ATREX_COUNT_SHIFT;
    out.wsum[2 * g] = ol.lo[base + i];
    out.wsum[2 * g + 1] = hi & (((uint64_t)1 << ATREX_COUNT_SHIFT) - 1);
    if (out.raw) {
      out.raw[2 * g] = ol.rlo[base + i];
      out.raw[2 * g + 1] = ol.rhi[base + i];
    }
  }
  if (o == 0 && tid < P) {
    S_out[2 * tid] = s_plo[tid];
    S_out[2 * tid + 1] = s_phi[tid];
  }
  if (o == 0 && tid == 0) {
    *G_out = R;
    *done = 1;
  }
}

// The owner lists appended to the row list (when the ranking is not done).
__global__ void k_lists_to_rows(OwnerLists ol, Rows rows, uint32_t* __restrict__ err) {
  const uint32_t o = blockIdx.x;
  const uint32_t c = ol.count[o];
  const size_t base = (size_t)o * ol.cap;
  for (uint32_t i0 = 0; i0 < c; i0 += blockDim.x) {  // uniform trip count (row_append)
    const uint32_t i = i0 + threadIdx.x;
    const bool v = i < c;
    row_append(rows, v, v ? ol.rk[base + i] : 0, v ? ol.lo[base + i] : 0, v ? ol.hi[base + i] : 0,
               (v && ol.rlo) ? ol.rlo[base + i] : 0, (v && ol.rhi) ? ol.rhi[base + i] : 0, err);
  }
}

// ---------------------------------------------------------------- partition engine
__device__ __forceinline__ void part_range(const PartSource& src, uint32_t w, uint64_t& b, uint64_t& e) {
  if (src.spill) {
    b = (uint64_t)w * src.scap;
    e = b + src.scount[w];
  } else {
    b = (uint64_t)w * src.per;
    e = b + src.per;
    if (e > src.ev.n) e = src.ev.n;
    if (b > e) b = e;
  }
}

constexpr uint32_t kNoSlot = ATREX_NO_SLOT;

constexpr int HIST_DEPTH = 4;  // groups of four keys in flight per lane in k_part_hist

// HOT: only the events whose key is not in the seeded image `seed` of S
// slots are counted (those k_part_scatter_hot turns into records).
template <bool HOT>
__global__ __launch_bounds__(1024) void k_part_hist(PartSource src, uint32_t BB, uint32_t* __restrict__ H,
                                                    const uint32_t* __restrict__ seed, uint32_t S) {
  extern __shared__ uint32_t s_h[];
  const uint32_t NB = 1u << BB, w = blockIdx.x, nw = gridDim.x, sh = 32 - BB;
  uint32_t* s_img = s_h + NB;  // [S], HOT only (16-byte aligned: NB >= 4)
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_h[i] = 0;
  if (HOT)
    for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) s_img[i] = seed[i];
  __syncthreads();
  auto cold = [&](uint32_t k) { return !HOT || image_slot(s_img, S, k) == kNoSlot; };
  uint64_t b, e;
  part_range(src, w, b, e);
  if (src.spill) {
    for (uint64_t i0 = b; i0 < e; i0 += blockDim.x) {  // uniform trip count
      const uint64_t i = i0 + threadIdx.x;
      const bool v = i < e;
      (void)count_in(s_h, v ? hash32(src.skey[i]) >> sh : 0, v);
    }
  } else {  // b is a multiple of 4: four keys per lane with one 16-byte load
    const uint64_t e4 = b + (e - b) / 4 * 4;
    // groups of four keys, iteration `it` covering groups it * blockDim.x +
    // [0, blockDim.x) (uniform trip count); a ring of HIST_DEPTH groups per
    // lane keeps that many loads in flight while one is counted
    const uint64_t ng = (e4 - b) / 4, iters = (ng + blockDim.x - 1) / blockDim.x;
    auto load = [&](uint64_t it, v4u& k) {
      const uint64_t gi = it * blockDim.x + threadIdx.x;
      if (gi < ng) k = __builtin_nontemporal_load((const v4u*)(src.ev.key + b + 4 * gi));
    };
    v4u ring[HIST_DEPTH];
#pragma unroll
    for (int d = 0; d < HIST_DEPTH; ++d) load(d, ring[d]);
    for (uint64_t it = 0; it < iters; it += HIST_DEPTH) {
#pragma unroll
      for (int d = 0; d < HIST_DEPTH; ++d) {
        if (it + d >= iters) break;
        const bool v = (it + d) * blockDim.x + threadIdx.x < ng;
        const v4u k = ring[d];
        if (it + d + HIST_DEPTH < iters) load(it + d + HIST_DEPTH, ring[d]);
        if (HOT) {  // the keys outside the image are spread over the buckets: plain atomics
          const uint32_t kv[4] = {k.x, k.y, k.z, k.w};
          bool c[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) c[j] = v && cold(kv[j]);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (c[j]) atomicAdd(&s_h[hash32(kv[j]) >> sh], 1u);
        } else {
          (void)count_in(s_h, hash32(k.x) >> sh, v);
          (void)count_in(s_h, hash32(k.y) >> sh, v);
          (void)count_in(s_h, hash32(k.z) >> sh, v);
          (void)count_in(s_h, hash32(k.w) >> sh, v);
        }
      }
    }
    for (uint64_t i = e4 + threadIdx.x; i < e; i += blockDim.x) {
      const uint32_t k = src.ev.key[i];
      if (cold(k)) atomicAdd(&s_h[hash32(k) >> sh], 1u);
    }
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) H[(size_t)i * nw + w] = s_h[i];
}

// Records: (share lo, share hi | phase << 33 | low hash bits << 36).  Each
// workgroup walks its event range in tiles of SC_TILE = 4 x 1024 events
// (eight events per thread need more than the 128 registers a 1024-thread
// workgroup allows).  Phase 1 takes every record's bucket and its rank among
// the tile's records of that bucket (an LDS counter) and requests its scale
// word; after a scan of the tile's bucket counts, phase 2 forms the Q96 share
// and places the record in LDS in bucket order; the tile is then written out
// as runs, consecutive lanes writing consecutive records of a bucket, while
// the next tile's events are loaded.

template <bool NO_APP>
__device__ __forceinline__ void load_group(const EventsDev& ev, uint64_t q, uint64_t e, Ev4& x) {
  if (q + 3 < e) {  // q is a multiple of 4: a whole, 16-byte aligned group
    load4<true, NO_APP>(ev.key, ev.app, ev.phase, ev.dur, q, x);
  } else {
    x.ph4 = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool in = q + j < e;
      x.key[j] = in ? ev.key[q + j] : 0;
      x.app[j] = in ? app_at<NO_APP>(ev.app, q + j) : 0;
      x.ph4 |= (in ? (uint32_t)ev.phase[q + j] : 0u) << (8 * j);
      x.dur[j] = in ? ev.dur[q + j] : 0;
    }
  }
}

// NO_APP: the events carry no application (every event is application 0).
template <bool RAW, bool SPILL, uint32_t SC_EPT, uint32_t SC_BLOCK, bool NO_APP = false>
__global__ __launch_bounds__(SC_BLOCK) void k_part_scatter(PartSource src, uint32_t A, uint32_t P,
                                                           const uint64_t* __restrict__ scale,
                                                           const uint64_t* __restrict__ bscale, uint32_t BB,
                                                           const uint32_t* __restrict__ O,
                                                           uint64_t* __restrict__ rec, uint64_t* __restrict__ rraw,
                                                           uint32_t* __restrict__ err) {
  extern __shared__ uint64_t sm64[];
  constexpr uint32_t NWV = SC_BLOCK / 64;
  constexpr uint32_t SC_TILE = SC_EPT * SC_BLOCK;
  const uint32_t NB = 1u << BB, w = blockIdx.x, nw = gridDim.x, tid = threadIdx.x;
  uint64_t* s_rec = sm64;                                  // [SC_TILE][2]
  uint64_t* s_raw = s_rec + 2 * SC_TILE;                   // [SC_TILE] RAW only
  uint16_t* s_bkt = (uint16_t*)(s_raw + (RAW ? SC_TILE : 0));  // [SC_TILE]
  uint32_t* s_cur = (uint32_t*)(s_bkt + SC_TILE);          // [NB] this workgroup's next record per bucket
  uint32_t* s_cnt = s_cur + NB;                            // [2][NB] records of the tile per bucket (by tile parity)
  uint32_t* s_off = s_cnt + 2 * NB;                        // [NB] tile offsets
  __shared__ uint32_t s_w[NWV];
  for (uint32_t i = tid; i < NB; i += SC_BLOCK) {
    s_cur[i] = O[(size_t)i * nw + w];
    s_cnt[i] = 0;
    s_cnt[NB + i] = 0;
  }
  uint64_t b, e;
  part_range(src, w, b, e);
  const uint32_t lowbits = 32 - BB;
  const uint64_t lowmask = ((uint64_t)1 << lowbits) - 1;
  bool bad = false;
  constexpr uint32_t G4 = SC_EPT / 4;  // groups of four events per thread, SC_BLOCK groups apart
  // the next tile's events are requested once the current tile's records are
  // placed in LDS, so that they arrive during its write-out
  Ev4 nxt[G4];
  if (!SPILL) {
#pragma unroll
    for (uint32_t g = 0; g < G4; ++g) load_group<NO_APP>(src.ev, b + 4 * ((uint64_t)g * SC_BLOCK + tid), e, nxt[g]);
  }
  // Four barriers per tile: the counters are double-buffered (the next
  // tile's are cleared during this tile's scan) and each bucket's position
  // moves on by the previous tile's count during the scan, so nothing follows
  // the write-out.
  constexpr uint32_t PERMAX = 4;  // buckets per thread in the scan (NB <= 4 * SC_BLOCK)
  const uint32_t per = (NB + SC_BLOCK - 1) / SC_BLOCK, b0 = tid * per;
  uint32_t prevcnt[PERMAX] = {0, 0, 0, 0};
  uint32_t parity = 0;
  __syncthreads();
  for (uint64_t t0 = b; t0 < e; t0 += SC_TILE, parity ^= 1u) {  // uniform trip count
    Ev4 evg[G4];
#pragma unroll
    for (uint32_t g = 0; g < G4; ++g) evg[g] = nxt[g];
    uint32_t* cnt = s_cnt + parity * NB;
    uint32_t* cnt_next = s_cnt + (parity ^ 1u) * NB;
    // phase 1: validity, bucket and rank of every record; the scale words
    // are requested here and used after the scan
    uint32_t hh[SC_EPT], rk[SC_EPT];  // hash; rank << 4 | exists << 3 | phase
    uint64_t dv[SC_EPT], sw[SC_EPT];
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j) {
      const uint64_t i = t0 + 4 * ((uint64_t)(j / 4) * SC_BLOCK + tid) + (j % 4);
      const bool vj = i < e;
      uint32_t key = 0;
      dv[j] = 0;
      sw[j] = 0;
      rk[j] = 0;
      if (SPILL) {
        key = vj ? src.skey[i] : 0;
      } else {
        const Ev4& ev = evg[j / 4];
        const uint32_t jj = j % 4;
        const uint32_t a = ev.app[jj], ph = ev.ph(jj);
        const int64_t dd = ev.dur[jj];
        const bool ok = a < A && ph < P && dd >= 0;
        bad |= vj && !ok;
        sw[j] = ok ? bscale[a * P + ph] : 0;
        dv[j] = ok ? (uint64_t)dd : 0;
        rk[j] = ok ? ph : 0u;
        key = ev.key[jj];
      }
      if (vj) rk[j] |= 8u;
      hh[j] = hash32(key);
    }
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j) rk[j] |= count_in(cnt, hh[j] >> lowbits, (rk[j] >> 3) & 1u) << 4;
    __syncthreads();
    // exclusive scan of the tile's bucket counts; the previous tile's counts
    // advance the positions, and the next tile's counters are cleared
    {
      uint32_t sum = 0;
#pragma unroll
      for (uint32_t k = 0; k < PERMAX; ++k) {
        if (k < per && b0 + k < NB) {
          const uint32_t c = cnt[b0 + k];
          s_cur[b0 + k] += prevcnt[k];
          prevcnt[k] = c;
          cnt_next[b0 + k] = 0;
          sum += c;
        }
      }
      const uint32_t lane = tid & 63, wave = tid >> 6;
      const uint32_t inc = wave_incl_scan_u32(sum);
      if (lane == 63) s_w[wave] = inc;
      __syncthreads();
      uint32_t off = 0;
      for (uint32_t x = 0; x < wave; ++x) off += s_w[x];
      uint32_t run = off + inc - sum;
#pragma unroll
      for (uint32_t k = 0; k < PERMAX; ++k)
        if (k < per && b0 + k < NB) { s_off[b0 + k] = run; run += prevcnt[k]; }
    }
    __syncthreads();
    // phase 2: the Q96 share of every record, placed in LDS in bucket order
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j) {
      if (!((rk[j] >> 3) & 1u)) continue;
      const uint32_t bk = hh[j] >> lowbits;
      uint64_t vl, vh, d = dv[j];
      uint32_t ph;
      if (SPILL) {
        const uint64_t i = t0 + 4 * ((uint64_t)(j / 4) * SC_BLOCK + tid) + (j % 4);
        vl = src.sval[2 * i];
        vh = src.sval[2 * i + 1] & (((uint64_t)1 << 40) - 1);
        ph = (uint32_t)(src.sval[2 * i + 1] >> 40);
        if (RAW) d = src.sraw[i];
      } else {
        ph = rk[j] & 7u;
        const uint64_t w = sw[j];
        if ((uint32_t)(w >> 56) <= 127u) {
          if ((d >> 32) == 0) {
            uint32_t h32;
            bscale_share32((uint32_t)d, (uint32_t)w, (uint32_t)(w >> 32), vl, h32);
            vh = h32;
          } else {
            bscale_share64(d, (uint32_t)w, (uint32_t)(w >> 32), vl, vh);
          }
        } else {  // rho outside [-8, 63] (rare): the general scale word, found again from the event
          const uint64_t i = t0 + 4 * ((uint64_t)(j / 4) * SC_BLOCK + tid) + (j % 4);
          const u128 x = event_share(d, scale[app_at<NO_APP>(src.ev.app, i) * P + ph]);
          vl = (uint64_t)x;
          vh = (uint64_t)(x >> 64);
        }
      }
      const uint32_t at = s_off[bk] + (rk[j] >> 4);
      s_rec[2 * at] = vl;
      s_rec[2 * at + 1] = vh | ((uint64_t)ph << 33) | (((uint64_t)hh[j] & lowmask) << 36);
      if (RAW) s_raw[at] = d;
      s_bkt[at] = (uint16_t)bk;
    }
    if (!SPILL && t0 + SC_TILE < e) {
#pragma unroll
      for (uint32_t g = 0; g < G4; ++g)
        load_group<NO_APP>(src.ev, t0 + SC_TILE + 4 * ((uint64_t)g * SC_BLOCK + tid), e, nxt[g]);
    }
    __syncthreads();
    const uint32_t nt = (uint32_t)min((uint64_t)SC_TILE, e - t0);
    for (uint32_t k = tid; k < nt; k += SC_BLOCK) {
      const uint32_t bb = s_bkt[k];
      const size_t pos = (size_t)s_cur[bb] + (k - s_off[bb]);
      v2l r;
      r.x = (long long)s_rec[2 * k];
      r.y = (long long)s_rec[2 * k + 1];
      *(v2l*)(rec + 2 * pos) = r;  // ordinary store: non-temporal ones ran ~1.5x slower on short runs
      if (RAW) rraw[pos] = s_raw[k];
    }
  }
  if (__any(bad) && (tid & 63) == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
}

// Pass B of a seeded table and the partition scatter in one pass over the
// events.  An event whose key is in the image `seed` (the sample's hottest
// keys, each in its own bucket; the same image in every workgroup) is
// added to this workgroup's LDS table of S slots x P two-word accumulators;
// every other event becomes a partition record, ranked, placed and written
// out in tiles as in k_part_scatter (k_part_hist<true> with the same image
// counts exactly these).  At the end the table goes to the owner regions as
// the LDS engine's does.  The table takes what LDS leaves beside the tile's
// staging, which holds 1 / STAGE_DIV (1 or 2) of a tile's records: a tile
// with more records is placed and written out in two rounds.
template <uint32_t SC_EPT, uint32_t SC_BLOCK, uint32_t STAGE_DIV>
__global__ __launch_bounds__(SC_BLOCK) void k_part_scatter_hot(PartSource src, uint32_t A, uint32_t P,
                                                               const uint64_t* __restrict__ scale,
                                                               const uint64_t* __restrict__ bscale, uint32_t BB,
                                                               const uint32_t* __restrict__ O,
                                                               uint64_t* __restrict__ rec,
                                                               const uint32_t* __restrict__ seed, uint32_t S,
                                                               OwnerRegions orr, Rows rows,
                                                               uint32_t* __restrict__ err) {
  extern __shared__ uint64_t sm64[];
  constexpr uint32_t NWV = SC_BLOCK / 64;
  constexpr uint32_t SC_TILE = SC_EPT * SC_BLOCK, CAP = SC_TILE / STAGE_DIV;
  const uint32_t NB = 1u << BB, w = blockIdx.x, nw = gridDim.x, tid = threadIdx.x, lane = tid & 63;
  const uint32_t SP = S * P, NE = SP + 64;
  uint64_t* s_rec = sm64;                                             // [CAP][2]
  unsigned long long* s_lo = (unsigned long long*)(s_rec + 2 * CAP);  // [SP + 64 per-lane dummies]
  unsigned long long* s_hi = s_lo + NE;                                   // [SP + 64]
  uint32_t* s_tag = (uint32_t*)(s_hi + NE);                               // [S], 16-byte aligned
  uint16_t* s_bkt = (uint16_t*)(s_tag + S);                               // [CAP]
  uint32_t* s_cur = (uint32_t*)(s_bkt + CAP);      // [NB] this workgroup's next record per bucket
  uint32_t* s_cnt = s_cur + NB;                    // [2][NB] records of the tile per bucket (by tile parity)
  uint32_t* s_off = s_cnt + 2 * NB;                // [NB] tile offsets
  uint32_t* s_ocnt = s_off + NB;                   // [ATREX_OWNERS]
  __shared__ uint32_t s_w[NWV];
  for (uint32_t i = tid; i < NB; i += SC_BLOCK) {
    s_cur[i] = O[(size_t)i * nw + w];
    s_cnt[i] = 0;
    s_cnt[NB + i] = 0;
  }
  for (uint32_t i = tid; i < NE; i += SC_BLOCK) {
    s_lo[i] = 0;
    s_hi[i] = 0;
  }
  for (uint32_t i = tid; i < S; i += SC_BLOCK) s_tag[i] = seed[i];
  for (uint32_t i = tid; i < ATREX_OWNERS; i += SC_BLOCK) s_ocnt[i] = 0;
  const uint32_t dummy = SP + lane;  // this lane's dummy entry
  uint64_t b, e;
  part_range(src, w, b, e);
  const uint32_t lowbits = 32 - BB;
  const uint64_t lowmask = ((uint64_t)1 << lowbits) - 1;
  bool bad = false;
  constexpr uint32_t G4 = SC_EPT / 4;
  Ev4 nxt[G4];
#pragma unroll
  for (uint32_t g = 0; g < G4; ++g) load_group<false>(src.ev, b + 4 * ((uint64_t)g * SC_BLOCK + tid), e, nxt[g]);
  constexpr uint32_t PERMAX = 4;  // buckets per thread in the scan (NB <= 4 * SC_BLOCK)
  const uint32_t per = (NB + SC_BLOCK - 1) / SC_BLOCK, b0 = tid * per;
  uint32_t prevcnt[PERMAX] = {0, 0, 0, 0};
  uint32_t parity = 0;
  __syncthreads();
  for (uint64_t t0 = b; t0 < e; t0 += SC_TILE, parity ^= 1u) {  // uniform trip count
    Ev4 evg[G4];
#pragma unroll
    for (uint32_t g = 0; g < G4; ++g) evg[g] = nxt[g];
    uint32_t* cnt = s_cnt + parity * NB;
    uint32_t* cnt_next = s_cnt + (parity ^ 1u) * NB;
    // phase 1: the table slot (hot) or the bucket and rank (cold) of every
    // event; the scale words are requested here and used after the scan
    uint32_t hh[SC_EPT], rk[SC_EPT], hs[SC_EPT];  // hash; rank << 4 | record << 3 | phase; slot
    uint64_t dv[SC_EPT], sw[SC_EPT];
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j) {
      const uint64_t i = t0 + 4 * ((uint64_t)(j / 4) * SC_BLOCK + tid) + (j % 4);
      const bool vj = i < e;
      const Ev4& ev = evg[j / 4];
      const uint32_t jj = j % 4;
      const uint32_t a = ev.app[jj], ph = ev.ph(jj), key = ev.key[jj];
      const int64_t dd = ev.dur[jj];
      const bool ok = a < A && ph < P && dd >= 0;
      bad |= vj && !ok;
      // a lane past the range (its event zero-filled) and an invalid event
      // take the zero scale word (no share): every share below, hot or not,
      // is formed, and the general scale word's path re-reads the event
      sw[j] = (vj && ok) ? bscale[a * P + ph] : 0;
      dv[j] = (vj && ok) ? (uint64_t)dd : 0;
      rk[j] = ok ? ph : 0u;
      hs[j] = vj ? image_slot(s_tag, S, key) : kNoSlot;
      if (vj && hs[j] == kNoSlot) rk[j] |= 8u;
      if (!ok) hs[j] = kNoSlot;  // an invalid event adds nothing (the call fails on it)
      hh[j] = hash32(key);
    }
    // ranks from plain LDS atomics: the records' keys are the colder ones,
    // spread over the buckets
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j)
      if ((rk[j] >> 3) & 1u) rk[j] |= atomicAdd(&cnt[hh[j] >> lowbits], 1u) << 4;
    __syncthreads();
    // exclusive scan of the tile's bucket counts; the previous tile's counts
    // advance the positions, and the next tile's counters are cleared
    uint32_t tot = 0;  // records of the tile
    {
      uint32_t sum = 0;
#pragma unroll
      for (uint32_t k = 0; k < PERMAX; ++k) {
        if (k < per && b0 + k < NB) {
          const uint32_t c = cnt[b0 + k];
          s_cur[b0 + k] += prevcnt[k];
          prevcnt[k] = c;
          cnt_next[b0 + k] = 0;
          sum += c;
        }
      }
      const uint32_t wave = tid >> 6;
      const uint32_t inc = wave_incl_scan_u32(sum);
      if (lane == 63) s_w[wave] = inc;
      __syncthreads();
      uint32_t off = 0;
      for (uint32_t x = 0; x < NWV; ++x) {
        const uint32_t v = s_w[x];
        if (x < wave) off += v;
        tot += v;
      }
      uint32_t run = off + inc - sum;
#pragma unroll
      for (uint32_t k = 0; k < PERMAX; ++k)
        if (k < per && b0 + k < NB) { s_off[b0 + k] = run; run += prevcnt[k]; }
    }
    __syncthreads();
    // phase 2: the Q96 share of every event; the records of the first round
    // (tile positions below CAP) placed in LDS in bucket order, then the hot
    // events added to the table without branches (a lane with nothing to add
    // adds into its own dummy entry): the low words first, their returned
    // values giving the carries, then the high words with the count
    auto place = [&](uint32_t j, uint32_t r0, const uint64_t* vlj, const uint64_t* vhj) {
      if ((rk[j] >> 3) & 1u) {
        const uint32_t bk = hh[j] >> lowbits;
        const uint32_t at = s_off[bk] + (rk[j] >> 4) - r0;
        if (at < CAP) {
          s_rec[2 * at] = vlj[j];
          s_rec[2 * at + 1] = vhj[j] | ((uint64_t)(rk[j] & 7u) << 33) | (((uint64_t)hh[j] & lowmask) << 36);
          s_bkt[at] = (uint16_t)bk;
        }
      }
    };
    auto write_out = [&](uint32_t r0) {
      const uint32_t m = min(CAP, tot - r0);
      for (uint32_t k = tid; k < m; k += SC_BLOCK) {
        const uint32_t bb = s_bkt[k];
        const size_t pos = (size_t)s_cur[bb] + (k + r0 - s_off[bb]);
        v2l r;
        r.x = (long long)s_rec[2 * k];
        r.y = (long long)s_rec[2 * k + 1];
        *(v2l*)(rec + 2 * pos) = r;
      }
    };
    uint64_t vl[SC_EPT], vh[SC_EPT];
#pragma unroll
    for (uint32_t j = 0; j < SC_EPT; ++j) {
      const uint64_t wv = sw[j], d = dv[j];
      const uint32_t ph = rk[j] & 7u;
      if ((uint32_t)(wv >> 56) <= 127u) {
        if ((d >> 32) == 0) {
          uint32_t h32;
          bscale_share32((uint32_t)d, (uint32_t)wv, (uint32_t)(wv >> 32), vl[j], h32);
          vh[j] = h32;
        } else {
          bscale_share64(d, (uint32_t)wv, (uint32_t)(wv >> 32), vl[j], vh[j]);
        }
      } else {  // rho outside [-8, 63] (rare): the general scale word, found again from the event
        const uint64_t i = t0 + 4 * ((uint64_t)(j / 4) * SC_BLOCK + tid) + (j % 4);  // < e: sw != 0 above
        const u128 x = i < e ? event_share(d, scale[app_at<false>(src.ev.app, i) * P + ph]) : (u128)0;
        vl[j] = (uint64_t)x;
        vh[j] = (uint64_t)(x >> 64);
      }
      place(j, 0, vl, vh);
    }
    {
      uint32_t at[SC_EPT];
#pragma unroll
      for (uint32_t j = 0; j < SC_EPT; ++j) at[j] = hs[j] != kNoSlot ? hs[j] * P + (rk[j] & 7u) : dummy;
      unsigned long long old[SC_EPT];
#pragma unroll
      for (uint32_t j = 0; j < SC_EPT; ++j) old[j] = atomicAdd(&s_lo[at[j]], (unsigned long long)vl[j]);
#pragma unroll
      for (uint32_t j = 0; j < SC_EPT; ++j) {
        const unsigned long long carry = (old[j] + vl[j] < old[j]) ? 1ull : 0ull;
        atomicAdd(&s_hi[at[j]], (unsigned long long)vh[j] + carry + (1ull << ATREX_COUNT_SHIFT));
      }
    }
    if (t0 + SC_TILE < e) {
#pragma unroll
      for (uint32_t g = 0; g < G4; ++g)
        load_group<false>(src.ev, t0 + SC_TILE + 4 * ((uint64_t)g * SC_BLOCK + tid), e, nxt[g]);
    }
    __syncthreads();
    write_out(0);
    if (STAGE_DIV > 1 && tot > CAP) {  // uniform: the second round
      __syncthreads();
#pragma unroll
      for (uint32_t j = 0; j < SC_EPT; ++j) place(j, CAP, vl, vh);
      __syncthreads();
      write_out(CAP);
    }
  }
  if (__any(bad) && lane == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
  __syncthreads();
  // the table -> owner regions (owner = top byte of the key hash); a region
  // that is full sends its rows straight to the row list
  for (uint32_t s0 = 0; s0 < S; s0 += SC_BLOCK) {
    const uint32_t sl = s0 + tid;
    const uint32_t t = sl < S ? s_tag[sl] : ATREX_EMPTY_KEY;
    bool spill_rows = false;
    if (t != ATREX_EMPTY_KEY) {
      const uint32_t o = hash32(t) >> 24;
      const uint32_t r = atomicAdd(&s_ocnt[o], 1u);
      if (r < orr.capo) {
        const size_t ri = ((size_t)w * ATREX_OWNERS + o) * orr.capo + r;
        orr.key[ri] = t;
        for (uint32_t ph = 0; ph < P; ++ph) {
          orr.acc[(ri * P + ph) * 2] = s_lo[sl * P + ph];
          orr.acc[(ri * P + ph) * 2 + 1] = s_hi[sl * P + ph];
        }
      } else {
        spill_rows = true;
      }
    }
    for (uint32_t ph = 0; ph < P; ++ph) {
      const size_t gi = (size_t)sl * P + ph;
      const uint64_t hi = spill_rows ? s_hi[gi] : 0;
      const bool want = spill_rows && (hi >> ATREX_COUNT_SHIFT) != 0;
      row_append(rows, want, ((uint64_t)t << 3) | ph, want ? s_lo[gi] : 0, hi, 0, 0, err);
    }
  }
  __syncthreads();
  for (uint32_t o = tid; o < ATREX_OWNERS; o += SC_BLOCK)
    orr.count[(size_t)w * ATREX_OWNERS + o] = min(s_ocnt[o], orr.capo);
}

// Work items = (bucket, chunk of at most CH records); item_start[b] = first
// item of bucket b, item_start[NB] = number of items.
__global__ __launch_bounds__(1024) void k_part_items(const uint32_t* __restrict__ O, const uint32_t* __restrict__ H,
                                                     uint32_t nw, uint32_t BB, uint32_t CH,
                                                     uint32_t* __restrict__ bstart, uint32_t* __restrict__ item_start) {
  __shared__ uint32_t s_w[16];
  const uint32_t NB = 1u << BB;
  const uint32_t per = (NB + 1023) / 1024;  // buckets per thread (contiguous)
  uint32_t cnt[4] = {0, 0, 0, 0};
  uint32_t tsum = 0;
  for (uint32_t k = 0; k < per && k < 4; ++k) {
    const uint32_t bkt = threadIdx.x * per + k;
    if (bkt < NB) {
      const uint32_t beg = O[(size_t)bkt * nw];
      const uint32_t end = O[(size_t)bkt * nw + nw - 1] + H[(size_t)bkt * nw + nw - 1];
      bstart[bkt] = beg;
      if (bkt == NB - 1) bstart[NB] = end;
      cnt[k] = (end - beg + CH - 1) / CH;
      tsum += cnt[k];
    }
  }
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = tsum;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d, 64);
    if (lane >= (uint32_t)d) inc += y;
  }
  if (lane == 63) s_w[wave] = inc;
  __syncthreads();
  uint32_t off = 0, total = 0;
  for (uint32_t i = 0; i < 16; ++i) {
    if (i < wave) off += s_w[i];
    total += s_w[i];
  }
  uint32_t run = off + inc - tsum;
  for (uint32_t k = 0; k < per && k < 4; ++k) {
    const uint32_t bkt = threadIdx.x * per + k;
    if (bkt < NB) {
      item_start[bkt] = run;
      run += cnt[k];
    }
  }
  if (threadIdx.x == 0) item_start[NB] = total;
}

// Per work item (bucket, chunk): an LDS table of S slots in buckets of four
// tags (the record's low hash bits; with the bucket they give the key back
// through the inverse mix) and per phase a two-word accumulator, plus 64
// per-lane dummy entries for lanes with nothing to add; four records per lane
// per step; the (at most two) entries most of a wave hits are summed in
// registers (HotPair) and added once at the end of the item.
template <bool RAW>
__global__ __launch_bounds__(1024) void k_part_aggregate(const uint64_t* __restrict__ rec,
                                                         const uint64_t* __restrict__ rraw, uint32_t BB, uint32_t CH,
                                                         const uint32_t* __restrict__ bstart,
                                                         const uint32_t* __restrict__ item_start, uint32_t P,
                                                         uint32_t S, Rows rows, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  __shared__ uint32_t s_wsum[16];
  __shared__ unsigned long long s_base;
  // low and high words of the [S * P] accumulators as two arrays (a wave's
  // 64-bit atomics then spread over twice the LDS banks of interleaved
  // pairs), each followed by 64 per-lane dummy entries for lanes with nothing
  // to add (never read); RAW: the same again
  const uint32_t SP = S * P, NE = SP + 64, region = 2 * NE;
  unsigned long long* lo_ = smem;
  unsigned long long* hi_ = smem + NE;
  unsigned long long* rlo_ = smem + region;  // RAW only
  unsigned long long* rhi_ = smem + region + NE;
  uint32_t* tag = (uint32_t*)(smem + (RAW ? 2 : 1) * region);  // [S], 16-byte aligned
  const uint32_t NB = 1u << BB, lowbits = 32 - BB, NBK = S / 4;
  const uint32_t lane = lane_of(), dummy = SP + lane;
  const uint32_t items = item_start[NB];
  auto bucket_tags = [&](uint32_t bq) -> uint4 { return *(const uint4*)&tag[4 * bq]; };
  auto find_slot = [&](uint32_t k, uint32_t bq, uint4 tv) -> int32_t {
    uint32_t probe = 0;
#pragma unroll 1
    for (uint32_t step = 0; step < 256; ++step) {
      if (tv.x == k) return (int32_t)(4 * bq);
      if (tv.y == k) return (int32_t)(4 * bq + 1);
      if (tv.z == k) return (int32_t)(4 * bq + 2);
      if (tv.w == k) return (int32_t)(4 * bq + 3);
      const uint32_t x = tv.x == EMPTY_TAG ? 0u : tv.y == EMPTY_TAG ? 1u : tv.z == EMPTY_TAG ? 2u
                       : tv.w == EMPTY_TAG ? 3u : 4u;
      if (x < 4) {
        const uint32_t t = atomicCAS(&tag[4 * bq + x], EMPTY_TAG, k);
        if (t == EMPTY_TAG || t == k) return (int32_t)(4 * bq + x);
      } else {
        if (++probe == 32) return -1;
        bq = (bq + 1 == NBK) ? 0 : bq + 1;
      }
      tv = bucket_tags(bq);
    }
    return -1;
  };
  for (uint32_t it = blockIdx.x; it < items; it += gridDim.x) {
    uint32_t lo_b = 0, hi_b = NB;  // bucket: last b with item_start[b] <= it
    while (hi_b - lo_b > 1) {
      const uint32_t mid = (lo_b + hi_b) / 2;
      if (item_start[mid] <= it) lo_b = mid; else hi_b = mid;
    }
    const uint32_t bkt = lo_b;
    const uint32_t c = it - item_start[bkt];
    const uint32_t r0 = bstart[bkt] + c * CH;
    const uint32_t r1 = min(bstart[bkt + 1], r0 + CH);
    for (uint32_t i = threadIdx.x; i < SP; i += blockDim.x) {
      lo_[i] = 0;
      hi_[i] = 0;
      if (RAW) { rlo_[i] = 0; rhi_[i] = 0; }
    }
    for (uint32_t i = threadIdx.x; i < S; i += blockDim.x) tag[i] = EMPTY_TAG;
    __syncthreads();
    // four records per lane per step; the next step's records are loaded
    // while this step accumulates (indices clamped into the item)
    HotPair<RAW> hot;
    hot.reset();
    bool first = true;
    v2l nr[4];
    uint64_t nd[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t ic = min(r0 + j * blockDim.x + threadIdx.x, r1 - 1);
      nr[j] = __builtin_nontemporal_load((const v2l*)(rec + 2 * (size_t)ic));
      nd[j] = RAW ? rraw[ic] : 0;
    }
    for (uint32_t base = r0; base < r1; base += 4 * blockDim.x) {  // uniform trip count
      uint64_t vlo[4], vhi[4], d[4];
      uint32_t low[4], ph[4], gi[4];
      bool valid[4];
      uint4 tv[4];
      v2l cr[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        cr[j] = nr[j];
        d[j] = nd[j];
      }
      if (base + 4 * blockDim.x < r1) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t ic = min(base + 4 * blockDim.x + j * blockDim.x + threadIdx.x, r1 - 1);
          nr[j] = __builtin_nontemporal_load((const v2l*)(rec + 2 * (size_t)ic));
          nd[j] = RAW ? rraw[ic] : 0;
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t i = base + j * blockDim.x + threadIdx.x;
        valid[j] = i < r1;
        vlo[j] = (uint64_t)cr[j].x;
        const uint64_t w1 = (uint64_t)cr[j].y;
        low[j] = (uint32_t)(w1 >> 36);
        ph[j] = (uint32_t)(w1 >> 33) & 7u;
        vhi[j] = w1 & (((uint64_t)1 << 33) - 1);
        tv[j] = bucket_tags((uint32_t)(((uint64_t)hash_mul(low[j]) * NBK) >> 32));
      }
      bool miss = false;
#pragma unroll
      for (int j = 0; j < 4; ++j) {  // branch-free match of the four tags
        const uint32_t k = low[j];
        const uint32_t bq = (uint32_t)(((uint64_t)hash_mul(k) * NBK) >> 32);
        const uint32_t mask = (tv[j].x == k ? 1u : 0u) | (tv[j].y == k ? 2u : 0u) | (tv[j].z == k ? 4u : 0u) |
                              (tv[j].w == k ? 8u : 0u);
        const bool hit = valid[j] && mask != 0;
        gi[j] = hit ? (4 * bq + (uint32_t)(__ffs(mask) - 1)) * P + ph[j] : 0xFFFFFFFFu;
        miss |= valid[j] && !hit;
      }
      if (__any(miss)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int32_t sl = -2;
          if (valid[j] && gi[j] == 0xFFFFFFFFu) {
            sl = find_slot(low[j], (uint32_t)(((uint64_t)hash_mul(low[j]) * NBK) >> 32), tv[j]);
            if (sl >= 0) gi[j] = (uint32_t)sl * P + ph[j];
          }
          const uint32_t key = unmix32((bkt << lowbits) | low[j]);
          row_append(rows, sl == -1, ((uint64_t)key << 3) | ph[j], vlo[j], vhi[j] + (1ull << ATREX_COUNT_SHIFT),
                     d[j], 0, err);
        }
      }
      // entries most of the wave hits are summed in registers
      if (first) {
        hot.choose(gi[0], 16);
        first = false;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (hot.take(gi[j], vlo[j], vhi[j], d[j])) gi[j] = 0xFFFFFFFFu;
      uint32_t at[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) at[j] = gi[j] != 0xFFFFFFFFu ? gi[j] : dummy;
      unsigned long long old[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) old[j] = atomicAdd(&lo_[at[j]], (unsigned long long)vlo[j]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        atomicAdd(&hi_[at[j]],
                  (unsigned long long)vhi[j] + ((old[j] + vlo[j] < old[j]) ? 1ull : 0ull) + (1ull << ATREX_COUNT_SHIFT));
      if (RAW) {
#pragma unroll
        for (int j = 0; j < 4; ++j) old[j] = atomicAdd(&rlo_[at[j]], (unsigned long long)d[j]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (old[j] + d[j] < old[j]) atomicAdd(&rhi_[at[j]], 1ull);
      }
    }
    hot.flush([&](uint32_t g, u128 tv, uint32_t c, u128 tr) {
      acc_add_n(&lo_[g], &hi_[g], tv, c);
      if (RAW) acc_add_plain(&rlo_[g], &rhi_[g], tr);
    });
    __syncthreads();
    // the item's rows: each thread takes a contiguous run of (slot, phase)
    // entries; one row-list reservation per workgroup
    const uint32_t per = (SP + blockDim.x - 1) / blockDim.x, e0 = threadIdx.x * per;
    auto present = [&](uint32_t i) {
      return i < SP && tag[i / P] != EMPTY_TAG && (hi_[i] >> ATREX_COUNT_SHIFT) != 0;
    };
    uint32_t mine = 0;
    for (uint32_t k = 0; k < per; ++k) mine += present(e0 + k) ? 1u : 0u;
    uint32_t inc = mine;
    const uint32_t wl = threadIdx.x & 63, wv = threadIdx.x >> 6;
    for (int dd = 1; dd < 64; dd <<= 1) {
      const uint32_t y = __shfl_up(inc, dd, 64);
      if (wl >= (uint32_t)dd) inc += y;
    }
    if (wl == 63) s_wsum[wv] = inc;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint32_t tot = 0;
      for (uint32_t x = 0; x < blockDim.x / 64; ++x) tot += s_wsum[x];
      s_base = atomicAdd(rows.count, (unsigned long long)tot);
    }
    __syncthreads();
    uint64_t pos = s_base + inc - mine;
    for (uint32_t x = 0; x < wv; ++x) pos += s_wsum[x];
    for (uint32_t k = 0; k < per; ++k) {
      const uint32_t i = e0 + k;
      if (!present(i)) continue;
      if (pos >= rows.cap) {
        atomicOr(err, ATREX_ERRBIT_CAPACITY);
        break;
      }
      const uint32_t sl = i / P, ph = i - sl * P;
      rows.rk[pos] = ((uint64_t)unmix32((bkt << lowbits) | tag[sl]) << 3) | ph;
      rows.lo[pos] = lo_[i];
      rows.hi[pos] = hi_[i];
      if (RAW) { rows.rlo[pos] = rlo_[i]; rows.rhi[pos] = rhi_[i]; }
      ++pos;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- rows -> groups
// One thread per run of equal sort keys (rows already ordered through idx).
__global__ void k_rows_reduce(Rows rows, const uint64_t* __restrict__ rk_sorted, const uint32_t* __restrict__ idx,
                              const uint32_t* __restrict__ starts, uint64_t G, SortedGroups out) {
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  const uint32_t b = starts[g], e = starts[g + 1];
  u128 x = 0, r = 0;
  for (uint32_t i = b; i < e; ++i) {
    const uint32_t j = idx[i];
    x += make_u128(rows.lo[j], rows.hi[j]);
    if (out.raw) r += make_u128(rows.rlo[j], rows.rhi[j]);
  }
  const uint64_t rk = rk_sorted[b];
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
}

__global__ void k_iota_rows(const Rows rows, uint64_t R, uint64_t* __restrict__ k, uint32_t* __restrict__ v) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= R) return;
  k[i] = rows.rk[i];
  v[i] = (uint32_t)i;
}

uint32_t grid_of(uint64_t n, uint32_t b) { return (uint32_t)((n + b - 1) / b); }

}  // namespace

uint32_t lds_table_slots(uint32_t P, bool raw, size_t lds_bytes) {
  const size_t per = 4 + (size_t)16 * P * (raw ? 2 : 1);
  const size_t fixed = 2048 + (size_t)64 * 16 * (raw ? 2 : 1);
  return (uint32_t)(((lds_bytes - fixed) / per) & ~(size_t)3);  // whole buckets of four
}

size_t lds_table_bytes(uint32_t P, bool raw, uint32_t S) {
  return ((size_t)S * P * 16 + 64 * 16) * (raw ? 2 : 1) + (size_t)S * 4;
}

constexpr uint32_t kScatterEpt = 4, kScatterBlock = 1024;
// k_part_scatter_hot: events per thread per tile, and the dynamic LDS it may
// take (static LDS beside it: the scan's wave sums)
constexpr uint32_t kHotEpt = 4, kHotStageDiv = 1;
constexpr size_t kHotLds = 160 * 1024 - 256;

static size_t scatter_smem(uint32_t BB, bool raw) {
  return (size_t)kScatterEpt * kScatterBlock * (16 + (raw ? 8 : 0) + 2) + ((size_t)4 << BB) * 4;
}

uint32_t part_scatter_wgs(uint32_t cus) { return std::min<uint32_t>(kMaxPartWG, cus); }


void launch_part_hist(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t BB, uint32_t* H) {
  hipLaunchKernelGGL(k_part_hist<false>, dim3(nwg), dim3(1024), (size_t)4 << BB, s, src, BB, H, nullptr, 0u);
}

void launch_part_hist_cold(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t BB, uint32_t* H,
                           const uint32_t* seed, uint32_t S) {
  hipLaunchKernelGGL(k_part_hist<true>, dim3(nwg), dim3(1024), ((size_t)4 << BB) + (size_t)4 * S, s, src, BB, H,
                     seed, S);
}

// LDS of k_part_scatter_hot: the staged records and their buckets, the
// bucket counters, the owner counters and the table of S slots.
static size_t hot_scatter_smem(uint32_t P, uint32_t BB, uint32_t S) {
  return (size_t)kHotEpt * kScatterBlock / kHotStageDiv * (16 + 2) + ((size_t)4 << BB) * 4 + (size_t)ATREX_OWNERS * 4 +
         ((size_t)S * P + 64) * 16 + (size_t)S * 4;
}

uint32_t hot_scatter_slots(uint32_t P, uint32_t BB) {
  const size_t fixed = hot_scatter_smem(P, BB, 0);
  if (fixed >= kHotLds) return 0;
  const uint32_t S = (uint32_t)((kHotLds - fixed) / (16 * (size_t)P + 4)) & ~3u;
  return S >= 8 ? S : 0;
}

void launch_hot_scatter(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t A, uint32_t P,
                        const uint64_t* scale, const uint64_t* bscale, uint32_t BB, const uint32_t* O, uint64_t* rec,
                        const uint32_t* seed, uint32_t S, const OwnerRegions& orr, const Rows& rows, uint32_t* err) {
  hipLaunchKernelGGL((k_part_scatter_hot<kHotEpt, kScatterBlock, kHotStageDiv>), dim3(nwg), dim3(kScatterBlock),
                     hot_scatter_smem(P, BB, S), s, src, A, P, scale, bscale, BB, O, rec, seed, S, orr, rows, err);
}

void launch_part_scatter(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t A, uint32_t P,
                         const uint64_t* scale, const uint64_t* bscale, uint32_t BB, const uint32_t* O, uint64_t* rec,
                         uint64_t* rraw, uint32_t* err) {
  const size_t smem = scatter_smem(BB, rraw != nullptr);
#define ATREX_SCATTER(R, S)                                                                                     \
  hipLaunchKernelGGL((k_part_scatter<R, S, kScatterEpt, kScatterBlock>), dim3(nwg), dim3(kScatterBlock), smem, s, \
                     src, A, P, scale, bscale, BB, O, rec, rraw, err)
  if (!src.spill && !src.ev.app) {  // events without applications (the host takes no raw time then)
    hipLaunchKernelGGL((k_part_scatter<false, false, kScatterEpt, kScatterBlock, true>), dim3(nwg),
                       dim3(kScatterBlock), smem, s, src, A, P, scale, bscale, BB, O, rec, rraw, err);
  } else if (rraw) {
    if (src.spill) ATREX_SCATTER(true, true); else ATREX_SCATTER(true, false);
  } else {
    if (src.spill) ATREX_SCATTER(false, true); else ATREX_SCATTER(false, false);
  }
#undef ATREX_SCATTER
}

void launch_part_items(hipStream_t s, const uint32_t* O, const uint32_t* H, uint32_t nw, uint32_t BB, uint32_t CH,
                       uint32_t* bstart, uint32_t* item_start) {
  hipLaunchKernelGGL(k_part_items, dim3(1), dim3(1024), 0, s, O, H, nw, BB, CH, bstart, item_start);
}

void launch_part_aggregate(hipStream_t s, const uint64_t* rec, const uint64_t* rraw, uint32_t BB, uint32_t CH,
                           const uint32_t* bstart, const uint32_t* item_start, uint32_t P, uint32_t S,
                           uint32_t nblocks, const Rows& rows, uint32_t* err) {
  const size_t smem = lds_table_bytes(P, rraw != nullptr, S);
  if (rraw)
    hipLaunchKernelGGL(k_part_aggregate<true>, dim3(nblocks), dim3(1024), smem, s, rec, rraw, BB, CH, bstart,
                       item_start, P, S, rows, err);
  else
    hipLaunchKernelGGL(k_part_aggregate<false>, dim3(nblocks), dim3(1024), smem, s, rec, rraw, BB, CH, bstart,
                       item_start, P, S, rows, err);
}

void launch_iota_rows(hipStream_t s, const Rows& rows, uint64_t R, uint64_t* k, uint32_t* v) {
  if (R) hipLaunchKernelGGL(k_iota_rows, dim3(grid_of(R, 256)), dim3(256), 0, s, rows, R, k, v);
}

void launch_rows_reduce(hipStream_t s, const Rows& rows, const uint64_t* rk_sorted, const uint32_t* idx,
                        const uint32_t* starts, uint64_t G, const SortedGroups& out) {
  if (G) hipLaunchKernelGGL(k_rows_reduce, dim3(grid_of(G, 256)), dim3(256), 0, s, rows, rk_sorted, idx, starts, G, out);
}

static uint32_t pow2_ge(uint32_t x) {
  uint32_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

uint32_t owner_list_slots(uint32_t P, bool raw) {
  const size_t budget = 160 * 1024 - 4096 - kRegionMap;
  uint32_t So = 1024;
  while (So > 64 && (size_t)So * (4 + 16 * P * (raw ? 2 : 1)) + (size_t)pow2_ge(So * P) * 8 > budget) So >>= 1;
  return So;
}


static size_t owner_finish_smem(uint32_t P, bool raw, uint32_t So) {
  return (size_t)So * P * 16 * (raw ? 2 : 1) + (size_t)pow2_ge(So * P) * 8 + (size_t)So * 4 + kRegionMap;
}

void launch_owner_finish(hipStream_t s, const OwnerRegions& orr, uint32_t nwg, uint32_t P, bool raw, uint32_t So,
                         const SpillIn& sp, const OwnerLists& ol, const Rows& rows, uint32_t* err) {
  const size_t smem = owner_finish_smem(P, raw, So);
  if (raw)
    hipLaunchKernelGGL(k_owner_finish<true>, dim3(ATREX_OWNERS), dim3(1024), smem, s, orr, nwg, P, So, sp, ol, rows,
                       err);
  else
    hipLaunchKernelGGL(k_owner_finish<false>, dim3(ATREX_OWNERS), dim3(1024), smem, s, orr, nwg, P, So, sp, ol, rows,
                       err);
}

void launch_rank_groups(hipStream_t s, const OwnerLists& ol, uint32_t P, const SpillIn& sp, const Rows& rows,
                        const uint32_t* err, const SortedGroups& out, uint64_t* S_out, unsigned long long* G_out,
                        uint32_t* done) {
  // rows staged: kRankMax, or fewer when the owner lists are long
  const size_t budget = 160 * 1024 - 4096 - (size_t)ol.cap * 16;
  const uint32_t rmax = (uint32_t)std::min<size_t>(kRankMax, budget / 4) & ~7u;
  const size_t smem = (size_t)rmax * 4 + (size_t)ol.cap * 16;
  hipLaunchKernelGGL(k_rank_groups, dim3(ATREX_OWNERS), dim3(1024), smem, s, ol, P, sp, rows, err, out, S_out, G_out,
                     done, rmax);
}

void launch_lists_to_rows(hipStream_t s, const OwnerLists& ol, const Rows& rows, uint32_t* err) {
  hipLaunchKernelGGL(k_lists_to_rows, dim3(ATREX_OWNERS), dim3(256), 0, s, ol, rows, err);
}

// Dynamic LDS limits: 160 KB less a margin that covers each kernel's static LDS.
hipError_t set_rows_smem_limits() {
  const void* fns[] = {(const void*)k_part_aggregate<true>, (const void*)k_part_aggregate<false>,
                       (const void*)k_part_hist<false>, (const void*)k_part_hist<true>,
                       (const void*)k_part_scatter<true, false, kScatterEpt, kScatterBlock>,
                       (const void*)k_part_scatter<true, true, kScatterEpt, kScatterBlock>,
                       (const void*)k_part_scatter<false, false, kScatterEpt, kScatterBlock>,
                       (const void*)k_part_scatter<false, true, kScatterEpt, kScatterBlock>,
                       (const void*)k_part_scatter<false, false, kScatterEpt, kScatterBlock, true>};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 2048);
    if (e != hipSuccess) return e;
  }
  {
    const hipError_t e = hipFuncSetAttribute((const void*)k_part_scatter_hot<kHotEpt, kScatterBlock, kHotStageDiv>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kHotLds);
    if (e != hipSuccess) return e;
  }
  const void* fo[] = {(const void*)k_owner_finish<true>, (const void*)k_owner_finish<false>,
                      (const void*)k_rank_groups};
  for (const void* f : fo) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 4096);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
