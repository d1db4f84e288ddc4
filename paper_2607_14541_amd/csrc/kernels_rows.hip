// kernels_rows.hip -- group rows and the radix-partition engine (gfx950).
//
// Every pass-B engine emits rows (sort key = key << 3 | phase, two-word
// accumulator X = W + count * 2^97, optional raw time); a radix sort on the
// sort key and a segmented sum turn the rows into the ordered groups.
//
//  * owner merge: the LDS engine leaves, per workgroup, its table split into
//    256 owner regions (owner = top byte of an invertible hash of the key);
//    one workgroup per owner sums the regions in an LDS table and emits rows.
//  * radix-partition engine (high key cardinality, and the LDS engine's
//    spilled events): per-workgroup bucket histograms of the top BB bits of the
//    key hash, one scan, a scatter of 16-byte records (Q96 share, phase, the
//    low 32 - BB hash bits), then per bucket chunk an LDS group-by that emits
//    rows; the key is recovered by inverting the hash.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t MAXPROBE_R = 32;
constexpr uint32_t EMPTY_TAG = 0xFFFFFFFFu;

// Invertible 32-bit mix (xorshift-multiply) and its inverse.
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

// ---------------------------------------------------------------- owner merge
template <bool RAW>
__global__ __launch_bounds__(1024) void k_owner_merge(OwnerRegions orr, uint32_t nwg, uint32_t P, uint32_t S,
                                                      Rows rows, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  __shared__ uint32_t s_pre[257];
  LdsTable<RAW> tb;
  tb.init(smem, S, P);
  tb.clear();
  const uint32_t o = blockIdx.x;
  if (threadIdx.x < 64) {  // prefix over the workgroups' row counts for this owner
    uint32_t run = 0;
    for (uint32_t w0 = 0; w0 < nwg; w0 += 64) {
      const uint32_t w = w0 + threadIdx.x;
      const uint32_t c = w < nwg ? orr.count[(size_t)w * ATREX_OWNERS + o] : 0;
      uint32_t inc = c;
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = __shfl_up(inc, d, 64);
        if (threadIdx.x >= (uint32_t)d) inc += y;
      }
      if (w < nwg) s_pre[w] = run + inc - c;
      run += __shfl(inc, 63, 64);
    }
    if (threadIdx.x == 0) s_pre[nwg] = run;
  }
  __syncthreads();
  const uint32_t total = s_pre[nwg];
  for (uint32_t base = 0; base < total; base += blockDim.x) {  // uniform trip count
    const uint32_t idx = base + threadIdx.x;
    const bool valid = idx < total;
    uint32_t key = 0, w = 0;
    size_t rec = 0;
    int32_t sl = -1;
    if (valid) {
      uint32_t lo_w = 0, hi_w = nwg;  // last w with s_pre[w] <= idx
      while (hi_w - lo_w > 1) {
        const uint32_t mid = (lo_w + hi_w) / 2;
        if (s_pre[mid] <= idx) lo_w = mid; else hi_w = mid;
      }
      w = lo_w;
      rec = ((size_t)w * ATREX_OWNERS + o) * orr.capo + (idx - s_pre[w]);
      key = orr.key[rec];
      sl = tb.slot(key);
    }
    for (uint32_t ph = 0; ph < P; ++ph) {
      uint64_t lo = 0, hi = 0, rl = 0, rh = 0;
      if (valid) {
        lo = orr.acc[(rec * P + ph) * 2];
        hi = orr.acc[(rec * P + ph) * 2 + 1];
        if (RAW) { rl = orr.raw[(rec * P + ph) * 2]; rh = orr.raw[(rec * P + ph) * 2 + 1]; }
      }
      const bool present = valid && (hi >> ATREX_COUNT_SHIFT) != 0;
      if (present && sl >= 0) {
        lds_add2(&tb.lo[sl * P + ph], &tb.hi[sl * P + ph], lo, hi);
        if (RAW) lds_add2(&tb.rlo[sl * P + ph], &tb.rhi[sl * P + ph], rl, rh);
      }
      row_append(rows, present && sl < 0, ((uint64_t)key << 3) | ph, lo, hi, rl, rh, err);
    }
  }
  __syncthreads();
  for (uint32_t base = 0; base < S * P; base += blockDim.x) {
    const uint32_t i = base + threadIdx.x;
    bool want = false;
    uint64_t rk = 0, lo = 0, hi = 0, rl = 0, rh = 0;
    if (i < S * P) {
      const uint32_t s = i / P, ph = i - s * P;
      const uint32_t t = tb.tag[s];
      hi = tb.hi[i];
      want = t != EMPTY_TAG && (hi >> ATREX_COUNT_SHIFT) != 0;
      rk = ((uint64_t)t << 3) | ph;
      lo = tb.lo[i];
      if (RAW) { rl = tb.rlo[i]; rh = tb.rhi[i]; }
    }
    row_append(rows, want, rk, lo, hi, rl, rh, err);
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

__global__ __launch_bounds__(1024) void k_part_hist(PartSource src, uint32_t BB, uint32_t* __restrict__ H) {
  extern __shared__ uint32_t s_h[];
  const uint32_t NB = 1u << BB, w = blockIdx.x, nw = gridDim.x;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_h[i] = 0;
  __syncthreads();
  uint64_t b, e;
  part_range(src, w, b, e);
  const uint32_t* keys = src.spill ? src.skey : src.ev.key;
  for (uint64_t i = b + threadIdx.x; i < e; i += blockDim.x) atomicAdd(&s_h[hash32(keys[i]) >> (32 - BB)], 1u);
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) H[(size_t)i * nw + w] = s_h[i];
}

template <bool RAW>
__global__ __launch_bounds__(1024) void k_part_scatter(PartSource src, uint32_t A, uint32_t P,
                                                       const uint64_t* __restrict__ scale, uint32_t BB,
                                                       const uint32_t* __restrict__ O, uint64_t* __restrict__ rec,
                                                       uint64_t* __restrict__ rraw, uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s_pos[];
  const uint32_t NB = 1u << BB, w = blockIdx.x, nw = gridDim.x;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_pos[i] = O[(size_t)i * nw + w];
  __syncthreads();
  uint64_t b, e;
  part_range(src, w, b, e);
  const uint32_t lowbits = 32 - BB;
  const uint64_t lowmask = ((uint64_t)1 << lowbits) - 1;
  bool bad = false;
  for (uint64_t i = b + threadIdx.x; i < e; i += blockDim.x) {
    uint32_t key, ph;
    uint64_t vlo, vhi, d = 0;
    if (src.spill) {
      key = src.skey[i];
      vlo = src.sval[2 * i];
      vhi = src.sval[2 * i + 1] & (((uint64_t)1 << 40) - 1);
      ph = (uint32_t)(src.sval[2 * i + 1] >> 40);
      if (RAW) d = src.sraw[i];
    } else {
      key = src.ev.key[i];
      const uint32_t a = src.ev.app[i];
      ph = src.ev.phase[i];
      const int64_t dd = src.ev.dur[i];
      const bool ok = a < A && ph < P && dd >= 0;
      bad |= !ok;
      const uint64_t sw = ok ? scale[(size_t)a * P + ph] : 0;
      const u128 v = event_share(ok ? (uint64_t)dd : 0, sw);
      vlo = (uint64_t)v;
      vhi = (uint64_t)(v >> 64);
      ph &= 7;
      d = ok ? (uint64_t)dd : 0;
    }
    const uint32_t h = hash32(key);
    const uint32_t pos = atomicAdd(&s_pos[h >> lowbits], 1u);
    rec[2 * (size_t)pos] = vlo;
    rec[2 * (size_t)pos + 1] = vhi | ((uint64_t)ph << 33) | (((uint64_t)h & lowmask) << 36);
    if (RAW) rraw[pos] = d;
  }
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(err, ATREX_ERRBIT_RANGE);
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

template <bool RAW>
__global__ __launch_bounds__(1024) void k_part_aggregate(const uint64_t* __restrict__ rec,
                                                         const uint64_t* __restrict__ rraw, uint32_t BB, uint32_t CH,
                                                         const uint32_t* __restrict__ bstart,
                                                         const uint32_t* __restrict__ item_start, uint32_t P,
                                                         uint32_t S, Rows rows, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long smem[];
  LdsTable<RAW> tb;
  tb.init(smem, S, P);
  const uint32_t NB = 1u << BB, lowbits = 32 - BB;
  const uint32_t items = item_start[NB];
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
    tb.clear();
    __syncthreads();
    for (uint32_t base = r0; base < r1; base += blockDim.x) {  // uniform trip count
      const uint32_t i = base + threadIdx.x;
      const bool valid = i < r1;
      uint64_t vlo = 0, w1 = 0, d = 0;
      if (valid) {
        vlo = rec[2 * (size_t)i];
        w1 = rec[2 * (size_t)i + 1];
        if (RAW) d = rraw[i];
      }
      const uint32_t low = (uint32_t)(w1 >> 36), ph = (uint32_t)(w1 >> 33) & 7u;
      const uint64_t vhi = w1 & (((uint64_t)1 << 33) - 1);
      const int32_t sl = valid ? tb.slot(low) : -1;
      if (valid && sl >= 0) {
        const uint32_t gi = (uint32_t)sl * P + ph;
        lds_add2(&tb.lo[gi], &tb.hi[gi], vlo, vhi + (1ull << ATREX_COUNT_SHIFT));
        if (RAW) lds_add2(&tb.rlo[gi], &tb.rhi[gi], d, 0);
      }
      const uint32_t key = unmix32((bkt << lowbits) | low);
      row_append(rows, valid && sl < 0, ((uint64_t)key << 3) | ph, vlo, vhi + (1ull << ATREX_COUNT_SHIFT), d, 0, err);
    }
    __syncthreads();
    for (uint32_t base = 0; base < S * P; base += blockDim.x) {
      const uint32_t i = base + threadIdx.x;
      bool want = false;
      uint64_t rk = 0, lo = 0, hi = 0, rl = 0, rh = 0;
      if (i < S * P) {
        const uint32_t s = i / P, ph = i - s * P;
        const uint32_t t = tb.tag[s];
        hi = tb.hi[i];
        want = t != EMPTY_TAG && (hi >> ATREX_COUNT_SHIFT) != 0;
        if (want) rk = ((uint64_t)unmix32((bkt << lowbits) | t) << 3) | ph;
        lo = tb.lo[i];
        if (RAW) { rl = tb.rlo[i]; rh = tb.rhi[i]; }
      }
      row_append(rows, want, rk, lo, hi, rl, rh, err);
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
  return (uint32_t)((lds_bytes - 2048) / per);
}

size_t lds_table_bytes(uint32_t P, bool raw, uint32_t S) { return (size_t)S * (4 + (size_t)16 * P * (raw ? 2 : 1)); }

void launch_owner_merge(hipStream_t s, const OwnerRegions& orr, uint32_t nwg, uint32_t P, bool raw, uint32_t S,
                        const Rows& rows, uint32_t* err) {
  const size_t smem = lds_table_bytes(P, raw, S);
  if (raw)
    hipLaunchKernelGGL(k_owner_merge<true>, dim3(ATREX_OWNERS), dim3(1024), smem, s, orr, nwg, P, S, rows, err);
  else
    hipLaunchKernelGGL(k_owner_merge<false>, dim3(ATREX_OWNERS), dim3(1024), smem, s, orr, nwg, P, S, rows, err);
}

void launch_part_hist(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t BB, uint32_t* H) {
  hipLaunchKernelGGL(k_part_hist, dim3(nwg), dim3(1024), (size_t)4 << BB, s, src, BB, H);
}

void launch_part_scatter(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t A, uint32_t P,
                         const uint64_t* scale, uint32_t BB, const uint32_t* O, uint64_t* rec, uint64_t* rraw,
                         uint32_t* err) {
  if (rraw)
    hipLaunchKernelGGL(k_part_scatter<true>, dim3(nwg), dim3(1024), (size_t)4 << BB, s, src, A, P, scale, BB, O, rec,
                       rraw, err);
  else
    hipLaunchKernelGGL(k_part_scatter<false>, dim3(nwg), dim3(1024), (size_t)4 << BB, s, src, A, P, scale, BB, O,
                       rec, rraw, err);
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

hipError_t set_rows_smem_limits() {
  const void* fns[] = {(const void*)k_owner_merge<true>, (const void*)k_owner_merge<false>,
                       (const void*)k_part_aggregate<true>, (const void*)k_part_aggregate<false>,
                       (const void*)k_part_hist, (const void*)k_part_scatter<true>, (const void*)k_part_scatter<false>};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - 2048);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
