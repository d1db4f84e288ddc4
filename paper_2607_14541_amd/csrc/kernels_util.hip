// kernels_util.hip -- fills, a u32 exclusive scan and an LSD radix sort of
// (u64 key, u32 value) pairs for gfx950 (wave64).
//
// Radix sort: 8-bit digits, tiles of 2048 items (256 threads x 8 rounds).
// Per pass: tile digit histograms -> one exclusive scan over the digit-major
// histogram -> stable scatter.  Within a round the rank of an item among the
// tile's earlier items with the same digit comes from eight wave ballots
// (lanes with an equal digit), per-wave digit counts in LDS, and a running
// per-digit count carried across rounds.
#include <algorithm>
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr int RS_BLOCK = 256;
constexpr int RS_ROUNDS = 8;
constexpr int RS_TILE = RS_BLOCK * RS_ROUNDS;
constexpr int RS_WAVES = RS_BLOCK / 64;

constexpr int SC_BLOCK = 256;
constexpr int SC_ITEMS = 8;
constexpr int SC_TILE = SC_BLOCK * SC_ITEMS;

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint64_t n, uint32_t v) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_copy_u32(uint32_t* __restrict__ dst, const uint32_t* __restrict__ src, uint64_t n) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ void k_fill_u64(uint64_t* __restrict__ p, uint64_t n, uint64_t v) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Copies of device status words into the context's host-mapped pinned buffer
// (one launch for every readback of a call, in place of one copy each).
// Lane l copies words l, l + 64, ... of the concatenated ranges; each lane's
// loads are all issued before its stores, so the copy costs one load latency.
constexpr uint32_t kPublishWordsPerLane = 8;

__global__ void k_publish(PublishList pl, uint32_t* __restrict__ dst, uint32_t* done, uint32_t seq) {
  uint32_t v[kPublishWordsPerLane], at[kPublishWordsPerLane];
  uint32_t e = 0, before = 0;  // range of word w, and the words of the ranges before it
#pragma unroll
  for (uint32_t k = 0; k < kPublishWordsPerLane; ++k) {
    const uint32_t w = threadIdx.x + 64 * k;
    while (e < pl.count && w >= before + pl.n32[e]) before += pl.n32[e++];
    at[k] = ~0u;
    if (e < pl.count) {
      v[k] = pl.src[e][w - before];
      at[k] = pl.off32[e] + (w - before);
    }
  }
#pragma unroll
  for (uint32_t k = 0; k < kPublishWordsPerLane; ++k)
    if (at[k] != ~0u) dst[at[k]] = v[k];
  for (uint32_t w = threadIdx.x + 64 * kPublishWordsPerLane;; w += 64) {  // more than 512 words
    while (e < pl.count && w >= before + pl.n32[e]) before += pl.n32[e++];
    if (e >= pl.count) break;
    dst[pl.off32[e] + (w - before)] = pl.src[e][w - before];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence_system();
    __hip_atomic_store(done, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

__global__ void k_sum_u32(const uint32_t* __restrict__ x, uint64_t n, uint64_t* __restrict__ out) {
  __shared__ uint64_t s[1024 / 64];
  uint64_t acc = 0;
  for (uint64_t i = threadIdx.x; i < n; i += blockDim.x) acc += x[i];
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_down((unsigned long long)acc, d, 64);
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (uint32_t w = 0; w < blockDim.x / 64; ++w) t += s[w];
    *out = t;
  }
}

// ---------------------------------------------------------------- scan
// Block-local exclusive scan of SC_TILE items (blocked: thread t owns items
// [t * SC_ITEMS, (t + 1) * SC_ITEMS) of the tile); block totals to sums[].
__global__ __launch_bounds__(SC_BLOCK) void k_scan_local(const uint32_t* in, uint32_t* out, uint64_t n,
                                                         uint32_t* __restrict__ sums) {
  __shared__ uint32_t s_w[SC_BLOCK / 64];
  const uint64_t base = (uint64_t)blockIdx.x * SC_TILE + (uint64_t)threadIdx.x * SC_ITEMS;
  uint32_t v[SC_ITEMS];
  uint32_t tsum = 0;
#pragma unroll
  for (int i = 0; i < SC_ITEMS; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0u;
    tsum += v[i];
  }
  // inclusive wave scan of thread sums
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = tsum;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(inc, d, 64);
    if (lane >= (uint32_t)d) inc += y;
  }
  if (lane == 63) s_w[wave] = inc;
  __syncthreads();
  uint32_t woff = 0, total = 0;
  for (int w = 0; w < SC_BLOCK / 64; ++w) {
    if (w < (int)wave) woff += s_w[w];
    total += s_w[w];
  }
  uint32_t run = woff + inc - tsum;
#pragma unroll
  for (int i = 0; i < SC_ITEMS; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ void k_scan_add(uint32_t* __restrict__ out, uint64_t n, const uint32_t* __restrict__ sums) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] += sums[i / SC_TILE];
}

// ---------------------------------------------------------------- radix sort
__global__ __launch_bounds__(RS_BLOCK) void k_rs_hist(const uint64_t* __restrict__ k, uint64_t n, int shift,
                                                      uint32_t ntiles, uint32_t* __restrict__ hist) {
  __shared__ uint32_t s_c[256];
  s_c[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t base = (uint64_t)blockIdx.x * RS_TILE;
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const uint64_t i = base + (uint64_t)r * RS_BLOCK + threadIdx.x;
    if (i < n) atomicAdd(&s_c[(k[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[(size_t)threadIdx.x * ntiles + blockIdx.x] = s_c[threadIdx.x];
}

__global__ __launch_bounds__(RS_BLOCK) void k_rs_scatter(const uint64_t* __restrict__ kin,
                                                         const uint32_t* __restrict__ vin,
                                                         uint64_t* __restrict__ kout, uint32_t* __restrict__ vout,
                                                         uint64_t n, int shift, uint32_t ntiles,
                                                         const uint32_t* __restrict__ offs) {
  __shared__ uint32_t s_goff[256];
  __shared__ uint32_t s_run[256];
  __shared__ uint32_t s_wc[RS_WAVES * 256];
  s_goff[threadIdx.x] = offs[(size_t)threadIdx.x * ntiles + blockIdx.x];
  s_run[threadIdx.x] = 0;
  for (int w = 0; w < RS_WAVES; ++w) s_wc[w * 256 + threadIdx.x] = 0;
  __syncthreads();
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t lt = (1ull << lane) - 1ull;
  const uint64_t base = (uint64_t)blockIdx.x * RS_TILE;
  for (int r = 0; r < RS_ROUNDS; ++r) {
    const uint64_t i = base + (uint64_t)r * RS_BLOCK + threadIdx.x;
    const bool valid = i < n;
    uint64_t key = 0;
    uint32_t val = 0, d = 0;
    if (valid) {
      key = kin[i];
      val = vin[i];
      d = (uint32_t)(key >> shift) & 255u;
    }
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      m &= bit ? bb : ~bb;
    }
    const uint32_t lrank = __popcll(m & lt);
    if (valid && lrank == 0) s_wc[wave * 256 + d] = __popcll(m);
    __syncthreads();
    if (valid) {
      uint32_t off = s_run[d];
      for (uint32_t w = 0; w < wave; ++w) off += s_wc[w * 256 + d];
      const uint32_t dst = s_goff[d] + off + lrank;
      kout[dst] = key;
      vout[dst] = val;
    }
    __syncthreads();
    {
      uint32_t add = 0;
      for (int w = 0; w < RS_WAVES; ++w) {
        add += s_wc[w * 256 + threadIdx.x];
        s_wc[w * 256 + threadIdx.x] = 0;
      }
      s_run[threadIdx.x] += add;
    }
    __syncthreads();
  }
}

uint64_t cdiv(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

}  // namespace

void launch_fill_u64(hipStream_t s, uint64_t* p, uint64_t n, uint64_t v) {
  if (n == 0) return;
  uint64_t nb = cdiv(n, 256);
  if (nb > 8192) nb = 8192;
  hipLaunchKernelGGL(k_fill_u64, dim3((uint32_t)nb), dim3(256), 0, s, p, n, v);
}

void launch_fill_u32(hipStream_t s, uint32_t* p, uint64_t n, uint32_t v) {
  if (n == 0) return;
  const uint64_t nb = std::min<uint64_t>(cdiv(n, 256), 8192);
  hipLaunchKernelGGL(k_fill_u32, dim3((uint32_t)nb), dim3(256), 0, s, p, n, v);
}

void launch_copy_u32(hipStream_t s, uint32_t* dst, const uint32_t* src, uint64_t n) {
  if (n == 0) return;
  const uint64_t nb = std::min<uint64_t>(cdiv(n, 256), 8192);
  hipLaunchKernelGGL(k_copy_u32, dim3((uint32_t)nb), dim3(256), 0, s, dst, src, n);
}

void launch_publish(hipStream_t s, const PublishList& pl, uint32_t* dst, uint32_t* done, uint32_t seq) {
  hipLaunchKernelGGL(k_publish, dim3(1), dim3(64), 0, s, pl, dst, done, seq);
}

void launch_sum_u32(hipStream_t s, const uint32_t* x, uint64_t n, uint64_t* out) {
  hipLaunchKernelGGL(k_sum_u32, dim3(1), dim3(1024), 0, s, x, n, out);
}

size_t scan_tmp_bytes(uint64_t n) {
  size_t b = 0;
  while (n > 1) {
    n = cdiv(n, SC_TILE);
    b += ((n * 4 + 255) / 256) * 256;
  }
  return b + 256;
}

void exclusive_scan_u32(hipStream_t s, const uint32_t* in, uint32_t* out, uint64_t n, void* tmp) {
  if (n == 0) return;
  const uint64_t nb = cdiv(n, SC_TILE);
  uint32_t* sums = (uint32_t*)tmp;
  hipLaunchKernelGGL(k_scan_local, dim3((uint32_t)nb), dim3(SC_BLOCK), 0, s, in, out, n, sums);
  if (nb > 1) {
    char* next = (char*)tmp + ((nb * 4 + 255) / 256) * 256;
    exclusive_scan_u32(s, sums, sums, nb, next);
    hipLaunchKernelGGL(k_scan_add, dim3((uint32_t)cdiv(n, 256)), dim3(256), 0, s, out, n, sums);
  }
}

size_t radix_sort_tmp_bytes(uint64_t n) {
  const uint64_t ntiles = cdiv(n > 0 ? n : 1, RS_TILE);
  const uint64_t h = 256 * ntiles;
  return ((h * 4 + 255) / 256) * 256 * 2 + scan_tmp_bytes(h);
}

void radix_sort_pairs(hipStream_t s, uint64_t* k0, uint32_t* v0, uint64_t* k1, uint32_t* v1, uint64_t n, int bits,
                      void* tmp) {
  if (n <= 1 || bits <= 0) return;
  const uint32_t ntiles = (uint32_t)cdiv(n, RS_TILE);
  const uint64_t h = 256ull * ntiles;
  uint32_t* hist = (uint32_t*)tmp;
  uint32_t* offs = (uint32_t*)((char*)tmp + ((h * 4 + 255) / 256) * 256);
  void* stmp = (char*)tmp + ((h * 4 + 255) / 256) * 256 * 2;
  const int passes = (bits + 7) / 8;
  uint64_t *ki = k0, *ko = k1;
  uint32_t *vi = v0, *vo = v1;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    hipLaunchKernelGGL(k_rs_hist, dim3(ntiles), dim3(RS_BLOCK), 0, s, ki, n, shift, ntiles, hist);
    exclusive_scan_u32(s, hist, offs, h, stmp);
    hipLaunchKernelGGL(k_rs_scatter, dim3(ntiles), dim3(RS_BLOCK), 0, s, ki, vi, ko, vo, n, shift, ntiles, offs);
    uint64_t* tk = ki; ki = ko; ko = tk;
    uint32_t* tv = vi; vi = vo; vo = tv;
  }
  if (ki != k0) {  // odd number of passes: copy back
    (void)hipMemcpyAsync(k0, ki, n * sizeof(uint64_t), hipMemcpyDeviceToDevice, s);
    (void)hipMemcpyAsync(v0, vi, n * sizeof(uint32_t), hipMemcpyDeviceToDevice, s);
  }
}
