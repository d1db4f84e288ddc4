// kernels_small.hip -- single-workgroup ordering of few group rows (at most
// ROWS_N): one launch that reads the row count from device memory, so the
// call needs no intermediate host synchronisation; more rows leave a "not
// done" flag and the caller uses the radix-sort path.  Sorting is a bitonic
// network in LDS.
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

}  // namespace

uint32_t small_rows_n() { return ROWS_N; }

void launch_small_rows(hipStream_t s, const Rows& rows, const SortedGroups& out, unsigned long long* G_out,
                       uint32_t* done) {
  hipLaunchKernelGGL(k_small_rows, dim3(1), dim3(NT), 0, s, rows, out, G_out, done);
}
