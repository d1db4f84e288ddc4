// kernels_join.hip -- gfx950 kernels of the host/device correlation join
// (§3.1): device kernel records take the label (operator/shape key, app,
// serving phase) of the host record with their correlation id, else of the
// graph record with their anchor, else of the host operator interval on their
// stream that contains their start; labelled records become the events of
// the weighting path.
//
// Two methods find the host record of an id:
// - the hash join: the host records go into two open-addressing tables in
//   device memory (one per id space, keyed by the nonzero 64-bit id, linear
//   probing; a slot is 16 bytes -- the id and the record index -- so that a
//   probe reads one 16-byte piece of one cache line), and one thread per
//   kernel record probes them;
// - the partitioned join: the host records and the probes (a kernel record's
//   nonzero correlation id and anchor) are scattered by the top bits of the
//   id's hash into buckets small enough for two LDS tables, and one workgroup
//   per bucket builds its tables in LDS and answers its probes, writing the
//   host record's index beside each kernel record.  The random global
//   atomics and probes of the hash join become streaming passes.
// An interval is then found by a binary search of the intervals (ascending by
// (stream, begin)), and the labelled records are written in kernel-record
// order at positions from an exclusive scan of their flags.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t kNoRef = 0xFFFFFFFFu;
constexpr uint32_t kRefInterval = 0x80000000u;  // ref bit: the label is an interval's (indices < 2^31)

__device__ __forceinline__ uint32_t id_hash(uint64_t id) { return hash32((uint32_t)id ^ hash32((uint32_t)(id >> 32))); }
__device__ __forceinline__ uint32_t id_slot(uint64_t id, uint32_t mask) { return id_hash(id) & mask; }

// Host records into the tables (kind 0: correlation ids, kind 1: anchors).
// A kind above 1, an id of 0 or an id met twice in one kind flags
// ATREX_ERRBIT_DUP (the call then fails with INVALID_ARG).
__global__ void k_join_build(JoinHost h, JoinTables t, uint32_t* __restrict__ err) {
  const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= h.n) return;
  const uint32_t kind = h.kind[j];
  const uint64_t id = h.id[j];
  if (kind > 1 || id == 0) {
    atomicOr(err, ATREX_ERRBIT_DUP);
    return;
  }
  uint64_t* slot = kind ? t.slot1 : t.slot0;
  uint32_t s = id_slot(id, t.mask);
  for (uint32_t probe = 0; probe <= t.mask; ++probe) {  // each table has at least twice the records' slots
    const unsigned long long prev = atomicCAS((unsigned long long*)&slot[2 * s], 0ull, (unsigned long long)id);
    if (prev == 0) {
      slot[2 * s + 1] = j;
      return;
    }
    if (prev == id) {
      atomicOr(err, ATREX_ERRBIT_DUP);
      return;
    }
    s = (s + 1) & t.mask;
  }
}

// Intervals must ascend by (stream, begin), with begin <= end and no overlap
// on a stream.
__global__ void k_join_check_intervals(JoinIntervals iv, uint32_t* __restrict__ err) {
  const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= iv.n) return;
  bool ok = iv.end[j] >= iv.begin[j];
  if (j > 0) {
    const uint32_t s0 = iv.stream[j - 1], s1 = iv.stream[j];
    ok = ok && (s1 > s0 || (s1 == s0 && iv.begin[j] >= iv.end[j - 1]));
  }
  if (!ok) atomicOr(err, ATREX_ERRBIT_DUP);
}

__device__ __forceinline__ uint32_t table_find(const uint64_t* __restrict__ slot, uint32_t mask, uint64_t id) {
  uint32_t s = id_slot(id, mask);
  for (uint32_t probe = 0; probe <= mask; ++probe) {
    const v2l kv = *(const v2l*)&slot[2 * s];  // the id and the record index together
    if ((uint64_t)kv.x == id) return (uint32_t)kv.y;
    if (kv.x == 0) return kNoRef;
    s = (s + 1) & mask;
  }
  return kNoRef;
}

// One thread per kernel record: its source (0 correlation id, 1 anchor,
// 2 interval, 3 none), the record that labels it (ref: a host record's index,
// or an interval's index with kRefInterval), and its flag for the
// compaction.  end < start flags ATREX_ERRBIT_RANGE.
// PART: the host record of each id was found by the partitioned join and
// stands in ref0 (correlation id) and ref1 (anchor); kNoRef where none.
// The records that need an interval (about a tenth) are gathered in LDS and
// searched by the workgroup's first waves, all lanes busy, instead of by a
// few lanes of every wave.
constexpr uint32_t kProbeBlock = 1024;

template <bool PART>
__global__ __launch_bounds__(kProbeBlock) void k_join_probe(JoinKernels k, JoinTables t,
                                                            const uint32_t* __restrict__ ref0,
                                                            const uint32_t* __restrict__ ref1, JoinIntervals iv,
                                                            uint8_t* __restrict__ source, uint32_t* __restrict__ ref,
                                                            uint32_t* __restrict__ flag,
                                                            unsigned long long* __restrict__ by,
                                                            uint32_t* __restrict__ err) {
  __shared__ uint32_t s_by[4], s_nt;
  __shared__ uint32_t s_task[kProbeBlock];  // the block's records that need an interval search
  if (threadIdx.x < 4) s_by[threadIdx.x] = 0;
  if (threadIdx.x == 0) s_nt = 0;
  __syncthreads();
  const uint64_t e0 = (uint64_t)blockIdx.x * kProbeBlock;
  const uint64_t e = e0 + threadIdx.x;
  auto label = [&](uint64_t i, uint32_t src, uint32_t r) {
    if (source) source[i] = (uint8_t)src;
    ref[i] = r;
    flag[i] = src < 3 ? 1u : 0u;
    atomicAdd(&s_by[src], 1u);
  };
  bool search = false;
  if (e < k.n) {
    const int64_t st = k.start[e], en = k.end[e];
    uint32_t src = 3, r = kNoRef;
    if (en < st) {
      atomicOr(err, ATREX_ERRBIT_RANGE);
    } else {
      const uint64_t c = k.corr[e], a = k.anchor[e];
      if (c != 0) r = PART ? ref0[e] : table_find(t.slot0, t.mask, c);
      if (r != kNoRef) {
        src = 0;
      } else {
        if (a != 0) r = PART ? ref1[e] : table_find(t.slot1, t.mask, a);
        if (r != kNoRef) src = 1;
        else search = iv.n != 0;
      }
    }
    if (!search) label(e, src, r);
  }
  {  // wave-aggregated append to the block's search list
    const uint64_t bm = __ballot(search);
    if (bm) {
      const uint32_t lane = threadIdx.x & 63, leader = __ffsll((unsigned long long)bm) - 1;
      uint32_t base = 0;
      if (lane == leader) base = atomicAdd(&s_nt, (uint32_t)__popcll(bm));
      base = __shfl(base, leader, 64);
      if (search) s_task[base + __popcll(bm & ((1ull << lane) - 1ull))] = threadIdx.x;
    }
  }
  __syncthreads();
  const uint32_t nt = s_nt;
  for (uint32_t q = threadIdx.x; q < nt; q += kProbeBlock) {
    const uint64_t i = e0 + s_task[q];
    const int64_t st = k.start[i];
    const uint32_t sm = k.stream[i];
    // the last interval with (stream, begin) <= (stream, start)
    uint64_t lo = 0, hi = iv.n;  // answer in [lo - 1, hi - 1]
    while (lo < hi) {
      const uint64_t mid = (lo + hi) / 2;
      const uint32_t ms = iv.stream[mid];
      if (ms < sm || (ms == sm && iv.begin[mid] <= st)) lo = mid + 1; else hi = mid;
    }
    const bool in = lo > 0 && iv.stream[lo - 1] == sm && st < iv.end[lo - 1];
    label(i, in ? 2u : 3u, in ? ((uint32_t)(lo - 1) | kRefInterval) : kNoRef);
  }
  __syncthreads();
  if (threadIdx.x < 4 && s_by[threadIdx.x]) atomicAdd(&by[threadIdx.x], (unsigned long long)s_by[threadIdx.x]);
}

// ---------------------------------------------------------------------------
// The partitioned join.  The passes over host and kernel records split them
// into gridDim.x contiguous ranges; bucket of an id = the top bb bits of its
// hash, slot in the bucket's LDS table = the next kJoinSlotBits bits.
constexpr uint32_t kJoinSlotBits = 12, kJoinSlots = 1u << kJoinSlotBits;  // per id space per bucket

__device__ __forceinline__ void join_range(uint64_t n, uint64_t& b, uint64_t& e) {
  const uint64_t per = (n + gridDim.x - 1) / gridDim.x;
  b = min(n, (uint64_t)blockIdx.x * per);
  e = min(n, b + per);
}

// Host records per bucket (records of kind > 1 or id 0 are not counted and
// flag ATREX_ERRBIT_DUP); H[bucket * gridDim.x + w].
__global__ __launch_bounds__(1024) void k_jp_hist_host(JoinHost h, uint32_t bb, uint32_t* __restrict__ H,
                                                       uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s_c[];  // [2^bb]
  const uint32_t NB = 1u << bb, sh = 32 - bb;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_c[i] = 0;
  __syncthreads();
  uint64_t b, e;
  join_range(h.n, b, e);
  bool bad = false;
  for (uint64_t j = b + threadIdx.x; j < e; j += blockDim.x) {
    const uint32_t kind = h.kind[j];
    const uint64_t id = h.id[j];
    if (kind > 1 || id == 0) {
      bad = true;
      continue;
    }
    atomicAdd(&s_c[id_hash(id) >> sh], 1u);
  }
  if (bad) atomicOr(err, ATREX_ERRBIT_DUP);
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) H[(size_t)i * gridDim.x + blockIdx.x] = s_c[i];
}

// The counted host records as (id, index << 1 | kind) at their bucket's
// positions O (exclusive scan of H).
__global__ __launch_bounds__(1024) void k_jp_scatter_host(JoinHost h, uint32_t bb, const uint32_t* __restrict__ O,
                                                          uint64_t* __restrict__ rec) {
  extern __shared__ uint32_t s_cur[];  // [2^bb]
  const uint32_t NB = 1u << bb, sh = 32 - bb;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_cur[i] = O[(size_t)i * gridDim.x + blockIdx.x];
  __syncthreads();
  uint64_t b, e;
  join_range(h.n, b, e);
  for (uint64_t j = b + threadIdx.x; j < e; j += blockDim.x) {
    const uint32_t kind = h.kind[j];
    const uint64_t id = h.id[j];
    if (kind > 1 || id == 0) continue;
    const uint32_t pos = atomicAdd(&s_cur[id_hash(id) >> sh], 1u);
    v2l r;
    r.x = (long long)id;
    r.y = (long long)(((uint64_t)j << 1) | kind);
    *(v2l*)(rec + 2 * (size_t)pos) = r;
  }
}

// Probes per bucket: a kernel record's nonzero correlation id (kind 0) and
// nonzero anchor (kind 1).  end < start flags ATREX_ERRBIT_RANGE.
__global__ __launch_bounds__(1024) void k_jp_hist_probe(JoinKernels k, uint32_t bb, uint32_t* __restrict__ H,
                                                        uint32_t* __restrict__ err) {
  extern __shared__ uint32_t s_c[];
  const uint32_t NB = 1u << bb, sh = 32 - bb;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_c[i] = 0;
  __syncthreads();
  uint64_t b, e;
  join_range(k.n, b, e);
  bool bad = false;
  for (uint64_t j = b + threadIdx.x; j < e; j += blockDim.x) {
    bad |= k.end[j] < k.start[j];
    const uint64_t c = k.corr[j], a = k.anchor[j];
    if (c) atomicAdd(&s_c[id_hash(c) >> sh], 1u);
    if (a) atomicAdd(&s_c[id_hash(a) >> sh], 1u);
  }
  if (bad) atomicOr(err, ATREX_ERRBIT_RANGE);
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) H[(size_t)i * gridDim.x + blockIdx.x] = s_c[i];
}

__global__ __launch_bounds__(1024) void k_jp_scatter_probe(JoinKernels k, uint32_t bb, const uint32_t* __restrict__ O,
                                                           uint64_t* __restrict__ rec) {
  extern __shared__ uint32_t s_cur[];
  const uint32_t NB = 1u << bb, sh = 32 - bb;
  for (uint32_t i = threadIdx.x; i < NB; i += blockDim.x) s_cur[i] = O[(size_t)i * gridDim.x + blockIdx.x];
  __syncthreads();
  uint64_t b, e;
  join_range(k.n, b, e);
  for (uint64_t j = b + threadIdx.x; j < e; j += blockDim.x) {
    const uint64_t ids[2] = {k.corr[j], k.anchor[j]};
#pragma unroll
    for (uint32_t kind = 0; kind < 2; ++kind) {
      if (!ids[kind]) continue;
      const uint32_t pos = atomicAdd(&s_cur[id_hash(ids[kind]) >> sh], 1u);
      v2l r;
      r.x = (long long)ids[kind];
      r.y = (long long)((j << 1) | kind);
      *(v2l*)(rec + 2 * (size_t)pos) = r;
    }
  }
}

// One workgroup per bucket: its host records into two LDS tables (one per id
// space; open addressing over kJoinSlots slots, id 0 = free), then its probes
// answered: ref0[e] / ref1[e] = the host record's index.  An id met twice in
// a space flags ATREX_ERRBIT_DUP; a table that fills up flags
// ATREX_ERRBIT_SPILL (the host then runs the hash join instead).  Hh/Oh and
// Hp/Op: counts and positions of the host records and probes, [bucket][nw].
__global__ __launch_bounds__(1024) void k_jp_bucket(const uint64_t* __restrict__ hrec, const uint32_t* __restrict__ Hh,
                                                    const uint32_t* __restrict__ Oh, const uint64_t* __restrict__ prec,
                                                    const uint32_t* __restrict__ Hp, const uint32_t* __restrict__ Op,
                                                    uint32_t nw, uint32_t bb, uint32_t* __restrict__ ref0,
                                                    uint32_t* __restrict__ ref1, uint32_t* __restrict__ err) {
  extern __shared__ unsigned long long s_id[];                  // [2][kJoinSlots]
  uint32_t* s_ix = (uint32_t*)(s_id + 2 * kJoinSlots);          // [2][kJoinSlots]
  const uint32_t bk = blockIdx.x, sh = 32 - bb - kJoinSlotBits;
  for (uint32_t i = threadIdx.x; i < 2 * kJoinSlots; i += blockDim.x) s_id[i] = 0;
  __syncthreads();
  const size_t c0 = (size_t)bk * nw, c1 = c0 + nw - 1;
  const uint32_t hs = Oh[c0], he = Oh[c1] + Hh[c1];
  bool dup = false, full = false;
  for (uint32_t i = hs + threadIdx.x; i < he; i += blockDim.x) {
    const uint64_t id = hrec[2 * (size_t)i], v = hrec[2 * (size_t)i + 1];
    const uint32_t kind = (uint32_t)v & 1u;
    unsigned long long* tid_ = s_id + kind * kJoinSlots;
    uint32_t sl = (id_hash(id) >> sh) & (kJoinSlots - 1);
    uint32_t probe = 0;
    for (; probe < kJoinSlots; ++probe) {
      const unsigned long long prev = atomicCAS(&tid_[sl], 0ull, (unsigned long long)id);
      if (prev == 0) {
        s_ix[kind * kJoinSlots + sl] = (uint32_t)(v >> 1);
        break;
      }
      if (prev == id) {
        dup = true;
        break;
      }
      sl = (sl + 1) & (kJoinSlots - 1);
    }
    full |= probe == kJoinSlots;
  }
  if (dup) atomicOr(err, ATREX_ERRBIT_DUP);
  if (full) atomicOr(err, ATREX_ERRBIT_SPILL);
  __syncthreads();
  const uint32_t ps = Op[c0], pe = Op[c1] + Hp[c1];
  for (uint32_t i = ps + threadIdx.x; i < pe; i += blockDim.x) {
    const uint64_t id = prec[2 * (size_t)i], v = prec[2 * (size_t)i + 1];
    const uint32_t kind = (uint32_t)v & 1u;
    const unsigned long long* tid_ = s_id + kind * kJoinSlots;
    uint32_t sl = (id_hash(id) >> sh) & (kJoinSlots - 1);
    for (uint32_t probe = 0; probe < kJoinSlots; ++probe) {
      const unsigned long long x = tid_[sl];
      if (x == id) {
        (kind ? ref1 : ref0)[v >> 1] = s_ix[kind * kJoinSlots + sl];
        break;
      }
      if (x == 0) break;
      sl = (sl + 1) & (kJoinSlots - 1);
    }
  }
}

// The labelled records as events, in kernel-record order.
__global__ void k_join_emit(JoinKernels k, JoinHost h, JoinIntervals iv, const uint32_t* __restrict__ ref,
                            const uint32_t* __restrict__ flag, const uint32_t* __restrict__ pos, JoinOut out,
                            uint64_t cap) {
  const uint64_t e = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= k.n || !flag[e]) return;
  const uint32_t p = pos[e], r = ref[e] & ~kRefInterval;
  if (p >= cap) return;
  if (ref[e] & kRefInterval) {
    out.key[p] = iv.key[r];
    out.app[p] = iv.app[r];
    out.phase[p] = iv.phase[r];
  } else {
    out.key[p] = h.key[r];
    out.app[p] = h.app[r];
    out.phase[p] = h.phase[r];
  }
  out.dur[p] = k.end[e] - k.start[e];
}

}  // namespace

void launch_join(hipStream_t s, const JoinKernels& k, const JoinHost& h, const JoinIntervals& iv,
                 const JoinTables& t, uint8_t* source, uint32_t* ref, uint32_t* flag, uint32_t* pos, void* scan_tmp,
                 const JoinOut& out, uint64_t cap, unsigned long long* words, uint32_t* err, int stage) {
  if (stage == 0) {  // tables and checks
    launch_fill_u64(s, t.slot0, 2 * ((uint64_t)t.mask + 1), 0);
    launch_fill_u64(s, t.slot1, 2 * ((uint64_t)t.mask + 1), 0);
    if (h.n) hipLaunchKernelGGL(k_join_build, dim3((uint32_t)((h.n + 255) / 256)), dim3(256), 0, s, h, t, err);
    if (iv.n)
      hipLaunchKernelGGL(k_join_check_intervals, dim3((uint32_t)((iv.n + 255) / 256)), dim3(256), 0, s, iv, err);
    if (k.n) {
      hipLaunchKernelGGL(k_join_probe<false>, dim3((uint32_t)((k.n + kProbeBlock - 1) / kProbeBlock)),
                         dim3(kProbeBlock), 0, s, k, t, nullptr, nullptr, iv, source, ref, flag, words, err);
      exclusive_scan_u32(s, flag, pos, k.n, scan_tmp);
    }
  } else if (k.n) {  // the events
    hipLaunchKernelGGL(k_join_emit, dim3((uint32_t)((k.n + 255) / 256)), dim3(256), 0, s, k, h, iv, ref, flag, pos,
                       out, cap);
  }
}

uint32_t join_part_bucket_bits(uint64_t nh) {
  uint32_t bb = kJoinMinBucketBits;
  while (bb < kJoinMaxBucketBits && ((nh + (1ull << bb) - 1) >> bb) > kJoinBucketHost) ++bb;
  return bb;
}

size_t join_part_bytes(uint64_t nk, uint64_t nh, uint32_t bb) {
  const size_t m = ((size_t)1 << bb) * kJoinPartWG * 4;
  return nh * 16 + 2 * nk * 16 + 2 * nk * 4 + 4 * m + 8 * 256;  // eight pieces, each 256-byte aligned
}

void launch_join_part(hipStream_t s, const JoinKernels& k, const JoinHost& h, const JoinIntervals& iv, uint32_t bb,
                      void* part, uint8_t* source, uint32_t* ref, uint32_t* flag, uint32_t* pos, void* scan_tmp,
                      unsigned long long* words, uint32_t* err) {
  const size_t m = ((size_t)1 << bb) * kJoinPartWG;
  char* p = (char*)part;
  auto take = [&](size_t bytes) {
    char* at = p;
    p += (bytes + 255) / 256 * 256;
    return at;
  };
  uint64_t* hrec = (uint64_t*)take(h.n * 16);
  uint64_t* prec = (uint64_t*)take(2 * k.n * 16);
  uint32_t* ref0 = (uint32_t*)take(k.n * 4);
  uint32_t* ref1 = (uint32_t*)take(k.n * 4);
  uint32_t* Hh = (uint32_t*)take(m * 4);
  uint32_t* Oh = (uint32_t*)take(m * 4);
  uint32_t* Hp = (uint32_t*)take(m * 4);
  uint32_t* Op = (uint32_t*)take(m * 4);
  const size_t cnt_smem = (size_t)4 << bb;
  launch_fill_u32(s, ref0, k.n, kNoRef);
  launch_fill_u32(s, ref1, k.n, kNoRef);
  hipLaunchKernelGGL(k_jp_hist_host, dim3(kJoinPartWG), dim3(1024), cnt_smem, s, h, bb, Hh, err);
  exclusive_scan_u32(s, Hh, Oh, m, scan_tmp);
  hipLaunchKernelGGL(k_jp_scatter_host, dim3(kJoinPartWG), dim3(1024), cnt_smem, s, h, bb, Oh, hrec);
  hipLaunchKernelGGL(k_jp_hist_probe, dim3(kJoinPartWG), dim3(1024), cnt_smem, s, k, bb, Hp, err);
  exclusive_scan_u32(s, Hp, Op, m, scan_tmp);
  hipLaunchKernelGGL(k_jp_scatter_probe, dim3(kJoinPartWG), dim3(1024), cnt_smem, s, k, bb, Op, prec);
  hipLaunchKernelGGL(k_jp_bucket, dim3(1u << bb), dim3(1024), (size_t)2 * kJoinSlots * 12, s, hrec, Hh, Oh, prec, Hp,
                     Op, kJoinPartWG, bb, ref0, ref1, err);
  if (iv.n)
    hipLaunchKernelGGL(k_join_check_intervals, dim3((uint32_t)((iv.n + 255) / 256)), dim3(256), 0, s, iv, err);
  if (k.n) {
    const JoinTables none{};
    hipLaunchKernelGGL(k_join_probe<true>, dim3((uint32_t)((k.n + kProbeBlock - 1) / kProbeBlock)),
                       dim3(kProbeBlock), 0, s, k, none, ref0, ref1, iv, source, ref, flag, words, err);
    exclusive_scan_u32(s, flag, pos, k.n, scan_tmp);
  }
}

hipError_t set_join_smem_limits() {
  const void* fns[] = {(const void*)k_jp_hist_host, (const void*)k_jp_scatter_host, (const void*)k_jp_hist_probe,
                       (const void*)k_jp_scatter_probe, (const void*)k_jp_bucket};
  for (const void* f : fns) {
    const hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, 128 * 1024);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
