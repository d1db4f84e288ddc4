// kernels_join.hip -- gfx950 kernels of the host/device correlation join
// (§3.1): device kernel records take the label (operator/shape key, app,
// serving phase) of the host record with their correlation id, else of the
// graph record with their anchor, else of the host operator interval on their
// stream that contains their start; labelled records become the events of
// the weighting path.
//
// A hash join: the host records go into two open-addressing tables in device
// memory (one per id space, keyed by the nonzero 64-bit id, linear probing;
// a slot is 16 bytes -- the id and the record index -- so that a probe reads
// one 16-byte piece of one cache line),
// one thread per kernel record probes them, and an interval is found by a
// binary search of the intervals (ascending by (stream, begin)).  The
// labelled records are then written in kernel-record order at positions from
// an exclusive scan of their flags.
#include "atrex_device.hpp"
#include "atrex_kernels.h"

namespace {

constexpr uint32_t kNoRef = 0xFFFFFFFFu;
constexpr uint32_t kRefInterval = 0x80000000u;  // ref bit: the label is an interval's (indices < 2^31)

__device__ __forceinline__ uint32_t id_slot(uint64_t id, uint32_t mask) {
  return hash32((uint32_t)id ^ hash32((uint32_t)(id >> 32))) & mask;
}

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
__global__ void k_join_probe(JoinKernels k, JoinTables t, JoinIntervals iv, uint8_t* __restrict__ source,
                             uint32_t* __restrict__ ref, uint32_t* __restrict__ flag,
                             unsigned long long* __restrict__ by, uint32_t* __restrict__ err) {
  __shared__ uint32_t s_by[4];
  if (threadIdx.x < 4) s_by[threadIdx.x] = 0;
  __syncthreads();
  const uint64_t e = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < k.n) {
    const int64_t st = k.start[e], en = k.end[e];
    uint32_t src = 3, r = kNoRef;
    if (en < st) {
      atomicOr(err, ATREX_ERRBIT_RANGE);
    } else {
      const uint64_t c = k.corr[e], a = k.anchor[e];
      if (c != 0) r = table_find(t.slot0, t.mask, c);
      if (r != kNoRef) {
        src = 0;
      } else {
        if (a != 0) r = table_find(t.slot1, t.mask, a);
        if (r != kNoRef) {
          src = 1;
        } else if (iv.n) {
          // the last interval with (stream, begin) <= (stream, start)
          const uint32_t sm = k.stream[e];
          uint64_t lo = 0, hi = iv.n;  // answer in [lo - 1, hi - 1]
          while (lo < hi) {
            const uint64_t mid = (lo + hi) / 2;
            const uint32_t ms = iv.stream[mid];
            if (ms < sm || (ms == sm && iv.begin[mid] <= st)) lo = mid + 1; else hi = mid;
          }
          if (lo > 0 && iv.stream[lo - 1] == sm && st < iv.end[lo - 1]) {
            src = 2;
            r = (uint32_t)(lo - 1) | kRefInterval;
          }
        }
      }
    }
    if (source) source[e] = (uint8_t)src;
    ref[e] = r;
    flag[e] = src < 3 ? 1u : 0u;
    atomicAdd(&s_by[src], 1u);
  }
  __syncthreads();
  if (threadIdx.x < 4 && s_by[threadIdx.x]) atomicAdd(&by[threadIdx.x], (unsigned long long)s_by[threadIdx.x]);
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
      hipLaunchKernelGGL(k_join_probe, dim3((uint32_t)((k.n + 255) / 256)), dim3(256), 0, s, k, t, iv, source, ref,
                         flag, words, err);
      exclusive_scan_u32(s, flag, pos, k.n, scan_tmp);
    }
  } else if (k.n) {  // the events
    hipLaunchKernelGGL(k_join_emit, dim3((uint32_t)((k.n + 255) / 256)), dim3(256), 0, s, k, h, iv, ref, flag, pos,
                       out, cap);
  }
}
