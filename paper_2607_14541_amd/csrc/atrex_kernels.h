// atrex_kernels.h -- host-visible launchers of the gfx950 kernels (one per
// kernel family), and the plain structs passed to them by value.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

struct EventsDev {
  const uint32_t* key;
  const uint32_t* app;
  const uint8_t* phase;
  const int64_t* dur;
  uint64_t n;
};

// Global per-(dictionary slot, phase) accumulators.
struct GroupTables {
  unsigned long long* dict;  // [mask + 1] key + 1, 0 = free
  uint32_t dict_mask;
  unsigned long long* acc;   // [(mask + 1) * P][2] lo, hi (count in hi bits 33..)
  unsigned long long* raw;   // [(mask + 1) * P][2] or null
};

// Groups ordered by (key, phase).
struct SortedGroups {
  uint32_t* key;
  uint8_t* phase;
  uint64_t* count;
  uint64_t* wsum;  // [G][2]
  uint64_t* raw;   // [G][2] or null
};

// kernels_aggregate.hip
hipError_t set_kernel_smem_limits();
void launch_pass_a_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                       unsigned long long* partial, unsigned long long* carry, uint32_t* err);
void launch_pass_a_reduce(hipStream_t s, const unsigned long long* partial, uint32_t nb, uint32_t G,
                          const unsigned long long* carry, uint64_t* T);
void launch_pass_a_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                          unsigned long long* T, uint32_t* err);
void launch_unpack_scale(hipStream_t s, const uint64_t* sw, uint64_t G, uint64_t* mant, int32_t* rho);
void launch_scale(hipStream_t s, const uint64_t* T, const uint32_t* c, const uint64_t* Csum, uint32_t A,
                  uint32_t P, uint64_t* scale);
void launch_pass_b_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                          const GroupTables& gt, bool raw, uint32_t nblocks, uint32_t* err);
size_t pass_b_lds_smem(uint32_t P, bool raw, uint32_t slots_log2);
void launch_pass_b_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                       const GroupTables& gt, bool raw, uint32_t slots_log2, uint32_t nblocks, uint32_t* err);
void launch_compact(hipStream_t s, const GroupTables& gt, uint32_t P, uint64_t max_groups, uint64_t* sk,
                    uint32_t* src, unsigned long long* counter, uint32_t* err);
void launch_gather_groups(hipStream_t s, const uint64_t* sk, const uint32_t* src, uint64_t G, const GroupTables& gt,
                          bool raw, const SortedGroups& out);

// kernels_util.hip
void launch_fill_u64(hipStream_t s, uint64_t* p, uint64_t n, uint64_t v);
void launch_sum_u32(hipStream_t s, const uint32_t* x, uint64_t n, uint64_t* out);
// LSD radix sort of (u64 key, u32 value) pairs on key bits [0, bits).  Stable.
// tmp must hold radix_sort_tmp_bytes(n); results end in (k0, v0).
size_t radix_sort_tmp_bytes(uint64_t n);
void radix_sort_pairs(hipStream_t s, uint64_t* k0, uint32_t* v0, uint64_t* k1, uint32_t* v1, uint64_t n, int bits,
                      void* tmp);
// Exclusive scan of u32 (n < 2^32), in place capable; tmp from scan_tmp_bytes(n).
size_t scan_tmp_bytes(uint64_t n);
void exclusive_scan_u32(hipStream_t s, const uint32_t* in, uint32_t* out, uint64_t n, void* tmp);

// kernels_normalize.hip
struct UnitTable {
  uint32_t* id;        // [num] operator or key id, ascending
  uint64_t* U;         // [num][2]
  double* w;           // [num]
};
void launch_phase_totals(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t* partials,
                         uint32_t nb, uint64_t* S);
void launch_group_weights(hipStream_t s, const SortedGroups& g, uint64_t G, const uint64_t* S, uint32_t* okey,
                          uint8_t* oph, uint64_t* ocount, uint64_t* owsum, uint64_t* oraw, double* oweight,
                          uint64_t* oS, uint32_t P);
// Segments of equal unit (key >> shift) in sorted groups: flags + scan -> starts.
void launch_unit_heads(hipStream_t s, const uint32_t* key, uint64_t G, int shift, uint32_t* flags);
void launch_unit_starts(hipStream_t s, const uint32_t* flags, const uint32_t* scan, uint64_t G, uint32_t* starts);
void launch_unit_U(hipStream_t s, const SortedGroups& g, uint64_t G, const uint32_t* starts, uint64_t nunits,
                   int shift, uint32_t P, uint64_t L, UnitTable t);
void launch_sum_u128(hipStream_t s, const uint64_t* x, uint64_t n, uint64_t* partials, uint32_t nb, uint64_t* out);
void launch_unit_weights(hipStream_t s, UnitTable t, uint64_t nunits, const uint64_t* total);

// score
void launch_score_validate(hipStream_t s, const double* S, uint64_t n, uint32_t* err);
void launch_score_keys(hipStream_t s, const uint32_t* score_key, const double* S, uint64_t n, uint64_t* k_key,
                       uint64_t* k_sval, uint32_t* idx);
void launch_dup_check(hipStream_t s, const uint64_t* sorted_keys, uint64_t n, uint32_t* err);
void launch_heads_u64(hipStream_t s, const uint64_t* k, uint64_t n, uint32_t* flags);
void launch_score_opkeys(hipStream_t s, const uint32_t* score_key, const uint32_t* idx, uint64_t n,
                         uint64_t* k_op);
void launch_score_ops(hipStream_t s, const uint32_t* score_key, const double* S, const uint32_t* order,
                      const uint32_t* starts, uint64_t nops, uint64_t n, UnitTable opt, uint64_t nops_trace,
                      uint32_t* r_op, uint64_t* r_U, double* r_S);
void launch_score_final(hipStream_t s, const uint32_t* r_op, const uint64_t* r_U, const double* r_S,
                        uint64_t nops, const uint64_t* totalU, uint32_t* op, double* op_weight, double* op_score,
                        double* s_agg, uint32_t* err);
