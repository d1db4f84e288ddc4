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

#define ATREX_OWNERS 256  // owner regions of the LDS engine (top byte of the key hash)

// Group rows: sort key = key << 3 | phase, accumulator X = lo + hi * 2^64 with
// hi = floor(W / 2^64) + count * 2^33, optional raw time (rlo, rhi).
struct Rows {
  uint64_t* rk;
  uint64_t* lo;
  uint64_t* hi;
  uint64_t* rlo;
  uint64_t* rhi;
  unsigned long long* count;
  uint64_t cap;
};

// LDS engine output: per (workgroup, owner) up to capo table rows.
struct OwnerRegions {
  uint32_t* key;    // [nwg][ATREX_OWNERS][capo]
  uint64_t* acc;    // [nwg][ATREX_OWNERS][capo][P][2]
  uint64_t* raw;    // same shape or null
  uint32_t* count;  // [nwg][ATREX_OWNERS]
  uint32_t capo;
};

// Input of the radix-partition engine: events [w * per, (w + 1) * per) per
// workgroup, or the LDS engine's spill regions.
struct PartSource {
  EventsDev ev;
  uint64_t per;
  const uint32_t* skey;
  const uint64_t* sval;
  const uint64_t* sraw;
  const uint32_t* scount;
  uint32_t scap;
  bool spill;
};

// The hot scatter's partition histogram as a side job of another kernel:
// range w = [w per, (w + 1) per) of key[0, n) (per a multiple of 4), its keys
// not in the seeded image (S slots, one bucket per key) counted per bucket
// (top BB bits of hash32) into H[bucket * nwg + w].
struct HistJob {
  const uint32_t* key;
  uint64_t n, per;
  uint32_t nwg, BB, S;
  const uint32_t* seed;
  uint32_t* H;
};

// Per-owner sorted group lists written by the owner merge of the LDS engine.
struct OwnerLists {
  uint64_t* rk;      // [ATREX_OWNERS][cap] sort keys key << 3 | phase, ascending within an owner
  uint32_t* dkey;    // every list's row keys (rk >> 3), densely and in no particular order
  unsigned long long* dcount;  // entries of dkey (zero before the owner merge)
  uint64_t* lo;      // accumulator low words
  uint64_t* hi;      // accumulator high words (W >> 64 | count << 33)
  uint64_t* rlo;     // raw time, nullable
  uint64_t* rhi;
  uint32_t* count;   // [ATREX_OWNERS] rows per owner
  uint64_t* part;    // [ATREX_OWNERS][P][2] per-phase partial sums of W
  uint32_t cap;      // rows per owner
};

// Spill records of the LDS engine as read back by the owner merge.
struct SpillIn {
  const uint32_t* key;
  const uint64_t* val;    // (share lo, share hi | phase << 40)
  const uint64_t* raw;    // nullable
  const uint32_t* count;  // [nwg]
  uint32_t cap;           // records per workgroup region
  uint32_t nwg;
  uint32_t inline_max;    // merged by the owners when the total is at most this
};

// Groups ordered by (key, phase).
struct SortedGroups {
  uint32_t* key;
  uint8_t* phase;
  uint64_t* count;
  uint64_t* wsum;  // [G][2]
  uint64_t* raw;   // [G][2] or null
};

// Outputs of the target-DSL share (DEVICE arrays of the caller).
struct ShareOut {
  uint32_t* key;       // [K]
  uint64_t* count;     // [K]
  uint64_t* dsl;       // [K][2]
  uint64_t* total;     // [K][2]
  double* share;       // [K]
  uint32_t* op;        // [I]
  uint32_t* op_shapes; // [I]
  double* op_share;    // [I]
};

// Observed runtime per unit (kernels_stats.hip): the unit lookup table
// (open addressing, key = (key << 3 | phase) + 1, 0 = free), the caller's
// outputs, and the requested quantiles (1e-5 steps).
struct StatsTable {
  uint64_t* key;  // [mask + 1]
  uint32_t* val;  // [mask + 1] unit index
  uint32_t mask;
};
struct StatsOut {
  uint32_t* key;
  uint8_t* phase;
  uint64_t* count;
  uint64_t* total;  // [U][2]
  double* mean;
  int64_t* min;
  int64_t* max;
  int64_t* quant;   // [U][nq]
};
struct StatsQ {
  uint32_t q[8];
  uint32_t n;
};
hipError_t set_stats_smem_limits();
uint32_t stats_small_max();
uint32_t stats_sel_chunk();
// unit heads, unit indices (scan), unit identity / count / total / mean, the
// per-unit counts and the lookup table; words[0] = number of units
void launch_stats_units(hipStream_t s, const SortedGroups& g, uint64_t G, bool by_phase, uint32_t* head,
                        uint32_t* uidx, void* scan_tmp, const StatsOut& out, uint64_t cap, uint32_t* ucount,
                        const StatsTable& t, unsigned long long* words);
// durations into their units' blocks; words[1] = the largest duration
void launch_stats_scatter(hipStream_t s, const EventsDev& ev, uint32_t P, bool by_phase, bool vec, uint32_t nblocks,
                          const StatsTable& t, const uint32_t* seg_start, uint32_t* cursor, int64_t* vals,
                          unsigned long long* words, uint32_t* err);
// the same placement in two passes with per-workgroup LDS counters (U <=
// stats_dense_units(); mat: U x nblocks counts, scanned in place)
uint32_t stats_dense_units();
void launch_stats_dense(hipStream_t s, const EventsDev& ev, uint32_t P, bool by_phase, bool vec, uint32_t nblocks,
                        const StatsTable& t, uint32_t U, uint32_t* mat, void* scan_tmp, const uint32_t* seg_start,
                        int64_t* vals, unsigned long long* words, uint32_t* err);
// units by size into three lists; words[2..4] = their lengths
void launch_stats_classify(hipStream_t s, const uint32_t* ucount, uint64_t U, uint32_t* tiny, uint32_t* small,
                           uint32_t* large, unsigned long long* words);
void launch_stats_sorts(hipStream_t s, const uint32_t* tiny, uint64_t ntiny, const uint32_t* small, uint64_t nsmall,
                        const uint32_t* seg_start, const int64_t* vals, const StatsQ& q, const StatsOut& out,
                        uint64_t cap);
// radix select over a batch of large units: state, chunk counts (into
// ccount[0..nb), scanned by the caller), rounds, outputs
void launch_select_init(hipStream_t s, const uint32_t* lu, uint32_t nb, const uint32_t* seg_start, const StatsQ& q,
                        uint64_t* prefix, uint32_t* want, uint32_t* ccount);
void launch_select_round(hipStream_t s, const uint32_t* lu, uint32_t nb, const uint32_t* cstart, uint32_t nchunks,
                         const uint32_t* seg_start, const int64_t* vals, uint32_t T, int shift, uint64_t* prefix,
                         uint32_t* want, uint32_t* hist);
void launch_select_out(hipStream_t s, const uint32_t* lu, uint32_t nb, const StatsQ& q, const uint64_t* prefix,
                       const StatsOut& out, uint64_t cap);

// Host/device correlation join (kernels_join.hip).
struct JoinKernels {
  const uint64_t* corr;
  const uint64_t* anchor;
  const uint32_t* stream;
  const int64_t* start;
  const int64_t* end;
  uint64_t n;
};
struct JoinHost {
  const uint8_t* kind;
  const uint64_t* id;
  const uint32_t* key;
  const uint32_t* app;
  const uint8_t* phase;
  uint64_t n;
};
struct JoinIntervals {
  const uint32_t* stream;
  const int64_t* begin;
  const int64_t* end;
  const uint32_t* key;
  const uint32_t* app;
  const uint8_t* phase;
  uint64_t n;
};
struct JoinTables {  // open addressing, 16-byte slots (id, record index), id 0 = free; one table per id space
  uint64_t* slot0;
  uint64_t* slot1;
  uint32_t mask;
};
struct JoinOut {
  uint32_t* key;
  uint32_t* app;
  uint8_t* phase;
  int64_t* dur;
};
// The hash join.  stage 0: tables, checks, probe and the scan of the flags
// (words[0..3]: records per source); stage 1: the labelled events
void launch_join(hipStream_t s, const JoinKernels& k, const JoinHost& h, const JoinIntervals& iv,
                 const JoinTables& t, uint8_t* source, uint32_t* ref, uint32_t* flag, uint32_t* pos, void* scan_tmp,
                 const JoinOut& out, uint64_t cap, unsigned long long* words, uint32_t* err, int stage);
// The partitioned join: 2^bb buckets of at most about kJoinBucketHost host
// records on average (join_part_bucket_bits), so that a bucket's ids fit two
// LDS tables; kJoinPartWG workgroups take the partition passes.  Its stage 0
// (launch_join_part, in `part` of join_part_bytes(...) bytes; scan_tmp for
// max(n kernel records, 2^bb * kJoinPartWG)) replaces the hash join's; a table
// that fills up flags ATREX_ERRBIT_SPILL, and the host then runs the hash
// join's stage 0 instead.  Stage 1 is the same.
constexpr uint32_t kJoinPartWG = 256, kJoinBucketHost = 2048, kJoinMinBucketBits = 4, kJoinMaxBucketBits = 15;
constexpr uint64_t kJoinPartMaxHost = (uint64_t)kJoinBucketHost << kJoinMaxBucketBits;
uint32_t join_part_bucket_bits(uint64_t n_host);
size_t join_part_bytes(uint64_t n_kernels, uint64_t n_host, uint32_t bb);
void launch_join_part(hipStream_t s, const JoinKernels& k, const JoinHost& h, const JoinIntervals& iv, uint32_t bb,
                      void* part, uint8_t* source, uint32_t* ref, uint32_t* flag, uint32_t* pos, void* scan_tmp,
                      unsigned long long* words, uint32_t* err);
hipError_t set_join_smem_limits();

// kernels_share.hip
hipError_t set_share_smem_limits();
// per-phase device time and counts of events without applications (global
// accumulators cleared by the caller), with the range checks
void launch_time_totals(hipStream_t s, const EventsDev& ev, uint32_t P, uint32_t nblocks, bool vec,
                        unsigned long long* T, unsigned long long* cnt, uint32_t* err);
// The target-DSL share from groups of phase 0 (outside) and 1 (inside the
// DSL); words[8]: key count, operator count, defined operators, the overall
// mean (as double bits), and its exact-sum chunks.
void launch_target_share(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t* hk, uint32_t* kidx,
                         uint32_t* ho, uint32_t* oidx, void* scan_tmp, const ShareOut& out, uint64_t kcap,
                         uint64_t ocap, double* share_all, uint32_t* op_first, unsigned long long* words);

// kernels_aggregate.hip
hipError_t set_kernel_smem_limits();
// pcount / cnt (nullable): per-block invocation counts of each (app, phase)
// and their sums (the launch with pcount set writes them; the reduce sums them).
void launch_pass_a_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                       unsigned long long* partial, unsigned long long* carry, uint32_t* pcount, uint32_t* err);
// The reduce reads the carry (extension) table and leaves it zero for the
// next pass A.
void launch_pass_a_reduce(hipStream_t s, const unsigned long long* partial, uint32_t nb, uint32_t G,
                          unsigned long long* carry, uint64_t* T, const uint32_t* c, const uint64_t* Csum,
                          uint32_t P, uint64_t* scale, void* bscale, const uint32_t* pcount, uint64_t* cnt);
void launch_pass_a_lds32(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                         uint32_t* partial, unsigned long long* ext, uint32_t* pcount, uint32_t* err);
void launch_pass_a_reduce32(hipStream_t s, const uint32_t* partial, uint32_t nb, uint32_t G,
                            unsigned long long* ext, uint64_t* T, const uint32_t* c, const uint64_t* Csum,
                            uint32_t P, uint64_t* scale, void* bscale, const uint32_t* pcount, uint64_t* cnt);
// hj (nullable): the hot scatter's partition histogram taken inside the
// range-split pass A (workgroup w < hj->nwg counts range w's cold keys); the
// launch then needs pass_a_hist_bytes(*hj) more LDS per workgroup.
void launch_pass_a_range(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t GR, uint32_t R,
                         uint32_t slices, uint32_t* partial, unsigned long long* ext, uint32_t* pcount,
                         const HistJob* hj, uint32_t* err);
size_t pass_a_hist_bytes(const HistJob& hj);
void launch_pass_a_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, uint32_t nblocks,
                          unsigned long long* T, unsigned long long* cnt, uint32_t* err);
void launch_unpack_scale(hipStream_t s, const uint64_t* sw, uint64_t G, uint64_t* mant, int32_t* rho);
// incremental refresh: T += T_run, cnt += n_run over G (app, phase) pairs,
// unless err has the range bit; and a plain device copy
void launch_fold_totals(hipStream_t s, uint64_t* T, uint64_t* cnt, const uint64_t* T_run, const uint64_t* n_run,
                        uint64_t G, const uint32_t* err);
void launch_copy_u64(hipStream_t s, uint64_t* dst, const uint64_t* src, uint64_t n);
// scale words (general form) and the 16-byte pass-B entries
void launch_scale(hipStream_t s, const uint64_t* T, const uint32_t* c, const uint64_t* Csum, uint32_t A,
                  uint32_t P, uint64_t* scale, void* bscale);
void launch_pass_b_global(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                          const GroupTables& gt, bool raw, uint32_t nblocks, uint32_t* err);
// LDS hash engine
uint32_t pass_b_lds_slots(uint32_t P, bool raw, size_t lds_bytes);
size_t pass_b_lds_smem(uint32_t P, bool raw, uint32_t S);
uint32_t spill_cap(uint64_t n, uint32_t nwg);
uint32_t owner_cap(uint32_t S);
void launch_pass_b_lds(hipStream_t s, const EventsDev& ev, uint32_t A, uint32_t P, const uint64_t* scale,
                       const void* bscale, bool raw, uint32_t S, uint32_t nblocks, const OwnerRegions& orr, uint32_t* spill_key,
                       uint64_t* spill_val, uint64_t* spill_raw, uint32_t* spill_count, uint32_t scap,
                       const Rows& rows, const uint32_t* seed, uint32_t* err);
// A tag table image of S slots holding the hottest keys of a sample of NS <=
// 2^18 events (tab_cap >= 2 NS, a power of two; list/idx and list2/idx2 hold
// tab_cap entries); *covered = sampled events of the placed keys.
void launch_seed(hipStream_t s, const uint32_t* key, uint64_t n, uint32_t NS, uint64_t* tab, uint32_t tab_cap,
                 uint32_t* cnt, uint64_t* list, uint32_t* idx, uint64_t* list2, uint32_t* idx2, void* sort_tmp,
                 uint32_t S, uint32_t* seed, unsigned long long* covered);
// Another image, of S slots, from the sorted list launch_seed left in `list`:
// window 2 places keys as the LDS engine looks them up (home bucket or the
// next), window 1 in their own bucket only (the hot scatter's lookup).
void launch_seed_image(hipStream_t s, const uint64_t* list, uint32_t tab_cap, uint32_t S, uint32_t window,
                       uint32_t* seed, unsigned long long* covered);
void launch_compact_rows(hipStream_t s, const GroupTables& gt, uint32_t P, const Rows& rows, uint32_t* err);

// kernels_rows.hip
hipError_t set_rows_smem_limits();
uint32_t lds_table_slots(uint32_t P, bool raw, size_t lds_bytes);
size_t lds_table_bytes(uint32_t P, bool raw, uint32_t S);
// owner merge into sorted per-owner lists (+ the spill records when few), then
// the global order of the lists' rows by ranking; rows the lists cannot take
// go to the row list and leave the ranking undone (done = 0)
uint32_t owner_list_slots(uint32_t P, bool raw);
constexpr uint32_t kRankMax = 16384;  // rows the one-launch ranking handles
void launch_owner_finish(hipStream_t s, const OwnerRegions& orr, uint32_t nwg, uint32_t P, bool raw, uint32_t So,
                         const SpillIn& sp, const OwnerLists& ol, const Rows& rows, uint32_t* err);
void launch_rank_groups(hipStream_t s, const OwnerLists& ol, uint32_t P, const SpillIn& sp, const Rows& rows,
                        const uint32_t* err, const SortedGroups& out, uint64_t* S_out, unsigned long long* G_out,
                        uint32_t* done);
void launch_lists_to_rows(hipStream_t s, const OwnerLists& ol, const Rows& rows, uint32_t* err);
constexpr uint32_t kMaxPartWG = 1024;  // partition workgroups over the events
uint32_t part_scatter_wgs(uint32_t cus);
void launch_part_hist(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t BB, uint32_t* H);
// the histogram of the events whose key is not in the seeded image (S slots)
void launch_part_hist_cold(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t BB, uint32_t* H,
                           const uint32_t* seed, uint32_t S);
// Slots of k_part_scatter_hot's table at P phases and 2^BB buckets (0: none fit).
uint32_t hot_scatter_slots(uint32_t P, uint32_t BB);
// Pass B with a seeded LDS table for the image's keys and the partition
// scatter for the other events (positions O from launch_part_hist_cold); the
// table goes to the owner regions [nwg][ATREX_OWNERS].
void launch_hot_scatter(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t A, uint32_t P,
                        const uint64_t* scale, const uint64_t* bscale, uint32_t BB, const uint32_t* O, uint64_t* rec,
                        const uint32_t* seed, uint32_t S, const OwnerRegions& orr, const Rows& rows, uint32_t* err);
void launch_part_scatter(hipStream_t s, const PartSource& src, uint32_t nwg, uint32_t A, uint32_t P,
                         const uint64_t* scale, const uint64_t* bscale, uint32_t BB, const uint32_t* O, uint64_t* rec,
                         uint64_t* rraw, uint32_t* err);
void launch_part_items(hipStream_t s, const uint32_t* O, const uint32_t* H, uint32_t nw, uint32_t BB, uint32_t CH,
                       uint32_t* bstart, uint32_t* item_start);
void launch_part_aggregate(hipStream_t s, const uint64_t* rec, const uint64_t* rraw, uint32_t BB, uint32_t CH,
                           const uint32_t* bstart, const uint32_t* item_start, uint32_t P, uint32_t S,
                           uint32_t nblocks, const Rows& rows, uint32_t* err);
void launch_iota_rows(hipStream_t s, const Rows& rows, uint64_t R, uint64_t* k, uint32_t* v);
void launch_rows_reduce(hipStream_t s, const Rows& rows, const uint64_t* rk_sorted, const uint32_t* idx,
                        const uint32_t* starts, uint64_t G, const SortedGroups& out);

// kernels_util.hip
void launch_fill_u64(hipStream_t s, uint64_t* p, uint64_t n, uint64_t v);
void launch_fill_u32(hipStream_t s, uint32_t* p, uint64_t n, uint32_t v);
void launch_copy_u32(hipStream_t s, uint32_t* dst, const uint32_t* src, uint64_t n);
// Up to kPublishMax device word ranges copied to a host-mapped buffer (32-bit words).
constexpr uint32_t kPublishMax = 16;
struct PublishList {
  const uint32_t* src[kPublishMax];
  uint32_t off32[kPublishMax], n32[kPublishMax];
  uint32_t count;
};
// After the copies, `done` (host-mapped) receives `seq` with a system-scope
// release, so a host that reads `seq` there (acquire) sees the copied words.
void launch_publish(hipStream_t s, const PublishList& pl, uint32_t* dst, uint32_t* done, uint32_t seq);
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
// caller-side group output arrays of phase_normalize
struct GroupsOut {
  uint32_t* key;
  uint8_t* phase;
  uint64_t* count;
  uint64_t* wsum;         // [G][2]
  uint64_t* raw;          // [G][2] or null
  double* weight;
  uint64_t* phase_total;  // [P][2]
};
// scratch of the three unit launches (see kernels_units.hip)
struct UnitScratch {
  uint64_t* keyU;      // [G][2], at each key's first group
  uint32_t* tileKeys;  // [tiles]
  uint64_t* tileKeyU;  // [tiles][2]
  uint32_t* tileRuns;  // [tiles]
  uint32_t* tileCont;  // [tiles]
  uint32_t* runOp;     // [tiles * 1024]
  uint64_t* runW;      // [tiles * 1024][2]
  uint32_t* runMask;   // [tiles * 1024]
  uint32_t* keyOff;    // [tiles]
  uint32_t* opBase;    // [tiles]
  uint32_t* runOff;    // [tiles]
  uint32_t* opMask;    // [max ops]
  uint64_t* totals;    // [2][2]: sum U over operators, over keys
};
uint64_t units_tiles(uint64_t G);
constexpr uint64_t kUnitsSmallMax = 8192;  // groups the one-workgroup unit kernel handles
// The score ranking's inputs and outputs (n <= kScoreRankMax units).
struct ScoreRankArgs {
  const uint32_t* score_key;
  const double* S;
  uint32_t n;
  uint32_t* sorted_op;
  double* sorted_S;
  uint32_t* err;
};
// Device-side group count for launch_units_rank: G (null: the host's G), the
// ordering's done flag, the group-by's error word, and the largest count
// taken (at most kUnitsSmallMax).
struct UnitsGuard {
  const unsigned long long* G;
  const uint32_t* done;
  const uint32_t* err;
  uint32_t gmax;
};
// G <= kUnitsSmallMax: the one-workgroup unit kernel, the score ranking and the
// group weights in one launch (they are independent).
void launch_units_rank(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t L, const uint64_t* S,
                       const GroupsOut& out, const UnitTable& ops, uint64_t maxOps, const UnitTable& keys,
                       unsigned long long* counts, uint32_t* err, const ScoreRankArgs& sr, const UnitsGuard& guard);
void launch_units(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t L, const uint64_t* S,
                  const GroupsOut& out, const UnitScratch& us, const UnitTable& ops, uint64_t maxOps,
                  const UnitTable& keys, unsigned long long* counts, uint32_t* err);
void launch_phase_totals(hipStream_t s, const SortedGroups& g, uint64_t G, uint32_t P, uint64_t* partials,
                         uint32_t nb, uint64_t* S);
// Segments of equal unit (key >> shift) in sorted groups: flags + scan -> starts.
void launch_unit_starts(hipStream_t s, const uint32_t* flags, const uint32_t* scan, uint64_t G, uint32_t* starts);
void launch_sum_u128(hipStream_t s, const uint64_t* x, uint64_t n, uint64_t* partials, uint32_t nb, uint64_t* out);
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
// Large-n score by operator segments: operator keys + identity order, the
// longest segment, and one workgroup per segment (segments <= kScoreSegMax).
constexpr uint32_t kScoreSegMax = 8192;
void launch_score_opiota(hipStream_t s, const uint32_t* score_key, uint64_t n, uint64_t* k_op, uint32_t* idx);
void launch_seg_maxlen(hipStream_t s, const uint32_t* flags, const uint32_t* scan, uint64_t n, const uint32_t* starts,
                       uint32_t* out);
void launch_score_seg(hipStream_t s, const uint32_t* score_key, const double* S, const uint32_t* order,
                      const uint32_t* starts, uint64_t nseg, uint32_t maxlen, const UnitTable& opt, uint64_t nops_trace,
                      uint32_t* r_op, uint64_t* r_U, double* r_S, uint32_t* err);
hipError_t set_normalize_smem_limits();
hipError_t set_units_smem_limits();
void launch_score_final(hipStream_t s, const uint32_t* r_op, const uint64_t* r_U, const double* r_S,
                        uint64_t nops, const uint64_t* totalU, uint32_t* op, double* op_weight, double* op_score,
                        double* s_agg, uint32_t* err);

// kernels_small.hip (one workgroup, up to small_rows_n() rows; *done = 0 when more)
uint32_t small_rows_n();
void launch_small_rows(hipStream_t s, const Rows& rows, const SortedGroups& out, unsigned long long* G_out,
                       uint32_t* done);
// score of at most kScoreRankMax units: ranking + one-workgroup finish
constexpr uint32_t kScoreRankMax = 8192;
// The operator table holds min(*nops_trace, maxOps) rows (the count the
// normalisation wrote on the device).
void launch_score_small(hipStream_t s, const uint32_t* score_key, const double* S, uint64_t n, uint32_t* sorted_op,
                        double* sorted_S, const UnitTable& opt, const unsigned long long* nops_trace, uint64_t maxOps,
                        uint32_t* op_out, double* w_out, double* s_out, double* s_agg, uint64_t* totU,
                        unsigned long long* nret, uint32_t* err);
// The second step of the above alone (after the ranking ran elsewhere).
void launch_score_final(hipStream_t s, uint64_t n, const uint32_t* sorted_op, const double* sorted_S,
                        const UnitTable& opt, const unsigned long long* nops_trace, uint64_t maxOps, uint32_t* op_out,
                        double* w_out, double* s_out, double* s_agg, uint64_t* totU, unsigned long long* nret);
hipError_t set_score_smem_limits();
