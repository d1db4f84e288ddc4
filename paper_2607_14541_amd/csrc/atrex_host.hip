// atrex_host.hip -- host side of the C ABI declared in include/atrex.h:
// parameter checks, workspace layout, kernel sequencing on the caller's
// stream, device error word readback, optional per-kernel hipEvent timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/atrex.h"
#include "atrex_kernels.h"

#define ATREX_ERRBIT_RANGE 1u
#define ATREX_ERRBIT_CAPACITY 2u
#define ATREX_ERRBIT_DUP 4u
#define ATREX_ERRBIT_SPILL 8u

namespace {

constexpr size_t kAlign = 256;
constexpr size_t kLdsBytes = 160 * 1024;
constexpr uint32_t kPassAThreads = 1024;  // one workgroup per CU (16 waves), two groups of loads in flight per lane
constexpr uint64_t kPartialRowsMax = 1024;  // pass-A workgroups with private partial rows
constexpr uint64_t kMaxWG = 256;            // persistent workgroups of the LDS engines
constexpr uint32_t kMaxBucketBits = 12;     // radix-partition buckets: at most 4096
constexpr uint32_t kChunk = 1u << 20;       // records per bucket chunk of the partition engine
constexpr uint32_t kMaxTimed = 64;
constexpr uint64_t kSeedMinEvents = 1ull << 22;  // events from which the LDS engine may be seeded
constexpr uint32_t kSeedSamples = 1u << 18;      // sampled events (the sample table has twice the slots)
constexpr uint64_t kStatsBatch = 8192;   // large units per radix-select batch
constexpr uint32_t kStatsTargets = 10;   // up to 8 quantiles, the minimum and the maximum
constexpr uint32_t kSpillInline = 16384;    // spill records the owner merge takes in

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
uint64_t next_pow2(uint64_t x) {
  uint64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Byte offsets of every workspace region (all 256-byte aligned).
struct Layout {
  size_t ctrl, T, carryA, partA, partC, nA, scale, bscale, dict, acc, raw;
  size_t T_run, n_run;  // incremental refresh: totals of the events folded so far
  size_t seed;          // tag table image of the LDS engine seeded with the hottest keys
  // observed runtime per unit (device-time contexts): unit counts and
  // segment starts, write cursors, lookup table, size-class lists, radix
  // select state of one batch of large units
  size_t st_cnt, st_start, st_cur, st_hkey, st_hval, st_tiny, st_small, st_large, st_cstart, st_prefix, st_want,
      st_hist, st_mat;
  uint64_t st_cap;  // lookup-table capacity (a power of two)
  size_t okey, oacc, oraw, ocount, skey, sval, sraw, scount;  // LDS engine outputs
  size_t ol_rk, ol_key, ol_lo, ol_hi, ol_rlo, ol_rhi, ol_count, ol_part;  // per-owner sorted lists
  size_t H, O, rec, rraw, bstart, istart;                     // partition engine
  size_t rk, rlo_acc, rhi_acc, rlo_raw, rhi_raw;              // rows
  size_t sk[3], sv[3], rs_tmp, scan_tmp;
  size_t g_key, g_ph, g_cnt, g_w, g_raw, S;
  size_t flags, scan, starts;
  size_t op_id, op_U, op_w, key_id, key_U, key_w;
  size_t r_op, r_U, r_S, partials, total;
  size_t u_keyU, u_tileKeys, u_tileKeyU, u_tileRuns, u_tileCont, u_runOp, u_runW, u_runMask, u_keyOff, u_opBase,
      u_runOff, u_opMask, u_totals;  // unit launches
  size_t bytes;
  uint64_t capD, maxG, maxK, maxS, maxSort, maxOps, partA_rows, maxRows;
  int passA;         // 0: 64-bit LDS table, 1: 32-bit LDS table, 2: global atomics
  uint32_t ldsSlots; // LDS hash engine slots
  uint32_t tabSlots; // owner-merge / bucket-aggregate LDS table slots
  uint32_t capo, scap;
  uint32_t oSlots;   // owner-list LDS table slots
};

struct Params {
  uint32_t P, A;
  uint64_t max_events, max_groups, max_keys, max_score;
  bool raw;
  bool count;    // invocation counts per (app, phase) in pass A
  bool compact;  // global-hash engine only: no per-event scratch, rows sized to the groups
  bool time;     // plain device-time group-by: no applications, identity scale (counts always on)
  bool incr;     // incremental refresh of an append-only log (counts always on)
};

constexpr uint32_t kPassARangesMax = 16;
constexpr uint32_t kPassASlices = 32;

// 32-bit LDS counters per range of the range-split pass A (a u32 count beside
// each with counting on); 64 per-lane spare counters follow the range
uint32_t pass_a_range_bins(bool count) { return (uint32_t)((kLdsBytes - 512) / (count ? 8 : 4)); }

// The pass-A variant for G_A = A * P (app, phase) pairs: the LDS entry grows
// by a 32-bit count with counting on.
int pass_a_mode(uint64_t G_A, bool count) {
  const uint64_t cb = count ? 4 : 0;
  if (G_A * (8 + cb) <= kLdsBytes - 1024) return 0;  // 64-bit LDS table
  if (G_A * (4 + cb) <= kLdsBytes - 512) return 1;   // 32-bit LDS table
  const uint64_t bins = pass_a_range_bins(count);
  if ((G_A + bins - 1) / bins <= kPassARangesMax) return 3;  // ranges of the table
  return 2;                                                  // global atomics
}

Layout make_layout(const Params& p) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes ? bytes : 1);
    return at;
  };
  const uint64_t GA = (uint64_t)p.A * p.P;
  L.maxG = p.max_groups;
  L.maxK = p.max_keys;
  L.maxS = p.max_score;
  L.maxSort = std::max<uint64_t>(std::max<uint64_t>(L.maxG, L.maxS), 1);
  L.capD = next_pow2(std::max<uint64_t>(1024, 2 * L.maxK));
  L.maxOps = std::min<uint64_t>(L.maxG, 65536);
  L.passA = pass_a_mode(GA, p.count);
  L.partA_rows = L.passA == 0 ? (p.compact ? kMaxWG : kPartialRowsMax)
                 : L.passA == 1 ? kMaxWG : L.passA == 3 ? kPassASlices : 0;
  L.ldsSlots = pass_b_lds_slots(p.P, p.raw, kLdsBytes);
  L.tabSlots = lds_table_slots(p.P, p.raw, kLdsBytes);
  L.capo = owner_cap(L.ldsSlots);
  L.scap = spill_cap(p.max_events, kMaxWG);
  // the global-hash engine emits one row per group; the others may emit a
  // group's rows from several workgroups or bucket chunks
  L.maxRows = p.compact ? L.maxG : 2 * L.maxG + (1 << 21);
  // regions of the LDS and partition engines (none in the compact layout)
  const uint64_t lds_eng = p.compact ? 0 : 1, part_eng = p.compact ? 0 : 1;
  L.maxSort = std::max<uint64_t>(L.maxSort, L.maxRows);
  const uint64_t accw = (p.raw ? 2 : 1);
  L.ctrl = take(4096);
  L.T = take(GA * 16);
  L.carryA = take(GA * 8);
  L.partA = take(L.partA_rows * GA * (L.passA == 0 ? 8 : 4));
  L.partC = take(p.count ? L.partA_rows * GA * 4 : 0);
  L.nA = take(p.count || p.time ? GA * 8 : 0);
  L.scale = take(GA * 8);
  L.bscale = take(GA * 8);
  L.seed = take(lds_eng * (size_t)L.ldsSlots * 4);
  L.T_run = take(p.incr ? GA * 16 : 0);
  L.n_run = take(p.incr ? GA * 8 : 0);
  {
    const uint64_t U = p.time ? L.maxG : 0, B = p.time ? kStatsBatch : 0;
    L.st_cap = next_pow2(std::max<uint64_t>(1024, 2 * U));
    L.st_cnt = take((U + 1) * 4);
    L.st_start = take((U + 1) * 4);
    L.st_cur = take(U * 4);
    L.st_hkey = take(p.time ? L.st_cap * 8 : 0);
    L.st_hval = take(p.time ? L.st_cap * 4 : 0);
    L.st_tiny = take(U * 4);
    L.st_small = take(U * 4);
    L.st_large = take(U * 4);
    L.st_cstart = take((B + 1) * 4);
    L.st_prefix = take(B * kStatsTargets * 8);
    L.st_want = take(B * kStatsTargets * 4);
    L.st_hist = take(B * kStatsTargets * 256 * 4);
    L.st_mat = take(std::min<uint64_t>(U, stats_dense_units()) * kMaxWG * 4);
  }
  L.dict = take(L.capD * 8);
  L.acc = take(L.capD * p.P * 16);
  L.raw = take(p.raw ? L.capD * p.P * 16 : 0);
  const uint64_t oslots = lds_eng * kMaxWG * ATREX_OWNERS * (uint64_t)L.capo;
  L.okey = take(oslots * 4);
  L.oacc = take(oslots * p.P * 16);
  L.oraw = take(p.raw ? oslots * p.P * 16 : 0);
  L.ocount = take(lds_eng * kMaxWG * ATREX_OWNERS * 4);
  const uint64_t sslots = lds_eng * kMaxWG * (uint64_t)L.scap;
  L.skey = take(sslots * 4);
  L.sval = take(sslots * 16);
  L.sraw = take(p.raw ? sslots * 8 : 0);
  L.scount = take(lds_eng * kMaxWG * 4);
  L.oSlots = owner_list_slots(p.P, p.raw);
  const uint64_t olrows = lds_eng * ATREX_OWNERS * L.oSlots * p.P;
  L.ol_rk = take(olrows * 8);
  L.ol_key = take(olrows * 4);
  L.ol_lo = take(olrows * 8);
  L.ol_hi = take(olrows * 8);
  L.ol_rlo = take(p.raw ? olrows * 8 : 0);
  L.ol_rhi = take(p.raw ? olrows * 8 : 0);
  L.ol_count = take(lds_eng * ATREX_OWNERS * 4);
  L.ol_part = take(lds_eng * ATREX_OWNERS * p.P * 16);
  const uint64_t hsz = part_eng * ((uint64_t)1 << kMaxBucketBits) * std::max<uint64_t>(kMaxWG, kMaxPartWG);
  L.H = take(hsz * 4);
  L.O = take(hsz * 4);
  L.rec = take(part_eng * p.max_events * 16);
  L.rraw = take(p.raw ? part_eng * p.max_events * 8 : 0);
  L.bstart = take(part_eng * (((uint64_t)1 << kMaxBucketBits) + 1) * 4);
  L.istart = take(part_eng * (((uint64_t)1 << kMaxBucketBits) + 1) * 4);
  L.rk = take(L.maxRows * 8);
  L.rlo_acc = take(L.maxRows * 8);
  L.rhi_acc = take(L.maxRows * 8);
  L.rlo_raw = take(p.raw ? L.maxRows * 8 : 0);
  L.rhi_raw = take(p.raw ? L.maxRows * 8 : 0);
  (void)accw;
  for (int i = 0; i < 3; ++i) {
    L.sk[i] = take(L.maxSort * 8);
    L.sv[i] = take(L.maxSort * 4);
  }
  L.rs_tmp = take(radix_sort_tmp_bytes(L.maxSort));
  L.scan_tmp = take(std::max(std::max(scan_tmp_bytes(L.maxSort + 1), scan_tmp_bytes(hsz)),
                             p.time ? scan_tmp_bytes(std::min<uint64_t>(L.maxG, stats_dense_units()) * kMaxWG) : 0));
  L.g_key = take(L.maxG * 4);
  L.g_ph = take(L.maxG);
  L.g_cnt = take(L.maxG * 8);
  L.g_w = take(L.maxG * 16);
  L.g_raw = take(p.raw ? L.maxG * 16 : 0);
  L.S = take(8 * 16);
  L.flags = take((L.maxSort + 1) * 4);
  L.scan = take((L.maxSort + 1) * 4);
  L.starts = take((L.maxSort + 2) * 4);
  L.op_id = take(L.maxOps * 4);
  L.op_U = take(L.maxOps * 16);
  L.op_w = take(L.maxOps * 8);
  L.key_id = take(L.maxG * 4);
  L.key_U = take(L.maxG * 16);
  L.key_w = take(L.maxG * 8);
  L.r_op = take(L.maxS * 4);
  L.r_U = take(L.maxS * 16);
  L.r_S = take(L.maxS * 8);
  L.partials = take(1024 * 8 * 16);
  const uint64_t ut = std::max<uint64_t>(1, units_tiles(L.maxG));
  L.u_keyU = take(L.maxG * 16);
  L.u_tileKeys = take(ut * 4);
  L.u_tileKeyU = take(ut * 16);
  L.u_tileRuns = take(ut * 4);
  L.u_tileCont = take(ut * 4);
  L.u_runOp = take(ut * 1024 * 4);
  L.u_runW = take(ut * 1024 * 16);
  L.u_runMask = take(ut * 1024 * 4);
  L.u_keyOff = take(ut * 4);
  L.u_opBase = take(ut * 4);
  L.u_runOff = take(ut * 4);
  L.u_opMask = take(L.maxOps * 4);
  L.u_totals = take(64);
  L.total = take(64);
  L.bytes = off;
  return L;
}

atrex_status check_params(const atrex_init_params* ip, Params* out) {
  if (!ip) return ATREX_E_INVALID_ARG;
  if (ip->num_phases < 1 || ip->num_phases > 8 || ip->num_apps < 1) return ATREX_E_INVALID_ARG;
  if (ip->max_events >= (1ull << 31)) return ATREX_E_INVALID_ARG;
  if ((uint64_t)ip->num_apps * ip->num_phases >= (1ull << 32)) return ATREX_E_INVALID_ARG;
  if ((unsigned)ip->path > (unsigned)ATREX_PATH_RADIX_SORT) return ATREX_E_INVALID_ARG;
  Params p;
  p.P = ip->num_phases;
  p.A = ip->num_apps;
  p.max_events = ip->max_events;
  p.max_groups = ip->max_groups ? ip->max_groups : std::max<uint64_t>(ip->max_events, 1);
  p.max_keys = ip->max_keys ? ip->max_keys : p.max_groups;
  p.max_score = ip->max_score ? ip->max_score : p.max_groups;
  if (p.max_groups >= (1ull << 32) || p.max_score >= (1ull << 31) || p.max_keys >= (1ull << 31))
    return ATREX_E_INVALID_ARG;
  p.raw = (ip->flags & ATREX_FLAG_RAW) != 0;
  p.count = (ip->flags & ATREX_FLAG_APP_COUNT) != 0;
  p.compact = false;
  p.time = (ip->flags & ATREX_FLAG_DEVICE_TIME) != 0;
  if (p.time && (p.A != 1 || p.raw)) return ATREX_E_INVALID_ARG;
  p.incr = (ip->flags & ATREX_FLAG_INCREMENTAL) != 0;
  if (p.incr && p.time) return ATREX_E_INVALID_ARG;
  if (p.incr) p.count = true;  // the counts of the whole log are kept too
  *out = p;
  return ATREX_OK;
}

struct Timed {
  const char* name;
  uint64_t items;
  hipEvent_t a, b;
};

uint64_t lcm_1_to(uint32_t P) {
  uint64_t l = 1;
  for (uint64_t k = 2; k <= P; ++k) {
    uint64_t a = l, b = k;
    while (b) {
      const uint64_t t = a % b;
      a = b;
      b = t;
    }
    l = l / a * k;
  }
  return l;
}

}  // namespace

struct atrex_ctx {
  Params p;
  Layout L;
  char* ws;
  hipStream_t s;
  atrex_path path;
  uint32_t flags;
  const uint32_t* app_weight;
  int state;  // 0 initialised, 1 aggregated, 2 normalised
  bool S_ready;  // the per-phase totals S were written by the ordering step
  uint64_t G, nops, nkeys;
  uint64_t n_folded;  // incremental refresh: events whose totals are in T_run / n_run
  uint64_t n_agg;     // events of the last successful group-by
  int cus;
  const char* path_used;
  std::vector<Timed> timed;
  size_t ntimed;
  // pinned, device-mapped host staging for device -> host readbacks of
  // status words: written by one k_publish launch per synchronisation
  char* pinned = nullptr;
  uint32_t* pinned_dev = nullptr;  // the same buffer as the device sees it
  size_t pinned_used = 0;
  uint32_t publish_seq = 0;  // last value k_publish wrote to the completion word
  bool plain_copies = false;  // a readback went through hipMemcpyAsync instead
  struct Pending {
    void* dst;
    const void* src;
    size_t off, bytes;
  };
  std::vector<Pending> pending;
  std::vector<float> last_ms;
  std::vector<const char*> last_names;
  std::vector<uint64_t> last_items;

  template <class T>
  T* at(size_t off) const {
    return reinterpret_cast<T*>(ws + off);
  }
  uint32_t* err() const { return at<uint32_t>(L.ctrl); }
  unsigned long long* counter() const { return at<unsigned long long>(L.ctrl + 64); }
  unsigned long long* row_count() const { return at<unsigned long long>(L.ctrl + 128); }
  Rows rows() const {
    Rows r;
    r.rk = at<uint64_t>(L.rk);
    r.lo = at<uint64_t>(L.rlo_acc);
    r.hi = at<uint64_t>(L.rhi_acc);
    r.rlo = p.raw ? at<uint64_t>(L.rlo_raw) : nullptr;
    r.rhi = p.raw ? at<uint64_t>(L.rhi_raw) : nullptr;
    r.count = row_count();
    r.cap = L.maxRows;
    return r;
  }
  OwnerRegions owners() const {
    OwnerRegions o;
    o.key = at<uint32_t>(L.okey);
    o.acc = at<uint64_t>(L.oacc);
    o.raw = p.raw ? at<uint64_t>(L.oraw) : nullptr;
    o.count = at<uint32_t>(L.ocount);
    o.capo = L.capo;
    return o;
  }
  uint64_t* Csum() const { return at<uint64_t>(L.ctrl + 1024); }
  double* sagg() const { return at<double>(L.ctrl + 1088); }
  unsigned long long* unit_counts() const { return at<unsigned long long>(L.ctrl + 256); }  // operators, keys
  GroupTables tables() const {
    GroupTables gt;
    gt.dict = at<unsigned long long>(L.dict);
    gt.dict_mask = (uint32_t)(L.capD - 1);
    gt.acc = at<unsigned long long>(L.acc);
    gt.raw = p.raw ? at<unsigned long long>(L.raw) : nullptr;
    return gt;
  }
  OwnerLists lists() const {
    OwnerLists l;
    l.rk = at<uint64_t>(L.ol_rk);
    l.dkey = at<uint32_t>(L.ol_key);
    l.dcount = at<unsigned long long>(L.ctrl + 224);
    l.lo = at<uint64_t>(L.ol_lo);
    l.hi = at<uint64_t>(L.ol_hi);
    l.rlo = p.raw ? at<uint64_t>(L.ol_rlo) : nullptr;
    l.rhi = p.raw ? at<uint64_t>(L.ol_rhi) : nullptr;
    l.count = at<uint32_t>(L.ol_count);
    l.part = at<uint64_t>(L.ol_part);
    l.cap = L.oSlots * p.P;
    return l;
  }
  SpillIn spills(uint32_t nwg) const {
    SpillIn sp;
    sp.key = at<uint32_t>(L.skey);
    sp.val = at<uint64_t>(L.sval);
    sp.raw = p.raw ? at<uint64_t>(L.sraw) : nullptr;
    sp.count = at<uint32_t>(L.scount);
    sp.cap = L.scap;
    sp.nwg = nwg;
    sp.inline_max = kSpillInline;
    return sp;
  }
  UnitScratch unit_scratch() const {
    UnitScratch u;
    u.keyU = at<uint64_t>(L.u_keyU);
    u.tileKeys = at<uint32_t>(L.u_tileKeys);
    u.tileKeyU = at<uint64_t>(L.u_tileKeyU);
    u.tileRuns = at<uint32_t>(L.u_tileRuns);
    u.tileCont = at<uint32_t>(L.u_tileCont);
    u.runOp = at<uint32_t>(L.u_runOp);
    u.runW = at<uint64_t>(L.u_runW);
    u.runMask = at<uint32_t>(L.u_runMask);
    u.keyOff = at<uint32_t>(L.u_keyOff);
    u.opBase = at<uint32_t>(L.u_opBase);
    u.runOff = at<uint32_t>(L.u_runOff);
    u.opMask = at<uint32_t>(L.u_opMask);
    u.totals = at<uint64_t>(L.u_totals);
    return u;
  }
  SortedGroups groups() const {
    SortedGroups g;
    g.key = at<uint32_t>(L.g_key);
    g.phase = at<uint8_t>(L.g_ph);
    g.count = at<uint64_t>(L.g_cnt);
    g.wsum = at<uint64_t>(L.g_w);
    g.raw = p.raw ? at<uint64_t>(L.g_raw) : nullptr;
    return g;
  }
  // timing helpers
  void begin_call() { ntimed = 0; }
  int tstart(const char* name, uint64_t items) {
    if (!(flags & ATREX_FLAG_TIMING) || ntimed >= timed.size()) return -1;
    Timed& t = timed[ntimed];
    t.name = name;
    t.items = items;
    (void)hipEventRecord(t.a, s);
    return (int)ntimed++;
  }
  void tstop(int i) {
    if (i >= 0) (void)hipEventRecord(timed[i].b, s);
  }
  void end_call() {
    if (!(flags & ATREX_FLAG_TIMING)) return;
    last_ms.clear();
    last_names.clear();
    last_items.clear();
    for (size_t i = 0; i < ntimed; ++i) {
      float ms = 0.f;
      (void)hipEventElapsedTime(&ms, timed[i].a, timed[i].b);
      last_ms.push_back(ms);
      last_names.push_back(timed[i].name);
      last_items.push_back(timed[i].items);
    }
  }
};

namespace {

// The kernels' dynamic LDS limits, set once per process.
hipError_t ensure_smem_limits() {
  static std::mutex mu;
  static bool done = false;
  std::lock_guard<std::mutex> lk(mu);
  if (done) return hipSuccess;
  const hipError_t e = set_kernel_smem_limits();
  if (e == hipSuccess) done = true;
  return e;
}

// ATREX_E_DEVICE, with the HIP error and where it was met on stderr (device
// errors are rare and otherwise carry no detail through the status code).
atrex_status device_error(hipError_t e, const char* where) {
  fprintf(stderr, "atrex: HIP error %d (%s) at %s\n", (int)e, hipGetErrorString(e), where);
  return ATREX_E_DEVICE;
}

atrex_status sync_status(atrex_ctx* c) {
  const hipError_t e1 = hipGetLastError();
  const hipError_t e2 = hipStreamSynchronize(c->s);
  if (e1 != hipSuccess) return device_error(e1, "a launch or call before the synchronisation");
  if (e2 != hipSuccess) return device_error(e2, "stream synchronisation");
  return ATREX_OK;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

constexpr size_t kPinnedBytes = 4096;
constexpr size_t kDoneOff = kPinnedBytes - 64;  // completion word, on a line of its own

// Device -> host readback of a few status words (a multiple of 4 bytes)
// through the context's mapped pinned buffer; sync_read() launches the copy
// and fills in the host values once it has completed.
void d2h(atrex_ctx* c, void* dst, const void* src, size_t bytes) {
  size_t off = (c->pinned_used + 7) / 8 * 8;
  if (!c->pinned_dev || off + bytes > kDoneOff || bytes % 4 != 0 || c->pending.size() >= kPublishMax) {
    (void)hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, c->s);  // plain (pageable) copy
    c->plain_copies = true;
    return;
  }
  c->pending.push_back({dst, src, off, bytes});
  c->pinned_used = off + bytes;
}

// Wait for k_publish's completion word to read `seq`: the stream's work up to
// and including the copies is then done (a stream runs its launches in order).
// The stream is queried every few hundred polls, so a device error or a
// publish that never wrote ends the wait with ATREX_E_DEVICE.
atrex_status wait_published(atrex_ctx* c, uint32_t seq) {
  const uint32_t* done = (const uint32_t*)(c->pinned + kDoneOff);
  for (uint32_t spin = 1;; ++spin) {
    if (__atomic_load_n(done, __ATOMIC_ACQUIRE) == seq) return ATREX_OK;
    if (spin % 256 == 0) {
      const hipError_t q = hipStreamQuery(c->s);
      if (q == hipSuccess) {
        // the stream has finished: the completion word is written; read it
        // again after a synchronisation before calling its absence an error
        const hipError_t e = hipStreamSynchronize(c->s);
        if (e == hipSuccess && __atomic_load_n(done, __ATOMIC_ACQUIRE) == seq) return ATREX_OK;
        return device_error(e != hipSuccess ? e : hipErrorUnknown, "completion word of the status readback");
      }
      if (q != hipErrorNotReady) return device_error(q, "stream query while waiting for the status readback");
    }
    __builtin_ia32_pause();
  }
}

// Ends a call's device work: copies the pending readbacks through one
// k_publish launch and waits for it by polling its completion word (a stream
// synchronisation wakes the host later); with timing on, or after a plain
// copy, by a stream synchronisation.
atrex_status sync_read(atrex_ctx* c) {
  atrex_status st = ATREX_OK;
  if (c->pinned_dev) {
    PublishList pl{};
    for (const auto& p : c->pending) {
      pl.src[pl.count] = (const uint32_t*)p.src;
      pl.off32[pl.count] = (uint32_t)(p.off / 4);
      pl.n32[pl.count] = (uint32_t)(p.bytes / 4);
      ++pl.count;
    }
    if (++c->publish_seq == 0) c->publish_seq = 1;  // 0 is the buffer's initial value
    launch_publish(c->s, pl, c->pinned_dev, c->pinned_dev + kDoneOff / 4, c->publish_seq);
    const bool poll = !c->plain_copies && !(c->flags & ATREX_FLAG_TIMING);
    const hipError_t le = hipGetLastError();
    if (le != hipSuccess) {
      (void)hipStreamSynchronize(c->s);
      st = device_error(le, "a launch or call before the status readback");
    } else {
      st = poll ? wait_published(c, c->publish_seq) : sync_status(c);
    }
  } else {
    st = sync_status(c);
  }
  for (const auto& p : c->pending) memcpy(p.dst, c->pinned + p.off, p.bytes);
  c->pending.clear();
  c->pinned_used = 0;
  c->plain_copies = false;
  return st;
}

#define TIMED(ctx, name, items, stmt) \
  do {                                \
    const int t_ = (ctx)->tstart(name, items); \
    stmt;                             \
    (ctx)->tstop(t_);                 \
  } while (0)

}  // namespace

namespace {

// The radix-partition engine over all events (spill = false) or over the LDS
// engine's spill regions: bucket histograms, scan, scatter of 16-byte records,
// work items, per-bucket-chunk LDS group-by -> rows.
// Radix-partition buckets: at least 256 (work for every CU even with one
// chunk per bucket; few buckets keep the scatter's runs long) and about half
// an LDS table of keys per bucket (with raw time the scatter's LDS tile
// leaves room for 2^11 buckets).
uint32_t bucket_bits(const atrex_ctx* c, uint64_t keys_est) {
  const uint32_t maxBB = c->p.raw ? kMaxBucketBits - 1 : kMaxBucketBits;
  uint32_t BB = 8;
  while (BB < maxBB && ((keys_est + (1ull << BB) - 1) >> BB) > c->L.tabSlots / 2) ++BB;
  return BB;
}

atrex_status run_partition(atrex_ctx* c, const EventsDev& d, const uint64_t* scale, bool spill, uint32_t nwg,
                           uint64_t nrec, uint64_t keys_est) {
  if (!spill) nwg = part_scatter_wgs((uint32_t)c->cus);  // event ranges: several workgroups per CU
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const uint32_t P = c->p.P;
  const uint32_t BB = bucket_bits(c, keys_est);
  PartSource src;
  src.ev = d;
  src.per = ((d.n + nwg - 1) / nwg + 3) / 4 * 4;
  src.skey = c->at<uint32_t>(L.skey);
  src.sval = c->at<uint64_t>(L.sval);
  src.sraw = c->p.raw ? c->at<uint64_t>(L.sraw) : nullptr;
  src.scount = c->at<uint32_t>(L.scount);
  src.scap = spill_cap(d.n, nwg);
  src.spill = spill;
  uint32_t* H = c->at<uint32_t>(L.H);
  uint32_t* O = c->at<uint32_t>(L.O);
  const uint64_t hn = ((uint64_t)1 << BB) * nwg;
  TIMED(c, spill ? "part_hist_spill" : "part_hist", nrec, launch_part_hist(s, src, nwg, BB, H));
  exclusive_scan_u32(s, H, O, hn, c->at<void>(L.scan_tmp));
  TIMED(c, spill ? "part_scatter_spill" : "part_scatter", nrec,
        launch_part_scatter(s, src, nwg, c->p.A, P, scale, c->at<uint64_t>(L.bscale), BB, O, c->at<uint64_t>(L.rec),
                            c->p.raw ? c->at<uint64_t>(L.rraw) : nullptr, c->err()));
  launch_part_items(s, O, H, nwg, BB, kChunk, c->at<uint32_t>(L.bstart), c->at<uint32_t>(L.istart));
  TIMED(c, spill ? "part_aggregate_spill" : "part_aggregate", nrec,
        launch_part_aggregate(s, c->at<uint64_t>(L.rec), c->p.raw ? c->at<uint64_t>(L.rraw) : nullptr, BB, kChunk,
                              c->at<uint32_t>(L.bstart), c->at<uint32_t>(L.istart), P, L.tabSlots,
                              (uint32_t)c->cus, c->rows(), c->err()));
  return ATREX_OK;
}

}  // namespace

extern "C" {

const char* atrex_status_str(atrex_status s) {
  switch (s) {
    case ATREX_OK: return "ok";
    case ATREX_E_INVALID_ARG: return "invalid argument";
    case ATREX_E_OUT_OF_RANGE: return "value out of range";
    case ATREX_E_STATE: return "call out of order";
    case ATREX_E_CAPACITY: return "capacity exceeded";
    case ATREX_E_DEVICE: return "HIP device error";
  }
  return "unknown status";
}

atrex_status atrex_workspace_bytes(const atrex_init_params* ip, size_t* bytes) {
  if (!bytes) return ATREX_E_INVALID_ARG;
  Params p;
  const atrex_status st = check_params(ip, &p);
  if (st != ATREX_OK) return st;
  *bytes = make_layout(p).bytes;
  return ATREX_OK;
}

atrex_status atrex_aggregate_init(const atrex_init_params* ip, atrex_ctx** out) {
  if (!out) return ATREX_E_INVALID_ARG;
  *out = nullptr;
  Params p;
  atrex_status st = check_params(ip, &p);
  if (st != ATREX_OK) return st;
  if ((!ip->app_weight_q16 && !p.time) || !ip->workspace || !aligned(ip->workspace, kAlign))
    return ATREX_E_INVALID_ARG;
  const Layout L = make_layout(p);
  if (ip->workspace_bytes < L.bytes) return ATREX_E_CAPACITY;
  if (ensure_smem_limits() != hipSuccess) return ATREX_E_DEVICE;
  atrex_ctx* c = new (std::nothrow) atrex_ctx();
  if (!c) return ATREX_E_INVALID_ARG;
  c->p = p;
  c->L = L;
  c->ws = (char*)ip->workspace;
  c->s = (hipStream_t)ip->stream;
  c->path = ip->path;
  c->flags = ip->flags;
  c->app_weight = p.time ? nullptr : ip->app_weight_q16;
  c->state = 0;
  c->S_ready = false;
  c->G = c->nops = c->nkeys = 0;
  c->n_folded = 0;
  c->path_used = "none";
  c->ntimed = 0;
  if (hipHostMalloc((void**)&c->pinned, kPinnedBytes, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) {
    c->pinned = nullptr;
  } else {
    memset(c->pinned, 0, kPinnedBytes);  // the completion word starts at 0
    if (hipHostGetDevicePointer((void**)&c->pinned_dev, c->pinned, 0) != hipSuccess)
      c->pinned_dev = nullptr;  // readbacks fall back to plain copies
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&c->cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    if (c->pinned) (void)hipHostFree(c->pinned);
    delete c;
    return ATREX_E_DEVICE;
  }
  if (c->flags & ATREX_FLAG_TIMING) {
    c->timed.resize(kMaxTimed);
    for (auto& t : c->timed) {
      if (hipEventCreate(&t.a) != hipSuccess || hipEventCreate(&t.b) != hipSuccess) {
        if (c->pinned) (void)hipHostFree(c->pinned);
        delete c;
        return ATREX_E_DEVICE;
      }
    }
  }
  // the pass-A carry table starts clear (each pass-A reduce clears it again)
  launch_fill_u64(c->s, c->at<uint64_t>(c->L.carryA), (uint64_t)p.A * p.P, 0);
  if (p.incr) {  // nothing folded yet
    launch_fill_u64(c->s, c->at<uint64_t>(c->L.T_run), 2 * (uint64_t)p.A * p.P, 0);
    launch_fill_u64(c->s, c->at<uint64_t>(c->L.n_run), (uint64_t)p.A * p.P, 0);
  }
  if (p.time) {  // no applications, no card-hour weights
    st = sync_status(c);
    if (st != ATREX_OK) {
      atrex_aggregate_destroy(c);
      return st;
    }
    *out = c;
    return ATREX_OK;
  }
  // C = sum_a c_a, checked > 0 (p_a = c_a / C must exist)
  launch_sum_u32(c->s, c->app_weight, p.A, c->Csum());
  uint64_t C = 0;
  d2h(c, &C, c->Csum(), 8);
  st = sync_read(c);
  if (st == ATREX_OK && C == 0) st = ATREX_E_INVALID_ARG;
  if (st != ATREX_OK) {
    atrex_aggregate_destroy(c);
    return st;
  }
  *out = c;
  return ATREX_OK;
}

namespace {

// State of one group-by between its enqueue and its completion.
struct AggRun {
  EventsDev d;
  atrex_path path;
  uint32_t nwg;
  const uint64_t* scale;
  uint64_t hdr[32];  // control words: error at byte 0, row counter at byte 128
};

// The group-by up to the ordering of the groups, enqueued; the control words
// are queued for readback into a->hdr (the caller synchronises, then calls
// aggregate_complete).
atrex_status aggregate_enqueue(atrex_ctx* c, const atrex_events* ev, AggRun* a) {
  if (!c || !ev) return ATREX_E_INVALID_ARG;
  if (c->state != 0) return ATREX_E_STATE;
  const uint64_t n = ev->n;
  if (n > c->p.max_events) return ATREX_E_CAPACITY;
  if (c->p.time ? ev->app != nullptr : (n > 0 && !ev->app)) return ATREX_E_INVALID_ARG;
  if (c->p.incr && n < c->n_folded) return ATREX_E_INVALID_ARG;  // the log only grows
  if (n > 0 && (!ev->key || !ev->phase || !ev->dur_ns)) return ATREX_E_INVALID_ARG;
  const uint32_t P = c->p.P, A = c->p.A;
  const uint64_t GA = (uint64_t)A * P;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  c->begin_call();
  EventsDev d;
  d.key = ev->key;
  d.app = ev->app;
  d.phase = ev->phase;
  d.dur = ev->dur_ns;
  d.n = n;
  const bool vec_ok = aligned(ev->key, 16) && aligned(ev->app, 16) && aligned(ev->phase, 4) &&
                      aligned(ev->dur_ns, 16);
  // pass A reads the events it folds: all of them, or with an incremental
  // context the ones past those folded before
  const uint64_t from = c->p.incr ? c->n_folded : 0;
  EventsDev dA = d;
  if (from) {
    dA.key = ev->key + from;
    dA.app = ev->app + from;
    dA.phase = ev->phase + from;
    dA.dur = ev->dur_ns + from;
    dA.n = n - from;
  }
  const uint64_t na = dA.n;
  const bool vecA = aligned(dA.key, 16) && aligned(dA.app, 16) && aligned(dA.phase, 4) && aligned(dA.dur, 16);
  GroupTables gt = c->tables();
  // clear the control words (the pass-A carry table is clear: init clears
  // it and every pass-A reduce leaves it so)
  launch_fill_u64(s, c->at<uint64_t>(L.ctrl), 64, 0);
  // The engine of pass B, chosen before pass A: the seed step below only
  // reads keys, and the hot scatter's histogram can then ride in pass A.
  atrex_path path = c->path;
  if (path == ATREX_PATH_AUTO) path = (c->p.max_keys <= L.ldsSlots) ? ATREX_PATH_LDS_HASH : ATREX_PATH_RADIX_SORT;
  if (c->p.compact) path = ATREX_PATH_GLOBAL_HASH;  // the only engine the compact layout holds
  // the LDS engine indexes its scale words with 24-bit multiplies
  if (path == ATREX_PATH_LDS_HASH && (uint64_t)A * P >= (1u << 24)) path = ATREX_PATH_RADIX_SORT;
  if (!vec_ok && path != ATREX_PATH_GLOBAL_HASH) path = ATREX_PATH_GLOBAL_HASH;
  const uint32_t nwg = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)c->cus, kMaxWG));
  atrex_status st = ATREX_OK;
  // More keys than one LDS table holds: when the hottest keys that fit the
  // table cover at least half of a sample of the events, the LDS engine
  // starts from those keys and spills the rest (the partition engine then
  // sees only the spilled events); otherwise the partition engine takes all.
  // (Events without applications take the partition engine as before.)
  // When the image leaves more than 1/16 of the sample to spill (and without
  // raw time), a smaller table beside the partition engine's tile takes the
  // hottest keys instead and the other events are partitioned in the same
  // pass (k_part_scatter_hot): no spill records are written and read again.
  const uint32_t* seed = nullptr;
  bool hot = false;
  uint32_t hotS = 0, hotBB = 0;
  if (c->path == ATREX_PATH_AUTO && path == ATREX_PATH_RADIX_SORT && !c->p.compact && vec_ok && ev->app &&
      n >= kSeedMinEvents &&
      (uint64_t)A * P < (1u << 24)) {
    unsigned long long* covered = c->at<unsigned long long>(L.ctrl + 3072);
    TIMED(c, "seed", kSeedSamples,
          launch_seed(s, ev->key, n, kSeedSamples, c->at<uint64_t>(L.rk), 2 * kSeedSamples,
                      c->at<uint32_t>(L.rlo_acc), c->at<uint64_t>(L.sk[0]), c->at<uint32_t>(L.sv[0]),
                      c->at<uint64_t>(L.sk[1]), c->at<uint32_t>(L.sv[1]), c->at<void>(L.rs_tmp), L.ldsSlots,
                      c->at<uint32_t>(L.seed), covered));
    uint64_t cov = 0;
    d2h(c, &cov, covered, 8);
    st = sync_read(c);
    if (st != ATREX_OK) return st;
    if (2 * cov >= kSeedSamples) {
      path = ATREX_PATH_LDS_HASH;
      seed = c->at<uint32_t>(L.seed);
      if (!c->p.raw && 16 * cov < 15 * (uint64_t)kSeedSamples) {
        hotBB = bucket_bits(c, c->p.max_keys);
        hotS = std::min(hot_scatter_slots(P, hotBB), L.ldsSlots);
        if (hotS) {
          TIMED(c, "seed_image", hotS,
                launch_seed_image(s, c->at<uint64_t>(L.sk[0]), 2 * kSeedSamples, hotS, 1, c->at<uint32_t>(L.seed),
                                  covered));
          hot = true;
        }
      }
    }
  }
  // the hot scatter's partition: ranges of the whole event array (pass A may
  // see only the new events of a log), counted inside the range-split pass A
  // when that is pass A's engine
  HistJob hj{};
  bool hist_in_a = false;
  if (hot) {
    hj.key = d.key;
    hj.n = n;
    hj.per = ((n + nwg - 1) / nwg + 3) / 4 * 4;
    hj.nwg = nwg;
    hj.BB = hotBB;
    hj.S = hotS;
    hj.seed = seed;
    hj.H = c->at<uint32_t>(L.H);
    hist_in_a = !c->p.time && L.passA == 3 && vecA;
  }
  // pass A, Eq. (2), and the Eq. (3) scale words of every (app, phase)
  uint64_t* T = c->at<uint64_t>(L.T);
  uint64_t* scale = c->at<uint64_t>(L.scale);
  // invocation counts per (app, phase): per-block partials, then their sums
  uint32_t* pcount = c->p.count ? c->at<uint32_t>(L.partC) : nullptr;
  uint64_t* nA = c->p.count || c->p.time ? c->at<uint64_t>(L.nA) : nullptr;
  if (c->p.time) {
    // no applications: per-phase device time and counts with the range
    // checks, and the identity scale (m = 2^55, rho = 0: each share is the
    // duration itself) in both word forms
    launch_fill_u64(s, T, 2 * (uint64_t)P, 0);
    launch_fill_u64(s, nA, P, 0);
    TIMED(c, "time_totals", na,
          launch_time_totals(s, dA, P, (uint32_t)c->cus, vecA, (unsigned long long*)T, (unsigned long long*)nA,
                             c->err()));
    launch_fill_u64(s, scale, P, (uint64_t)64 << 56);
    launch_fill_u64(s, c->at<uint64_t>(L.bscale), P, ((uint64_t)63 << 56) | ((uint64_t)1 << 55));
  } else if (L.passA == 0 && vecA) {
    // one workgroup per CU (two groups of loads in flight per lane): two per
    // CU ran as one after the other (the SIMDs favour the older one) and
    // doubled the partial rows for the reduce
    uint64_t nb = std::min<uint64_t>((uint64_t)c->cus, L.partA_rows);
    nb = std::max<uint64_t>(1, std::min<uint64_t>(nb, (na / 4 + kPassAThreads - 1) / kPassAThreads));
    TIMED(c, "pass_a", na,
          launch_pass_a_lds(s, dA, A, P, (uint32_t)nb, c->at<unsigned long long>(L.partA),
                            c->at<unsigned long long>(L.carryA), pcount, c->err()));
    TIMED(c, "pass_a_reduce", GA,
          launch_pass_a_reduce(s, c->at<unsigned long long>(L.partA), (uint32_t)nb, (uint32_t)GA,
                               c->at<unsigned long long>(L.carryA), T, c->app_weight, c->Csum(), P, scale,
                               c->at<void>(L.bscale), pcount, nA));
  } else if (L.passA == 3 && vecA) {
    // with the histogram inside, its counters and image take LDS from the bins
    const uint32_t hist_bins =
        hist_in_a ? (uint32_t)((pass_a_hist_bytes(hj) + 16 + (c->p.count ? 7 : 3)) / (c->p.count ? 8 : 4)) : 0;
    const uint32_t bins = pass_a_range_bins(c->p.count) - hist_bins;
    const uint32_t R = (uint32_t)((GA + bins - 1) / bins);
    const uint32_t GR = (uint32_t)((GA + R - 1) / R);
    TIMED(c, "pass_a_range", na,
          launch_pass_a_range(s, dA, A, P, GR, R, kPassASlices, c->at<uint32_t>(L.partA),
                              c->at<unsigned long long>(L.carryA), pcount, hist_in_a ? &hj : nullptr, c->err()));
    TIMED(c, "pass_a_reduce", GA,
          launch_pass_a_reduce32(s, c->at<uint32_t>(L.partA), kPassASlices, (uint32_t)GA,
                                 c->at<unsigned long long>(L.carryA), T, c->app_weight, c->Csum(), P, scale,
                                 c->at<void>(L.bscale), pcount, nA));
  } else if (L.passA == 1 && vecA) {
    const uint64_t nb = std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)c->cus, kMaxWG));
    TIMED(c, "pass_a", na,
          launch_pass_a_lds32(s, dA, A, P, (uint32_t)nb, c->at<uint32_t>(L.partA), c->at<unsigned long long>(L.carryA),
                              pcount, c->err()));
    TIMED(c, "pass_a_reduce", GA,
          launch_pass_a_reduce32(s, c->at<uint32_t>(L.partA), (uint32_t)nb, (uint32_t)GA,
                                 c->at<unsigned long long>(L.carryA), T, c->app_weight, c->Csum(), P, scale,
                                 c->at<void>(L.bscale), pcount, nA));
  } else {
    launch_fill_u64(s, T, GA * 2, 0);
    if (nA) launch_fill_u64(s, nA, GA, 0);
    TIMED(c, "pass_a_global", na,
          launch_pass_a_global(s, dA, A, P, (uint32_t)std::max<uint64_t>(1, (uint64_t)c->cus * 8), (unsigned long long*)T,
                               (unsigned long long*)nA, c->err()));
    // scale, Eq. (3) (the column-sum kernels of the other modes compute it with T)
    TIMED(c, "scale", GA, launch_scale(s, T, c->app_weight, c->Csum(), A, P, scale, c->at<void>(L.bscale)));
  }
  if (c->p.incr) {
    // the totals of the whole log: those folded before plus the new events'
    // (skipped on the device after a range error), and the scale from them
    launch_fold_totals(s, T, nA, c->at<uint64_t>(L.T_run), c->at<uint64_t>(L.n_run), GA, c->err());
    TIMED(c, "scale", GA, launch_scale(s, T, c->app_weight, c->Csum(), A, P, scale, c->at<void>(L.bscale)));
  }
  // pass B, Eq. (2)-(3): every engine emits rows (key << 3 | phase, Q96 sum)
  const Rows rows = c->rows();
  if (hot) {
    c->path_used = "hot_scatter";
    PartSource src{};
    src.ev = d;
    src.per = hj.per;
    src.spill = false;
    uint32_t* H = c->at<uint32_t>(L.H);
    uint32_t* O = c->at<uint32_t>(L.O);
    if (!hist_in_a) TIMED(c, "part_hist_cold", n, launch_part_hist_cold(s, src, nwg, hotBB, H, seed, hotS));
    exclusive_scan_u32(s, H, O, ((uint64_t)1 << hotBB) * nwg, c->at<void>(L.scan_tmp));
    TIMED(c, "hot_scatter", n,
          launch_hot_scatter(s, src, nwg, A, P, scale, c->at<uint64_t>(L.bscale), hotBB, O, c->at<uint64_t>(L.rec),
                             seed, hotS, c->owners(), rows, c->err()));
    launch_fill_u32(s, c->at<uint32_t>(L.scount), nwg, 0);  // the owner merge finds no spill records
    TIMED(c, "owner_finish", (uint64_t)nwg * ATREX_OWNERS,
          launch_owner_finish(s, c->owners(), nwg, P, false, L.oSlots, c->spills(nwg), c->lists(), rows, c->err()));
    launch_lists_to_rows(s, c->lists(), rows, c->err());
    launch_part_items(s, O, H, nwg, hotBB, kChunk, c->at<uint32_t>(L.bstart), c->at<uint32_t>(L.istart));
    TIMED(c, "part_aggregate_cold", n,
          launch_part_aggregate(s, c->at<uint64_t>(L.rec), nullptr, hotBB, kChunk, c->at<uint32_t>(L.bstart),
                                c->at<uint32_t>(L.istart), P, L.tabSlots, (uint32_t)c->cus, rows, c->err()));
    path = ATREX_PATH_RADIX_SORT;  // rows from here on as from the partition engine
  } else if (path == ATREX_PATH_LDS_HASH) {
    c->path_used = seed ? "lds_hash_seeded" : "lds_hash";
    const uint32_t scap = spill_cap(n, nwg);
    TIMED(c, "pass_b_lds", n,
          launch_pass_b_lds(s, d, A, P, scale, c->at<void>(L.bscale), c->p.raw, L.ldsSlots, nwg, c->owners(), c->at<uint32_t>(L.skey),
                            c->at<uint64_t>(L.sval), c->p.raw ? c->at<uint64_t>(L.sraw) : nullptr,
                            c->at<uint32_t>(L.scount), scap, rows, seed, c->err()));
    TIMED(c, "owner_finish", (uint64_t)nwg * ATREX_OWNERS,
          launch_owner_finish(s, c->owners(), nwg, P, c->p.raw, L.oSlots, c->spills(nwg), c->lists(), rows,
                              c->err()));
  } else if (path == ATREX_PATH_RADIX_SORT) {
    c->path_used = "radix_sort";
    st = run_partition(c, d, scale, false, nwg, n, c->p.max_keys);
    if (st != ATREX_OK) return st;
  } else {
    c->path_used = "global_hash";
    launch_fill_u64(s, c->at<uint64_t>(L.dict), L.capD, 0);
    launch_fill_u64(s, c->at<uint64_t>(L.acc), L.capD * P * 2, 0);
    if (c->p.raw) launch_fill_u64(s, c->at<uint64_t>(L.raw), L.capD * P * 2, 0);
    TIMED(c, "pass_b_global", n,
          launch_pass_b_global(s, d, A, P, scale, gt, c->p.raw, (uint32_t)c->cus * 8, c->err()));
    TIMED(c, "compact_rows", L.capD * P, launch_compact_rows(s, gt, P, rows, c->err()));
  }
  // rows -> groups ordered by (key, phase): the owner lists ranked in one
  // launch (LDS engine), or one workgroup when the rows are few
  unsigned long long* smallG = c->at<unsigned long long>(L.ctrl + 192);
  uint32_t* smallDone = c->at<uint32_t>(L.ctrl + 200);
  if (path == ATREX_PATH_LDS_HASH)
    TIMED(c, "rank_groups", 0,
          launch_rank_groups(s, c->lists(), P, c->spills(nwg), rows, c->err(), c->groups(), c->at<uint64_t>(L.S),
                             smallG, smallDone));
  else
    TIMED(c, "small_rows", 0, launch_small_rows(s, rows, c->groups(), smallG, smallDone));
  a->d = d;
  a->path = path;
  a->nwg = nwg;
  a->scale = scale;
  d2h(c, a->hdr, c->at<uint64_t>(L.ctrl), sizeof(a->hdr));
  return ATREX_OK;
}

// The rest of the group-by once a->hdr has been read back: the fallbacks the
// control words ask for (each with its own waits) and the group count.
// *fast: the ordering finished in one launch and nothing more was enqueued.
atrex_status aggregate_complete(atrex_ctx* c, AggRun* a, uint64_t* num_groups, bool* fast) {
  *fast = false;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const Rows rows = c->rows();
  const atrex_path path = a->path;
  const EventsDev& d = a->d;
  const uint64_t n = d.n;
  const uint32_t nwg = a->nwg;
  const uint64_t* scale = a->scale;
  uint64_t* hdr = a->hdr;
  unsigned long long* smallG = c->at<unsigned long long>(L.ctrl + 192);
  uint32_t* smallDone = c->at<uint32_t>(L.ctrl + 200);
  atrex_status st = ATREX_OK;
  if ((uint32_t)hdr[0] & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  // the ranking also wrote S[ph]
  bool ranked = path == ATREX_PATH_LDS_HASH && !((uint32_t)hdr[0] & ATREX_ERRBIT_SPILL) && (uint32_t)hdr[25];
  if (path == ATREX_PATH_LDS_HASH && !((uint32_t)hdr[0] & ATREX_ERRBIT_SPILL) && !(uint32_t)hdr[25]) {
    // not ranked in one launch: the lists (and the spill records when too many
    // for the owner merge) become rows for the general ordering
    launch_lists_to_rows(s, c->lists(), rows, c->err());
    if (hdr[26] > kSpillInline) {
      st = run_partition(c, d, scale, true, nwg, 0, c->p.max_keys);
      if (st != ATREX_OK) return st;
    }
    TIMED(c, "small_rows", 0, launch_small_rows(s, rows, c->groups(), smallG, smallDone));
    d2h(c, hdr, c->at<uint64_t>(L.ctrl), sizeof(a->hdr));
    st = sync_read(c);
    if (st != ATREX_OK) return st;
  }
  if (path == ATREX_PATH_LDS_HASH && ((uint32_t)hdr[0] & ATREX_ERRBIT_SPILL)) {
    // a spill region overflowed: partition every event instead
    launch_fill_u64(s, c->at<uint64_t>(L.ctrl), 64, 0);
    c->path_used = "lds_hash+radix_all";
    st = run_partition(c, d, scale, false, nwg, n, c->p.max_keys);
    if (st != ATREX_OK) return st;
    TIMED(c, "small_rows", 0, launch_small_rows(s, rows, c->groups(), smallG, smallDone));
    d2h(c, hdr, c->at<uint64_t>(L.ctrl), sizeof(a->hdr));
    st = sync_read(c);
    if (st != ATREX_OK) return st;
    if ((uint32_t)hdr[0] & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  }
  if ((uint32_t)hdr[0] & ATREX_ERRBIT_CAPACITY) return ATREX_E_CAPACITY;
  const uint64_t R = hdr[16];  // row counter at byte 128
  if (R > L.maxRows) return ATREX_E_CAPACITY;
  uint64_t G = 0;
  if ((uint32_t)hdr[25]) {  // done by the one-workgroup kernel (flag at byte 200)
    G = hdr[24];
    *fast = ranked;  // ranked in one launch, nothing enqueued since
  } else if (R) {
    uint64_t* K0 = c->at<uint64_t>(L.sk[0]);
    uint32_t* V0 = c->at<uint32_t>(L.sv[0]);
    launch_iota_rows(s, rows, R, K0, V0);
    TIMED(c, "sort_rows", R,
          radix_sort_pairs(s, K0, V0, c->at<uint64_t>(L.sk[1]), c->at<uint32_t>(L.sv[1]), R, 35,
                           c->at<void>(L.rs_tmp)));
    uint32_t* flags = c->at<uint32_t>(L.flags);
    uint32_t* scan = c->at<uint32_t>(L.scan);
    uint32_t* starts = c->at<uint32_t>(L.starts);
    launch_heads_u64(s, K0, R, flags);
    exclusive_scan_u32(s, flags, scan, R, c->at<void>(L.scan_tmp));
    launch_unit_starts(s, flags, scan, R, starts);
    uint32_t tail[2] = {0, 0};
    d2h(c, &tail[0], scan + (R - 1), 4);
    d2h(c, &tail[1], flags + (R - 1), 4);
    st = sync_read(c);
    if (st != ATREX_OK) return st;
    G = (uint64_t)tail[0] + tail[1];
    if (G > L.maxG) return ATREX_E_CAPACITY;
    TIMED(c, "rows_reduce", G, launch_rows_reduce(s, rows, K0, V0, starts, G, c->groups()));
    st = sync_read(c);
    if (st != ATREX_OK) return st;
  }
  if (G > L.maxG) return ATREX_E_CAPACITY;
  c->n_agg = n;
  if (c->p.incr) {  // the refresh stands: the totals of the whole log become the folded ones
    const uint64_t GA = (uint64_t)c->p.A * c->p.P;
    launch_copy_u64(s, c->at<uint64_t>(L.T_run), c->at<uint64_t>(L.T), 2 * GA);
    launch_copy_u64(s, c->at<uint64_t>(L.n_run), c->at<uint64_t>(L.nA), GA);
    c->n_folded = n;
  }
  c->end_call();
  c->G = G;
  c->S_ready = ranked;
  c->state = 1;
  *num_groups = G;
  return ATREX_OK;
}

}  // namespace

atrex_status atrex_aggregate_events(atrex_ctx* c, const atrex_events* ev, uint64_t* num_groups) {
  if (!c || !ev || !num_groups) return ATREX_E_INVALID_ARG;
  AggRun a;
  atrex_status st = aggregate_enqueue(c, ev, &a);
  if (st != ATREX_OK) return st;
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  bool fast = false;
  return aggregate_complete(c, &a, num_groups, &fast);
}

namespace {

atrex_status normalize_check(atrex_ctx* c, const atrex_groups* out) {
  if (!c || !out) return ATREX_E_INVALID_ARG;
  if (c->state < 1) return ATREX_E_STATE;
  if (!out->phase_total) return ATREX_E_INVALID_ARG;
  if (c->G > 0 && (!out->key || !out->phase || !out->count || !out->wsum || !out->weight)) return ATREX_E_INVALID_ARG;
  if (out->raw_ns && !c->p.raw) return ATREX_E_INVALID_ARG;
  return ATREX_OK;
}

// Enqueues the per-phase totals (when the ordering step did not write them),
// the group weights and Eq. (3) per operator and per key; the counts of
// operators and keys go to the control words at byte 256.
void normalize_enqueue(atrex_ctx* c, const atrex_groups* out) {
  const uint64_t G = c->G;
  const uint32_t P = c->p.P;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const SortedGroups g = c->groups();
  uint64_t* S = c->at<uint64_t>(L.S);
  if (!c->S_ready) {
    const uint32_t nb = (uint32_t)std::min<uint64_t>(1024, std::max<uint64_t>(1, (G + 255) / 256));
    TIMED(c, "phase_totals", G, launch_phase_totals(s, g, G, P, c->at<uint64_t>(L.partials), nb, S));
  }
  GroupsOut o{out->key, out->phase, out->count, (uint64_t*)out->wsum, (uint64_t*)out->raw_ns, out->weight,
              (uint64_t*)out->phase_total};
  UnitTable ot{c->at<uint32_t>(L.op_id), c->at<uint64_t>(L.op_U), c->at<double>(L.op_w)};
  UnitTable kt{c->at<uint32_t>(L.key_id), c->at<uint64_t>(L.key_U), c->at<double>(L.key_w)};
  TIMED(c, "units", G,
        launch_units(s, g, G, P, lcm_1_to(P), S, o, c->unit_scratch(), ot, L.maxOps, kt, c->unit_counts(), c->err()));
}

// After the readback of the counts (h) and the error word (e).
atrex_status normalize_finish(atrex_ctx* c, const uint64_t h[2], uint32_t e, uint64_t* num_ops, uint64_t* num_keys) {
  if (e & ATREX_ERRBIT_CAPACITY) return ATREX_E_CAPACITY;
  c->nops = h[0];
  c->nkeys = h[1];
  if (num_ops) *num_ops = c->nops;
  if (num_keys) *num_keys = c->nkeys;
  c->state = 2;
  return ATREX_OK;
}

}  // namespace

atrex_status atrex_phase_normalize(atrex_ctx* c, const atrex_groups* out, uint64_t* num_ops, uint64_t* num_keys) {
  atrex_status st = normalize_check(c, out);
  if (st != ATREX_OK) return st;
  c->begin_call();
  normalize_enqueue(c, out);
  uint64_t h[2] = {0, 0};
  uint32_t e = 0;
  d2h(c, h, c->unit_counts(), sizeof(h));
  d2h(c, &e, c->err(), sizeof(e));
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  c->end_call();
  return normalize_finish(c, h, e, num_ops, num_keys);
}

atrex_status atrex_op_weights(atrex_ctx* c, uint32_t* op, atrex_u128* U, double* w) {
  if (!c) return ATREX_E_INVALID_ARG;
  if (c->state < 2) return ATREX_E_STATE;
  if (c->nops && (!op || !U || !w)) return ATREX_E_INVALID_ARG;
  if (c->nops) {
    (void)hipMemcpyAsync(op, c->at<void>(c->L.op_id), c->nops * 4, hipMemcpyDeviceToDevice, c->s);
    (void)hipMemcpyAsync(U, c->at<void>(c->L.op_U), c->nops * 16, hipMemcpyDeviceToDevice, c->s);
    (void)hipMemcpyAsync(w, c->at<void>(c->L.op_w), c->nops * 8, hipMemcpyDeviceToDevice, c->s);
  }
  return sync_read(c);
}

atrex_status atrex_key_weights(atrex_ctx* c, uint32_t* key, atrex_u128* U, double* omega) {
  if (!c) return ATREX_E_INVALID_ARG;
  if (c->state < 2) return ATREX_E_STATE;
  if (c->nkeys && (!key || !U || !omega)) return ATREX_E_INVALID_ARG;
  if (c->nkeys) {
    (void)hipMemcpyAsync(key, c->at<void>(c->L.key_id), c->nkeys * 4, hipMemcpyDeviceToDevice, c->s);
    (void)hipMemcpyAsync(U, c->at<void>(c->L.key_U), c->nkeys * 16, hipMemcpyDeviceToDevice, c->s);
    (void)hipMemcpyAsync(omega, c->at<void>(c->L.key_w), c->nkeys * 8, hipMemcpyDeviceToDevice, c->s);
  }
  return sync_read(c);
}

namespace {

atrex_status score_check(atrex_ctx* c, const uint32_t* score_key, const double* sv, uint64_t n, const double* s_agg) {
  if (!c || !s_agg) return ATREX_E_INVALID_ARG;
  if (c->state < 2) return ATREX_E_STATE;
  if (n == 0 || !score_key || !sv) return ATREX_E_INVALID_ARG;
  if (n > c->L.maxS) return ATREX_E_CAPACITY;
  return ATREX_OK;
}

// Readback words of the ranking score path.
struct ScoreWords {
  uint64_t tot[2], nret;
  uint32_t err;
  double sagg;
};

// n <= kScoreRankMax: ranking + one workgroup (validation, duplicates,
// medians, Eq. (6)).  The operator count comes from the control words the
// normalisation wrote, so nothing waits for the host in between.
// clear_err: start from a clear error word (a call of its own); the one-call
// path keeps the normalisation's bits, which the score's checks do not read.
void score_small_enqueue(atrex_ctx* c, const uint32_t* score_key, const double* sv, uint64_t n, uint32_t* op,
                         double* op_weight, double* op_score, bool clear_err, ScoreWords* w) {
  const Layout& L = c->L;
  hipStream_t s = c->s;
  if (clear_err) launch_fill_u64(s, c->at<uint64_t>(L.ctrl), 1, 0);
  UnitTable opt{c->at<uint32_t>(L.op_id), c->at<uint64_t>(L.op_U), c->at<double>(L.op_w)};
  uint64_t* tot = c->at<uint64_t>(L.total) + 4;
  unsigned long long* nret = c->at<unsigned long long>(L.ctrl + 320);
  // outputs go straight to the caller's arrays when given, else to scratch
  uint32_t* o_op = op ? op : c->at<uint32_t>(L.r_op);
  double* o_w = op_weight ? op_weight : c->at<double>(L.sk[0]);
  double* o_s = op_score ? op_score : c->at<double>(L.sk[1]);
  TIMED(c, "score", n,
        launch_score_small(s, score_key, sv, n, c->at<uint32_t>(L.sv[2]), c->at<double>(L.sk[2]), opt,
                           c->unit_counts(), L.maxOps, o_op, o_w, o_s, c->sagg(), tot, nret, c->err()));
  d2h(c, &w->err, c->err(), 4);
  d2h(c, w->tot, tot, 16);
  d2h(c, &w->nret, nret, 8);
  d2h(c, &w->sagg, c->sagg(), 8);
}

// The one-call path with G <= kUnitsSmallMax and a ranking score: the same
// work as normalize_enqueue + score_small_enqueue (without clearing the error
// word), in three launches instead of five.
void units_score_enqueue(atrex_ctx* c, const atrex_groups* out, const uint32_t* score_key, const double* sv,
                         uint64_t n, uint32_t* op, double* op_weight, double* op_score, ScoreWords* w) {
  const uint64_t G = c->G;
  const uint32_t P = c->p.P;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const SortedGroups g = c->groups();
  uint64_t* S = c->at<uint64_t>(L.S);
  if (!c->S_ready) {
    const uint32_t nb = (uint32_t)std::min<uint64_t>(1024, std::max<uint64_t>(1, (G + 255) / 256));
    launch_phase_totals(s, g, G, P, c->at<uint64_t>(L.partials), nb, S);
  }
  GroupsOut o{out->key, out->phase, out->count, (uint64_t*)out->wsum, (uint64_t*)out->raw_ns, out->weight,
              (uint64_t*)out->phase_total};
  UnitTable ot{c->at<uint32_t>(L.op_id), c->at<uint64_t>(L.op_U), c->at<double>(L.op_w)};
  UnitTable kt{c->at<uint32_t>(L.key_id), c->at<uint64_t>(L.key_U), c->at<double>(L.key_w)};
  uint32_t* sorted_op = c->at<uint32_t>(L.sv[2]);
  double* sorted_S = c->at<double>(L.sk[2]);
  const ScoreRankArgs sr{score_key, sv, (uint32_t)n, sorted_op, sorted_S, c->err()};
  launch_units_rank(s, g, G, P, lcm_1_to(P), S, o, ot, L.maxOps, kt, c->unit_counts(), c->err(), sr,
                    UnitsGuard{nullptr, nullptr, nullptr, 0});
  uint64_t* tot = c->at<uint64_t>(L.total) + 4;
  unsigned long long* nret = c->at<unsigned long long>(L.ctrl + 320);
  uint32_t* o_op = op ? op : c->at<uint32_t>(L.r_op);
  double* o_w = op_weight ? op_weight : c->at<double>(L.sk[0]);
  double* o_s = op_score ? op_score : c->at<double>(L.sk[1]);
  launch_score_final(s, n, sorted_op, sorted_S, ot, c->unit_counts(), L.maxOps, o_op, o_w, o_s, c->sagg(), tot, nret);
  d2h(c, &w->err, c->err(), 4);
  d2h(c, w->tot, tot, 16);
  d2h(c, &w->nret, nret, 8);
  d2h(c, &w->sagg, c->sagg(), 8);
}

atrex_status score_small_finish(const ScoreWords& w, uint64_t* num_ops, double* s_agg) {
  if (w.err & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  if (w.err & ATREX_ERRBIT_DUP) return ATREX_E_INVALID_ARG;
  if (w.tot[0] == 0 && w.tot[1] == 0) return ATREX_E_INVALID_ARG;  // no retained weight
  *s_agg = w.sagg;
  if (num_ops) *num_ops = w.nret;
  return ATREX_OK;
}

}  // namespace

atrex_status atrex_weighted_score(atrex_ctx* c, const uint32_t* score_key, const double* sv, uint64_t n, uint32_t* op,
                                  double* op_weight, double* op_score, uint64_t* num_ops, double* s_agg) {
  atrex_status st = score_check(c, score_key, sv, n, s_agg);
  if (st != ATREX_OK) return st;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  c->begin_call();
  if (n <= kScoreRankMax) {
    ScoreWords w{};
    score_small_enqueue(c, score_key, sv, n, op, op_weight, op_score, true, &w);
    st = sync_read(c);
    if (st != ATREX_OK) return st;
    c->end_call();
    return score_small_finish(w, num_ops, s_agg);
  }
  uint64_t *K0 = c->at<uint64_t>(L.sk[0]), *K1 = c->at<uint64_t>(L.sk[1]), *K2 = c->at<uint64_t>(L.sk[2]);
  uint32_t *V0 = c->at<uint32_t>(L.sv[0]), *V1 = c->at<uint32_t>(L.sv[1]), *V2 = c->at<uint32_t>(L.sv[2]);
  void* rtmp = c->at<void>(L.rs_tmp);
  uint32_t* flags = c->at<uint32_t>(L.flags);
  uint32_t* scan = c->at<uint32_t>(L.scan);
  uint32_t* starts = c->at<uint32_t>(L.starts);
  uint32_t* maxlen = c->at<uint32_t>(L.ctrl + 336);
  launch_fill_u64(s, c->at<uint64_t>(L.ctrl), 1, 0);
  launch_fill_u64(s, c->at<uint64_t>(L.ctrl + 336), 1, 0);
  TIMED(c, "score_validate", n, launch_score_validate(s, sv, n, c->err()));
  // operator segments (stable sort of the units by operator)
  launch_score_opiota(s, score_key, n, K0, V0);
  TIMED(c, "score_sort_op", n, radix_sort_pairs(s, K0, V0, K1, V1, n, 16, rtmp));
  launch_heads_u64(s, K0, n, flags);
  exclusive_scan_u32(s, flags, scan, n, c->at<void>(L.scan_tmp));
  launch_unit_starts(s, flags, scan, n, starts);
  launch_seg_maxlen(s, flags, scan, n, starts, maxlen);
  uint32_t hdr[4] = {0, 0, 0, 0};
  d2h(c, &hdr[0], c->err(), 4);
  d2h(c, &hdr[1], scan + (n - 1), 4);
  d2h(c, &hdr[2], flags + (n - 1), 4);
  d2h(c, &hdr[3], maxlen, 4);
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  if (hdr[0] & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  uint64_t nr = (uint64_t)hdr[1] + hdr[2];
  UnitTable opt{c->at<uint32_t>(L.op_id), c->at<uint64_t>(L.op_U), c->at<double>(L.op_w)};
  uint32_t* r_op = c->at<uint32_t>(L.r_op);
  uint64_t* r_U = c->at<uint64_t>(L.r_U);
  double* r_S = c->at<double>(L.r_S);
  if (hdr[3] <= kScoreSegMax) {
    // per operator in LDS: duplicate check, median, U
    TIMED(c, "score_seg", nr,
          launch_score_seg(s, score_key, sv, V0, starts, nr, hdr[3], opt, c->nops, r_op, r_U, r_S, c->err()));
  } else {
    // an operator with more than kScoreSegMax units: (key) order for the
    // duplicate check, (op, S) order for the medians, by global sorts
    launch_score_keys(s, score_key, sv, n, K0, K2, V2);
    (void)hipMemcpyAsync(V0, V2, n * 4, hipMemcpyDeviceToDevice, s);
    TIMED(c, "score_sort_keys", n, radix_sort_pairs(s, K0, V0, K1, V1, n, 32, rtmp));
    launch_dup_check(s, K0, n, c->err());
    TIMED(c, "score_sort_S", n, radix_sort_pairs(s, K2, V2, K1, V1, n, 64, rtmp));
    launch_score_opkeys(s, score_key, V2, n, K0);
    TIMED(c, "score_sort_op_S", n, radix_sort_pairs(s, K0, V2, K1, V1, n, 16, rtmp));
    launch_heads_u64(s, K0, n, flags);
    exclusive_scan_u32(s, flags, scan, n, c->at<void>(L.scan_tmp));
    launch_unit_starts(s, flags, scan, n, starts);
    TIMED(c, "score_ops", nr, launch_score_ops(s, score_key, sv, V2, starts, nr, n, opt, c->nops, r_op, r_U, r_S));
  }
  uint64_t* tot = c->at<uint64_t>(L.total) + 4;
  const uint32_t nb = (uint32_t)std::min<uint64_t>(1024, std::max<uint64_t>(1, (nr + 255) / 256));
  launch_sum_u128(s, r_U, nr, c->at<uint64_t>(L.partials), nb, tot);
  uint64_t totU[2] = {0, 0};
  uint32_t e2 = 0;
  d2h(c, &e2, c->err(), 4);
  d2h(c, totU, tot, 16);
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  if (e2 & ATREX_ERRBIT_DUP) return ATREX_E_INVALID_ARG;          // a key scored twice
  if (totU[0] == 0 && totU[1] == 0) return ATREX_E_INVALID_ARG;  // no retained weight
  TIMED(c, "score_final", nr,
        launch_score_final(s, r_op, r_U, r_S, nr, tot, op, op_weight, op_score, c->sagg(), c->err()));
  double h = 0.0;
  d2h(c, &h, c->sagg(), 8);
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  c->end_call();
  *s_agg = h;
  if (num_ops) *num_ops = nr;
  return ATREX_OK;
}

namespace {

// The one-call path's speculation: with the LDS engine the groups are usually
// ordered in one launch, so the unit kernel, the group weights and the score
// are enqueued right behind the group-by, before its readback.  The unit and
// weight parts check the ordering's flags on the device (k_units_rank's
// guard); their error bits and the score's go to words of their own, so that
// the group-by's words read back unchanged.
void speculate_enqueue(atrex_ctx* c, const atrex_groups* out, uint64_t out_capacity, const uint32_t* score_key,
                       const double* sv, uint64_t n, uint32_t* op, double* op_weight, double* op_score,
                       uint64_t h[2], uint32_t* units_err_host, ScoreWords* w) {
  const uint32_t P = c->p.P;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const SortedGroups g = c->groups();
  uint64_t* S = c->at<uint64_t>(L.S);
  GroupsOut o{out->key, out->phase, out->count, (uint64_t*)out->wsum, (uint64_t*)out->raw_ns, out->weight,
              (uint64_t*)out->phase_total};
  UnitTable ot{c->at<uint32_t>(L.op_id), c->at<uint64_t>(L.op_U), c->at<double>(L.op_w)};
  UnitTable kt{c->at<uint32_t>(L.key_id), c->at<uint64_t>(L.key_U), c->at<double>(L.key_w)};
  uint32_t* units_err = c->at<uint32_t>(L.ctrl + 480);
  uint32_t* score_err = c->at<uint32_t>(L.ctrl + 484);
  uint32_t* sorted_op = c->at<uint32_t>(L.sv[2]);
  double* sorted_S = c->at<double>(L.sk[2]);
  const ScoreRankArgs sr{score_key, sv, (uint32_t)n, sorted_op, sorted_S, score_err};
  const uint32_t gmax = (uint32_t)std::min<uint64_t>(std::min<uint64_t>(kUnitsSmallMax, out_capacity), L.maxG);
  const UnitsGuard guard{c->at<unsigned long long>(L.ctrl + 192), c->at<uint32_t>(L.ctrl + 200), c->err(), gmax};
  launch_units_rank(s, g, 0, P, lcm_1_to(P), S, o, ot, L.maxOps, kt, c->unit_counts(), units_err, sr, guard);
  uint64_t* tot = c->at<uint64_t>(L.total) + 4;
  unsigned long long* nret = c->at<unsigned long long>(L.ctrl + 320);
  uint32_t* o_op = op ? op : c->at<uint32_t>(L.r_op);
  double* o_w = op_weight ? op_weight : c->at<double>(L.sk[0]);
  double* o_s = op_score ? op_score : c->at<double>(L.sk[1]);
  launch_score_final(s, n, sorted_op, sorted_S, ot, c->unit_counts(), L.maxOps, o_op, o_w, o_s, c->sagg(), tot, nret);
  d2h(c, h, c->unit_counts(), 16);
  d2h(c, units_err_host, units_err, 4);
  d2h(c, &w->err, score_err, 4);
  d2h(c, w->tot, tot, 16);
  d2h(c, &w->nret, nret, 8);
  d2h(c, &w->sagg, c->sagg(), 8);
}

}  // namespace

atrex_status atrex_run(atrex_ctx* c, const atrex_events* ev, const atrex_groups* out, uint64_t out_capacity,
                       const uint32_t* score_key, const double* sv, uint64_t n_score, uint32_t* op, double* op_weight,
                       double* op_score, atrex_run_result* r) {
  if (!c || !ev || !out || !r) return ATREX_E_INVALID_ARG;
  *r = atrex_run_result{};
  atrex_status st = atrex_aggregate_reset(c);
  if (st != ATREX_OK) return st;
  // back to back only where the score call could not fail its argument checks
  const bool fused = n_score > 0 && n_score <= kScoreRankMax && n_score <= c->L.maxS && score_key && sv &&
                     !(c->flags & ATREX_FLAG_TIMING);
  const bool out_ok = out->phase_total && out->key && out->phase && out->count && out->wsum && out->weight &&
                      (!out->raw_ns || c->p.raw);
  AggRun a;
  st = aggregate_enqueue(c, ev, &a);
  if (st != ATREX_OK) return st;
  const bool spec = fused && out_ok && out_capacity > 0 && a.path == ATREX_PATH_LDS_HASH;
  uint64_t h[2] = {0, 0};
  uint32_t units_err = 0;
  ScoreWords w{};
  if (spec) speculate_enqueue(c, out, out_capacity, score_key, sv, n_score, op, op_weight, op_score, h, &units_err, &w);
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  uint64_t G = 0;
  bool fast = false;
  st = aggregate_complete(c, &a, &G, &fast);
  if (st != ATREX_OK) return st;
  r->num_groups = G;
  if (G > out_capacity) return ATREX_E_CAPACITY;
  if (spec && fast && G <= kUnitsSmallMax) {  // the speculation stands (the device took the same decision)
    r->one_wait = 1;
    st = normalize_finish(c, h, units_err, &r->num_ops, &r->num_keys);
    if (st != ATREX_OK) return st;
    return score_small_finish(w, &r->num_scored_ops, &r->s_agg);
  }
  st = normalize_check(c, out);
  if (st != ATREX_OK) return st;
  if (!fused) {  // the calls one by one (timing on, no score, the large score path, or an argument error)
    st = atrex_phase_normalize(c, out, &r->num_ops, &r->num_keys);
    if (st != ATREX_OK || n_score == 0) return st;
    return atrex_weighted_score(c, score_key, sv, n_score, op, op_weight, op_score, &r->num_scored_ops, &r->s_agg);
  }
  // normalisation and score enqueued back to back, one readback for both
  c->begin_call();
  w = ScoreWords{};
  if (c->G <= kUnitsSmallMax) {
    // the one-workgroup unit kernel, the score ranking and the group weights
    // in one launch, then the score's one-workgroup finish
    units_score_enqueue(c, out, score_key, sv, n_score, op, op_weight, op_score, &w);
    d2h(c, h, c->unit_counts(), sizeof(h));
  } else {
    normalize_enqueue(c, out);
    d2h(c, h, c->unit_counts(), sizeof(h));
    score_small_enqueue(c, score_key, sv, n_score, op, op_weight, op_score, false, &w);
  }
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  // the normalisation's error bits are still in the word the score read back
  st = normalize_finish(c, h, w.err, &r->num_ops, &r->num_keys);
  if (st != ATREX_OK) return st;
  return score_small_finish(w, &r->num_scored_ops, &r->s_agg);
}

atrex_status atrex_get_app_totals(atrex_ctx* c, atrex_u128* T, uint64_t* n, uint64_t* mant, int32_t* rho) {
  if (!c || !T) return ATREX_E_INVALID_ARG;
  if (n && !c->p.count && !c->p.time) return ATREX_E_INVALID_ARG;
  if (c->state < 1) return ATREX_E_STATE;
  const uint64_t GA = (uint64_t)c->p.A * c->p.P;
  (void)hipMemcpyAsync(T, c->at<void>(c->L.T), GA * 16, hipMemcpyDeviceToDevice, c->s);
  if (n) (void)hipMemcpyAsync(n, c->at<void>(c->L.nA), GA * 8, hipMemcpyDeviceToDevice, c->s);
  if (mant || rho) launch_unpack_scale(c->s, c->at<uint64_t>(c->L.scale), GA, mant, rho);
  return sync_read(c);
}

atrex_status atrex_refresh(atrex_ctx* c, const atrex_events* log, uint64_t n_new, uint64_t* num_groups) {
  if (!c || !log || !num_groups) return ATREX_E_INVALID_ARG;
  if (!c->p.incr || log->n < n_new || log->n - n_new != c->n_folded) return ATREX_E_INVALID_ARG;
  return atrex_aggregate_events(c, log, num_groups);
}

atrex_status atrex_refresh_state(atrex_ctx* c, atrex_u128* T, uint64_t* n, uint64_t* n_folded) {
  if (!c || !T || !n || !n_folded || !c->p.incr) return ATREX_E_INVALID_ARG;
  const uint64_t GA = (uint64_t)c->p.A * c->p.P;
  launch_copy_u64(c->s, (uint64_t*)T, c->at<uint64_t>(c->L.T_run), 2 * GA);
  launch_copy_u64(c->s, n, c->at<uint64_t>(c->L.n_run), GA);
  const atrex_status st = sync_read(c);
  if (st == ATREX_OK) *n_folded = c->n_folded;
  return st;
}

atrex_status atrex_refresh_restore(atrex_ctx* c, const atrex_u128* T, const uint64_t* n, uint64_t n_folded) {
  if (!c || !T || !n || !c->p.incr || n_folded > c->p.max_events) return ATREX_E_INVALID_ARG;
  if (c->state != 0) return ATREX_E_STATE;
  const uint64_t GA = (uint64_t)c->p.A * c->p.P;
  launch_copy_u64(c->s, c->at<uint64_t>(c->L.T_run), (const uint64_t*)T, 2 * GA);
  launch_copy_u64(c->s, c->at<uint64_t>(c->L.n_run), n, GA);
  const atrex_status st = sync_read(c);
  if (st == ATREX_OK) c->n_folded = n_folded;
  return st;
}

atrex_status atrex_unit_stats(atrex_ctx* c, const atrex_events* ev, int by_phase, const uint32_t* q_1e5, uint32_t nq,
                              const atrex_stats_out* out, uint64_t capacity, uint64_t* num_units) {
  if (!c || !ev || !out || !num_units || nq > 8 || (nq && !q_1e5)) return ATREX_E_INVALID_ARG;
  if (!c->p.time) return ATREX_E_INVALID_ARG;
  if (c->state < 1) return ATREX_E_STATE;
  if (ev->app || ev->n != c->n_agg || (ev->n && (!ev->key || !ev->phase || !ev->dur_ns))) return ATREX_E_INVALID_ARG;
  if (capacity && (!out->key || !out->phase || !out->count || !out->total_ns || !out->mean_ns || !out->min_ns ||
                   !out->max_ns || (nq && !out->quantile_ns)))
    return ATREX_E_INVALID_ARG;
  StatsQ q{};
  for (uint32_t j = 0; j < nq; ++j) {
    if (q_1e5[j] < 1 || q_1e5[j] > 100000) return ATREX_E_INVALID_ARG;
    q.q[j] = q_1e5[j];
  }
  q.n = nq;
  const Layout& L = c->L;
  hipStream_t s = c->s;
  const uint64_t G = c->G, n = ev->n;
  StatsOut so;
  so.key = out->key;
  so.phase = out->phase;
  so.count = out->count;
  so.total = (uint64_t*)out->total_ns;
  so.mean = out->mean_ns;
  so.min = out->min_ns;
  so.max = out->max_ns;
  so.quant = out->quantile_ns;
  StatsTable t;
  t.key = c->at<uint64_t>(L.st_hkey);
  t.val = c->at<uint32_t>(L.st_hval);
  t.mask = (uint32_t)(L.st_cap - 1);
  unsigned long long* words = c->at<unsigned long long>(L.ctrl + 2048);
  uint32_t* ucount = c->at<uint32_t>(L.st_cnt);
  uint32_t* seg = c->at<uint32_t>(L.st_start);
  int64_t* vals = c->at<int64_t>(L.rec);
  c->begin_call();
  launch_fill_u64(s, (uint64_t*)words, 8, 0);
  launch_fill_u32(s, c->err(), 1, 0);
  launch_fill_u64(s, t.key, L.st_cap, 0);
  launch_fill_u32(s, ucount, G + 1, 0);  // G + 1 counts (the scan's last entry is the total)
  // units, their counts and totals, the lookup table; segment starts
  TIMED(c, "stats_units", G,
        launch_stats_units(s, c->groups(), G, by_phase != 0, c->at<uint32_t>(L.flags), c->at<uint32_t>(L.scan),
                           c->at<void>(L.scan_tmp), so, capacity, ucount, t, words));
  exclusive_scan_u32(s, ucount, seg, G + 1, c->at<void>(L.scan_tmp));
  uint64_t w0 = 0;
  d2h(c, &w0, words, 8);
  atrex_status st = sync_read(c);
  if (st != ATREX_OK) return st;
  const uint64_t U = w0;
  EventsDev d;
  d.key = ev->key;
  d.app = nullptr;
  d.phase = ev->phase;
  d.dur = ev->dur_ns;
  d.n = n;
  const bool vec = aligned(ev->key, 16) && aligned(ev->phase, 4) && aligned(ev->dur_ns, 16);
  const uint32_t nwg = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>((uint64_t)c->cus, kMaxWG));
  if (U <= stats_dense_units()) {  // per-workgroup LDS counters: two passes, no global atomics
    TIMED(c, "stats_scatter", n,
          launch_stats_dense(s, d, c->p.P, by_phase != 0, vec, nwg, t, (uint32_t)U, c->at<uint32_t>(L.st_mat),
                             c->at<void>(L.scan_tmp), seg, vals, words, c->err()));
  } else {
    launch_copy_u32(s, c->at<uint32_t>(L.st_cur), seg, U);
    TIMED(c, "stats_scatter", n,
          launch_stats_scatter(s, d, c->p.P, by_phase != 0, vec, nwg, t, seg, c->at<uint32_t>(L.st_cur), vals, words,
                               c->err()));
  }
  uint32_t* tiny = c->at<uint32_t>(L.st_tiny);
  uint32_t* small = c->at<uint32_t>(L.st_small);
  uint32_t* large = c->at<uint32_t>(L.st_large);
  launch_stats_classify(s, ucount, U, tiny, small, large, words);
  uint64_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  uint32_t e = 0;
  d2h(c, w, words, sizeof(w));
  d2h(c, &e, c->err(), 4);
  st = sync_read(c);
  if (st != ATREX_OK) return st;
  if (e & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  if (e & ATREX_ERRBIT_CAPACITY) return ATREX_E_INVALID_ARG;  // not the events that were aggregated
  const uint64_t vmax = w[1], ntiny = w[2], nsmall = w[3], nlarge = w[4];
  TIMED(c, "stats_sorts", ntiny + nsmall, launch_stats_sorts(s, tiny, ntiny, small, nsmall, seg, vals, q, so, capacity));
  if (nlarge) {
    int bits = 0;
    while (bits < 64 && (vmax >> bits)) ++bits;
    const int rounds = std::max(1, (bits + 7) / 8);
    const uint32_t T = nq + 2;
    uint32_t* cstart = c->at<uint32_t>(L.st_cstart);
    uint64_t* prefix = c->at<uint64_t>(L.st_prefix);
    uint32_t* want = c->at<uint32_t>(L.st_want);
    uint32_t* hist = c->at<uint32_t>(L.st_hist);
    for (uint64_t b0 = 0; b0 < nlarge; b0 += kStatsBatch) {
      const uint32_t nb = (uint32_t)std::min<uint64_t>(kStatsBatch, nlarge - b0);
      launch_fill_u32(s, cstart, nb + 1, 0);
      launch_select_init(s, large + b0, nb, seg, q, prefix, want, cstart);
      exclusive_scan_u32(s, cstart, cstart, nb + 1, c->at<void>(L.scan_tmp));
      uint32_t nchunks = 0;
      d2h(c, &nchunks, cstart + nb, 4);
      st = sync_read(c);
      if (st != ATREX_OK) return st;
      for (int r = 0; r < rounds; ++r)
        TIMED(c, "stats_select", nchunks,
              launch_select_round(s, large + b0, nb, cstart, nchunks, seg, vals, T, 8 * (rounds - 1 - r), prefix,
                                  want, hist));
      launch_select_out(s, large + b0, nb, q, prefix, so, capacity);
    }
  }
  st = sync_read(c);
  c->end_call();
  if (st != ATREX_OK) return st;
  *num_units = U;
  return U > capacity ? ATREX_E_CAPACITY : ATREX_OK;
}

// ---------------------------------------------------------------------------
// Host/device correlation join.
namespace {
struct JoinLayout {
  size_t ctrl, slot0, slot1, ref, flag, pos, scan_tmp, bytes;
  uint64_t cap;
  bool part;    // the partitioned join (its buffers share the hash tables' space)
  uint32_t bb;  // its bucket bits for max_host
};

bool join_params_ok(const atrex_join_params* p) {
  return p && p->max_kernels < (1ull << 31) && p->max_host < (1ull << 31) && p->method <= ATREX_JOIN_PARTITION &&
         !(p->method == ATREX_JOIN_PARTITION && p->max_host > kJoinPartMaxHost);
}

JoinLayout join_layout(const atrex_join_params* p) {
  JoinLayout L;
  size_t off = 0;
  auto take = [&](size_t b) {
    const size_t at = off;
    off += align_up(b ? b : 1);
    return at;
  };
  const uint64_t nk = std::max<uint64_t>(p->max_kernels, 1);
  L.part = p->method != ATREX_JOIN_HASH && p->max_host <= kJoinPartMaxHost;
  L.bb = join_part_bucket_bits(p->max_host);
  L.cap = next_pow2(std::max<uint64_t>(1024, 2 * p->max_host));
  L.ctrl = take(256);
  L.ref = take(nk * 4);
  L.flag = take(nk * 4);
  L.pos = take(nk * 4);
  const uint64_t scan_n = L.part ? std::max<uint64_t>(nk, ((uint64_t)1 << L.bb) * kJoinPartWG) : nk;
  L.scan_tmp = take(scan_tmp_bytes(scan_n));
  // the hash tables, or in the same space the partitioned join's buffers
  // (the hash join runs after it only when it gave up)
  const size_t tables = align_up(L.cap * 16) * 2;
  const size_t shared = L.part ? std::max(tables, join_part_bytes(nk, p->max_host, L.bb)) : tables;
  const size_t at = take(shared);
  L.slot0 = at;
  L.slot1 = at + align_up(L.cap * 16);
  L.bytes = off;
  return L;
}
}  // namespace

atrex_status atrex_join_workspace_bytes(const atrex_join_params* p, size_t* bytes) {
  if (!join_params_ok(p) || !bytes) return ATREX_E_INVALID_ARG;
  *bytes = join_layout(p).bytes;
  return ATREX_OK;
}

atrex_status atrex_correlate(const atrex_join_params* p, const atrex_kernel_records* k, const atrex_host_records* h,
                             const atrex_interval_records* iv, const atrex_event_out* out, uint64_t out_capacity,
                             uint8_t* source, atrex_join_result* r) {
  if (!join_params_ok(p) || !k || !h || !out || !r || !p->workspace || !aligned(p->workspace, kAlign))
    return ATREX_E_INVALID_ARG;
  *r = atrex_join_result{};
  const JoinLayout L = join_layout(p);
  if (p->workspace_bytes < L.bytes || k->n > p->max_kernels || h->n > p->max_host) return ATREX_E_CAPACITY;
  if (k->n && (!k->corr || !k->anchor || !k->stream || !k->start_ns || !k->end_ns)) return ATREX_E_INVALID_ARG;
  if (h->n && (!h->kind || !h->id || !h->key || !h->app || !h->phase)) return ATREX_E_INVALID_ARG;
  const uint64_t ni = iv ? iv->n : 0;
  if (ni >= (1ull << 31)) return ATREX_E_INVALID_ARG;
  if (ni && (!iv->stream || !iv->begin_ns || !iv->end_ns || !iv->key || !iv->app || !iv->phase))
    return ATREX_E_INVALID_ARG;
  if (out_capacity && (!out->key || !out->app || !out->phase || !out->dur_ns)) return ATREX_E_INVALID_ARG;
  if (L.part && ensure_smem_limits() != hipSuccess) return ATREX_E_DEVICE;
  char* ws = (char*)p->workspace;
  hipStream_t s = (hipStream_t)p->stream;
  JoinKernels jk{k->corr, k->anchor, k->stream, k->start_ns, k->end_ns, k->n};
  JoinHost jh{h->kind, h->id, h->key, h->app, h->phase, h->n};
  JoinIntervals ji{};
  if (ni) ji = JoinIntervals{iv->stream, iv->begin_ns, iv->end_ns, iv->key, iv->app, iv->phase, ni};
  JoinTables t{(uint64_t*)(ws + L.slot0), (uint64_t*)(ws + L.slot1), (uint32_t)(L.cap - 1)};
  JoinOut jo{out->key, out->app, out->phase, out->dur_ns};
  uint32_t* err = (uint32_t*)(ws + L.ctrl);
  unsigned long long* words = (unsigned long long*)(ws + L.ctrl + 64);
  uint32_t* flag = (uint32_t*)(ws + L.flag);
  uint32_t* ref = (uint32_t*)(ws + L.ref);
  uint32_t* pos = (uint32_t*)(ws + L.pos);
  uint32_t e = 0;
  bool hash = !L.part;
  if (L.part) {
    launch_fill_u64(s, (uint64_t*)(ws + L.ctrl), 32, 0);
    launch_join_part(s, jk, jh, ji, join_part_bucket_bits(h->n), ws + L.slot0, source, ref, flag, pos,
                     ws + L.scan_tmp, words, err);
    (void)hipMemcpyAsync(&e, err, 4, hipMemcpyDeviceToHost, s);
    if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return ATREX_E_DEVICE;
    hash = (e & ATREX_ERRBIT_SPILL) != 0;  // a bucket's ids did not fit its LDS tables
  }
  if (hash) {
    launch_fill_u64(s, (uint64_t*)(ws + L.ctrl), 32, 0);
    launch_join(s, jk, jh, ji, t, source, ref, flag, pos, ws + L.scan_tmp, jo, out_capacity, words, err, 0);
  }
  launch_join(s, jk, jh, ji, t, source, ref, flag, pos, ws + L.scan_tmp, jo, out_capacity, words, err, 1);
  uint32_t tail[2] = {0, 0};
  uint64_t by[4] = {0, 0, 0, 0};
  (void)hipMemcpyAsync(&e, err, 4, hipMemcpyDeviceToHost, s);
  (void)hipMemcpyAsync(by, words, sizeof(by), hipMemcpyDeviceToHost, s);
  if (k->n) {
    (void)hipMemcpyAsync(&tail[0], pos + (k->n - 1), 4, hipMemcpyDeviceToHost, s);
    (void)hipMemcpyAsync(&tail[1], flag + (k->n - 1), 4, hipMemcpyDeviceToHost, s);
  }
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) return ATREX_E_DEVICE;
  r->method_used = hash ? ATREX_JOIN_HASH : ATREX_JOIN_PARTITION;
  if (e & ATREX_ERRBIT_DUP) return ATREX_E_INVALID_ARG;
  if (e & ATREX_ERRBIT_RANGE) return ATREX_E_OUT_OF_RANGE;
  r->labelled = (uint64_t)tail[0] + tail[1];
  for (int i = 0; i < 4; ++i) r->by_source[i] = by[i];
  return r->labelled > out_capacity ? ATREX_E_CAPACITY : ATREX_OK;
}

atrex_status atrex_target_share(atrex_ctx* c, const atrex_share_out* out, uint64_t key_capacity,
                                uint64_t op_capacity, atrex_share_result* r) {
  if (!c || !out || !r) return ATREX_E_INVALID_ARG;
  if (!c->p.time || c->p.P != 2) return ATREX_E_INVALID_ARG;
  if (c->state < 1) return ATREX_E_STATE;
  if (key_capacity && (!out->key || !out->count || !out->dsl_ns || !out->total_ns || !out->share))
    return ATREX_E_INVALID_ARG;
  if (op_capacity && (!out->op || !out->op_shapes || !out->op_share)) return ATREX_E_INVALID_ARG;
  const Layout& L = c->L;
  ShareOut so;
  so.key = out->key;
  so.count = out->count;
  so.dsl = (uint64_t*)out->dsl_ns;
  so.total = (uint64_t*)out->total_ns;
  so.share = out->share;
  so.op = out->op;
  so.op_shapes = out->op_shapes;
  so.op_share = out->op_share;
  unsigned long long* words = c->at<unsigned long long>(L.ctrl + 2048);
  c->begin_call();
  TIMED(c, "target_share", c->G,
        launch_target_share(c->s, c->groups(), c->G, c->at<uint32_t>(L.flags), c->at<uint32_t>(L.scan),
                            c->at<uint32_t>(L.sv[0]), c->at<uint32_t>(L.sv[1]), c->at<void>(L.scan_tmp), so,
                            key_capacity, op_capacity, c->at<double>(L.sk[0]), c->at<uint32_t>(L.starts), words));
  uint64_t w[4] = {0, 0, 0, 0};
  d2h(c, w, words, sizeof(w));
  const atrex_status st = sync_read(c);
  c->end_call();
  if (st != ATREX_OK) return st;
  r->num_keys = w[0];
  r->num_ops = w[1];
  r->defined_ops = w[2];
  memcpy(&r->adoption, &w[3], sizeof(double));
  if (w[0] > key_capacity || w[1] > op_capacity) return ATREX_E_CAPACITY;
  return ATREX_OK;
}

atrex_status atrex_kernel_times(atrex_ctx* c, const char** names, float* ms, uint64_t* items, int cap, int* count) {
  if (!c || !count) return ATREX_E_INVALID_ARG;
  const int n = (int)std::min<size_t>((size_t)std::max(cap, 0), c->last_ms.size());
  for (int i = 0; i < n; ++i) {
    if (names) names[i] = c->last_names[i];
    if (ms) ms[i] = c->last_ms[i];
    if (items) items[i] = c->last_items[i];
  }
  *count = n;
  return ATREX_OK;
}

const char* atrex_path_used(atrex_ctx* c) { return c ? c->path_used : "none"; }

atrex_status atrex_aggregate_reset(atrex_ctx* c) {
  if (!c) return ATREX_E_INVALID_ARG;
  c->state = 0;
  c->S_ready = false;
  c->G = c->nops = c->nkeys = 0;
  return ATREX_OK;
}

atrex_status atrex_aggregate_destroy(atrex_ctx* c) {
  if (!c) return ATREX_E_INVALID_ARG;
  if (c->pinned) (void)hipHostFree(c->pinned);
  for (auto& t : c->timed) {
    (void)hipEventDestroy(t.a);
    (void)hipEventDestroy(t.b);
  }
  delete c;
  return ATREX_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// atrex_run without a context or workspace, for callers that cannot allocate.
// Its device memory is `scratch`, one copy per GPU for the life of the
// process.  Host code never uses the array's name as an address (it is a
// host-side stand-in): each device's address comes from hipGetSymbolAddress
// on the first call with that device current.
namespace {
constexpr int kNoAllocDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kNoAllocDevices];
}  // namespace

static __device__ __align__(256) unsigned char scratch[ATREX_NOALLOC_SCRATCH_BYTES];

namespace {
hipError_t scratch_on_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kNoAllocDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}
}  // namespace

extern "C" atrex_status atrex_run_noalloc(const atrex_noalloc_params* np, const atrex_events* ev,
                                          const atrex_groups* out, uint64_t out_capacity, const uint32_t* score_key,
                                          const double* sv, uint64_t n_score, uint32_t* op, double* op_weight,
                                          double* op_score, atrex_run_result* r) {
  if (!np || !ev || !out || !r) return ATREX_E_INVALID_ARG;
  *r = atrex_run_result{};
  if (!np->app_weight_q16 || np->num_phases < 1 || np->num_phases > 8 || np->num_apps < 1)
    return ATREX_E_INVALID_ARG;
  if (ev->n > ATREX_NOALLOC_MAX_EVENTS || out_capacity > ATREX_NOALLOC_MAX_GROUPS ||
      n_score > ATREX_NOALLOC_MAX_SCORE || (uint64_t)np->num_apps * np->num_phases > ATREX_NOALLOC_MAX_PAIRS)
    return ATREX_E_CAPACITY;
  // the layout of this call's sizes, in the compact form (global-hash engine)
  atrex_init_params ip{};
  ip.num_phases = np->num_phases;
  ip.num_apps = np->num_apps;
  ip.app_weight_q16 = np->app_weight_q16;
  ip.max_events = std::max<uint64_t>(ev->n, 1);
  ip.max_groups = std::max<uint64_t>(out_capacity, 1);
  ip.max_keys = ip.max_groups;
  ip.max_score = std::max<uint64_t>(n_score, 1);
  ip.path = ATREX_PATH_GLOBAL_HASH;
  Params p;
  atrex_status st = check_params(&ip, &p);
  if (st != ATREX_OK) return st;
  p.compact = true;
  const Layout L = make_layout(p);
  if (L.bytes > ATREX_NOALLOC_SCRATCH_BYTES) return ATREX_E_CAPACITY;
  if (ensure_smem_limits() != hipSuccess) return ATREX_E_DEVICE;
  void* ws = nullptr;
  if (scratch_on_device(&ws) != hipSuccess) return ATREX_E_DEVICE;
  // the context lives on the stack; without a mapped host buffer its status
  // readbacks are plain copies into its own host words
  atrex_ctx c;
  c.p = p;
  c.L = L;
  c.ws = (char*)ws;
  c.s = (hipStream_t)np->stream;
  c.path = ATREX_PATH_GLOBAL_HASH;
  c.flags = 0;
  c.app_weight = np->app_weight_q16;
  c.state = 0;
  c.S_ready = false;
  c.G = c.nops = c.nkeys = 0;
  c.path_used = "none";
  c.ntimed = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&c.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return ATREX_E_DEVICE;
  // the array keeps the previous call's contents: clear what must start at
  // zero (the pass-A carry table; the call clears or writes everything else),
  // with a fill kernel, and compute C = sum c_a as init does
  launch_fill_u64(c.s, c.at<uint64_t>(L.carryA), (uint64_t)p.A * p.P, 0);
  launch_sum_u32(c.s, c.app_weight, p.A, c.Csum());
  uint64_t C = 0;
  d2h(&c, &C, c.Csum(), 8);
  st = sync_read(&c);
  if (st != ATREX_OK) return st;
  if (C == 0) return ATREX_E_INVALID_ARG;
  return atrex_run(&c, ev, out, out_capacity, score_key, sv, n_score, op, op_weight, op_score, r);
}
