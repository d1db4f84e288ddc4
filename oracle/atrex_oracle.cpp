/*
 * atrex_oracle.cpp -- plain CPU oracle for the trace-event -> importance-weight
 * path.  TEST INFRASTRUCTURE ONLY (see atrex_oracle.h): used by the tests, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product path.
 *
 * Written for obviousness, not speed: std::map group-bys, unsigned __int128
 * sums, a bit-serial 256-bit division, one thread.  Each step names the part
 * of the paper it computes:
 *   pass A  -- §3.4 Eq. (2): D_a^phi, the per-(application, phase) device time
 *   scale   -- §3.4 Eq. (3): p_a / D_a^phi as a Q96 fixed-point factor
 *   pass B  -- §3.4 Eq. (2)-(3): sum over kernels and invocations of
 *              p_a * d / D_a^phi per (operator/shape key, phase)
 *   weights -- §3.4 Eq. (3): per-phase share, phase average over Phi_i,
 *              normalisation over retained operators
 *   score   -- §3.6 Eq. (4)-(6): S_j validity, per-operator median, weighted sum
 */
#include "atrex_oracle.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <new>
#include <thread>
#include <utility>
#include <vector>

typedef unsigned __int128 u128;

namespace {

/* ---------------- 256-bit unsigned integer (4 x 64-bit limbs, LE) -------- */
struct U256 {
  uint64_t w[4];
};

U256 u256_from(u128 x) {
  U256 r;
  r.w[0] = (uint64_t)x;
  r.w[1] = (uint64_t)(x >> 64);
  r.w[2] = 0;
  r.w[3] = 0;
  return r;
}

int u256_bitlen(const U256 &a) {
  for (int i = 3; i >= 0; --i)
    if (a.w[i]) return 64 * i + 64 - __builtin_clzll(a.w[i]);
  return 0;
}

int u256_bit(const U256 &a, int i) { return (int)((a.w[i / 64] >> (i % 64)) & 1u); }

/* a * 2^s for 0 <= s < 256; bits shifted beyond 2^256 are lost (callers keep
 * every operand far below that and check it). */
U256 u256_shl(const U256 &a, int s) {
  U256 r = {{0, 0, 0, 0}};
  const int limb = s / 64, bit = s % 64;
  for (int i = 3; i >= limb; --i) {
    uint64_t v = a.w[i - limb] << bit;
    if (bit != 0 && i - limb - 1 >= 0) v |= a.w[i - limb - 1] >> (64 - bit);
    r.w[i] = v;
  }
  return r;
}

int u256_cmp(const U256 &a, const U256 &b) {
  for (int i = 3; i >= 0; --i)
    if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
  return 0;
}

/* a - b, requires a >= b. */
U256 u256_sub(const U256 &a, const U256 &b) {
  U256 r;
  uint64_t borrow = 0;
  for (int i = 0; i < 4; ++i) {
    const uint64_t t = a.w[i] - b.w[i];
    const uint64_t b1 = a.w[i] < b.w[i];
    r.w[i] = t - borrow;
    const uint64_t b2 = t < borrow;
    borrow = b1 | b2;
  }
  return r;
}

/* c * t for a 64-bit c and 128-bit t (schoolbook, two partial products). */
U256 u256_mul_64_128(uint64_t c, u128 t) {
  const u128 p0 = (u128)c * (uint64_t)t;          /* weight 2^0  */
  const u128 p1 = (u128)c * (uint64_t)(t >> 64);  /* weight 2^64 */
  U256 r;
  r.w[0] = (uint64_t)p0;
  const u128 mid = (p0 >> 64) + (u128)(uint64_t)p1;
  r.w[1] = (uint64_t)mid;
  const u128 top = (p1 >> 64) + (mid >> 64);
  r.w[2] = (uint64_t)top;
  r.w[3] = (uint64_t)(top >> 64);
  return r;
}

/* floor(num / den), den != 0: restoring binary long division, one quotient
 * bit per step from the top (Knuth, TAOCP vol. 2, §4.3.1, radix 2). */
U256 u256_div(const U256 &num, const U256 &den) {
  U256 q = {{0, 0, 0, 0}}, rem = {{0, 0, 0, 0}};
  for (int i = u256_bitlen(num) - 1; i >= 0; --i) {
    rem = u256_shl(rem, 1);
    rem.w[0] |= (uint64_t)u256_bit(num, i);
    if (u256_cmp(rem, den) >= 0) {
      rem = u256_sub(rem, den);
      q.w[i / 64] |= (uint64_t)1 << (i % 64);
    }
  }
  return q;
}

/* ---------------- the context ---------------------------------------------- */
enum State { ST_INIT = 0, ST_AGGREGATED = 1, ST_NORMALIZED = 2 };

struct AppAcc {   /* per (application, phase) */
  u128 total;     /* D_a^phi, Eq. (2) */
  uint64_t count;
};

struct GroupAcc { /* per (key, phase) */
  uint64_t count; /* invocations */
  u128 wsum;      /* sum of v_e (Q96 share) */
  u128 raw;       /* sum of dur (plain device time) */
};

const int kMantBits = 56; /* m in [2^55, 2^56) */

}  // namespace

struct atrex_oracle {
  uint32_t P, A;
  std::vector<uint32_t> c;  /* c_a, Q16 */
  uint64_t C;               /* sum_a c_a */
  State state;
  std::map<std::pair<uint32_t, uint32_t>, AppAcc> app;      /* (a, ph)  */
  std::map<std::pair<uint32_t, uint32_t>, uint64_t> mant;   /* (a, ph) -> m */
  std::map<std::pair<uint32_t, uint32_t>, int32_t> rho;     /* (a, ph) -> rho */
  std::map<std::pair<uint32_t, uint32_t>, GroupAcc> group;  /* (key, ph) */
  std::vector<u128> phase_total;                            /* S_ph */
};

namespace {

/* Scale factor of one (application, phase): the Q96 value of p_a / D_a^phi
 * (Eq. (3)), as a 56-bit mantissa m and exponent rho with
 * m * 2^(rho-55) <= 2^96 * c_a / (C * T) < (m + 1) * 2^(rho-55). */
void scale_entry(uint32_t c_a, uint64_t C, u128 T, uint64_t *m, int32_t *rho) {
  if (T == 0 || c_a == 0) { /* no device time, or no card-hours: no share */
    *m = 0;
    *rho = 0;
    return;
  }
  const U256 X = u256_shl(u256_from((u128)c_a), 96); /* 2^96 * c_a */
  const U256 Y = u256_mul_64_128(C, T);               /* C * T      */
  /* X / Y lies in (2^(r0-1), 2^(r0+1)), so floor(log2(X/Y)) is r0 or r0-1. */
  const int r0 = u256_bitlen(X) - u256_bitlen(Y);
  const bool at_least = r0 >= 0 ? u256_cmp(X, u256_shl(Y, r0)) >= 0
                                : u256_cmp(u256_shl(X, -r0), Y) >= 0;
  const int r = at_least ? r0 : r0 - 1;
  /* m = floor(X * 2^(55-r) / Y), written with non-negative shifts. */
  const int s_num = r < kMantBits - 1 ? kMantBits - 1 - r : 0;
  const int s_den = r > kMantBits - 1 ? r - (kMantBits - 1) : 0;
  const U256 q = u256_div(u256_shl(X, s_num), u256_shl(Y, s_den));
  if (q.w[1] | q.w[2] | q.w[3] || q.w[0] < ((uint64_t)1 << (kMantBits - 1)) ||
      q.w[0] >= ((uint64_t)1 << kMantBits))
    std::abort(); /* cannot happen: 2^r <= X/Y < 2^(r+1) */
  *m = q.w[0];
  *rho = r;
}

/* v = floor(d * m * 2^(rho - 55)), the Q96 share of one invocation. */
u128 event_share(int64_t d, uint64_t m, int32_t rho) {
  const u128 p = (u128)(uint64_t)d * m; /* < 2^63 * 2^56 */
  const int sh = rho - (kMantBits - 1);
  return sh >= 0 ? (p << sh) : (p >> (-sh));
}

uint64_t lcm_1_to(uint32_t P) {
  uint64_t l = 1;
  for (uint64_t k = 2; k <= P; ++k) {
    uint64_t a = l, b = k;
    while (b) { uint64_t t = a % b; a = b; b = t; }
    l = l / a * k;
  }
  return l;
}

double to_double(u128 x) { return (double)x; /* round to nearest, ties to even */ }

void put128(uint64_t *dst, size_t i, u128 x) {
  dst[2 * i] = (uint64_t)x;
  dst[2 * i + 1] = (uint64_t)(x >> 64);
}

/* Eq. (3) at a chosen granularity: unit(key) maps a key to an operator (or to
 * itself).  U = (L_P / |Phi|) * sum over phases of the unit's W, where Phi is
 * the set of phases in which the unit has at least one invocation. */
template <class UnitOf>
std::map<uint32_t, u128> eq3_units(const atrex_oracle *o, UnitOf unit) {
  std::map<uint32_t, std::vector<u128>> w;     /* unit -> W per phase */
  std::map<uint32_t, std::vector<uint64_t>> n; /* unit -> count per phase */
  for (const auto &kv : o->group) {
    const uint32_t u = unit(kv.first.first);
    auto &wv = w[u];
    auto &nv = n[u];
    if (wv.empty()) { wv.assign(o->P, 0); nv.assign(o->P, 0); }
    wv[kv.first.second] += kv.second.wsum;
    nv[kv.first.second] += kv.second.count;
  }
  const uint64_t L = lcm_1_to(o->P);
  std::map<uint32_t, u128> U;
  for (const auto &kv : w) {
    const std::vector<uint64_t> &nv = n[kv.first];
    uint64_t phases = 0;
    u128 sum = 0;
    for (uint32_t ph = 0; ph < o->P; ++ph)
      if (nv[ph] > 0) { ++phases; sum += kv.second[ph]; }
    U[kv.first] = phases ? (u128)(L / phases) * sum : 0;
  }
  return U;
}

}  // namespace

extern "C" {

int atrex_oracle_init(uint32_t num_phases, uint32_t num_apps,
                      const uint32_t *app_weight_q16, atrex_oracle **out) {
  if (!out) return ATREX_ORACLE_E_INVALID_ARG;
  *out = nullptr;
  if (num_phases < 1 || num_phases > 8 || num_apps < 1 || !app_weight_q16)
    return ATREX_ORACLE_E_INVALID_ARG;
  uint64_t C = 0;
  for (uint32_t a = 0; a < num_apps; ++a) C += app_weight_q16[a];
  if (C == 0) return ATREX_ORACLE_E_INVALID_ARG; /* p_a = c_a / C undefined */
  atrex_oracle *o = new (std::nothrow) atrex_oracle();
  if (!o) return ATREX_ORACLE_E_INVALID_ARG;
  o->P = num_phases;
  o->A = num_apps;
  o->c.assign(app_weight_q16, app_weight_q16 + num_apps);
  o->C = C;
  o->state = ST_INIT;
  *out = o;
  return ATREX_ORACLE_OK;
}

int atrex_oracle_aggregate_events(atrex_oracle *o, const uint32_t *key,
                                  const uint32_t *app, const uint8_t *phase,
                                  const int64_t *dur_ns, uint64_t n,
                                  uint64_t *num_groups) {
  if (!o || !num_groups) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state != ST_INIT) return ATREX_ORACLE_E_STATE;
  if (n >= ((uint64_t)1 << 31)) return ATREX_ORACLE_E_INVALID_ARG;
  if (n > 0 && (!key || !app || !phase || !dur_ns)) return ATREX_ORACLE_E_INVALID_ARG;
  /* O0: validate every event. */
  for (uint64_t e = 0; e < n; ++e)
    if (app[e] >= o->A || phase[e] >= o->P || dur_ns[e] < 0)
      return ATREX_ORACLE_E_OUT_OF_RANGE;
  /* Pass A, Eq. (2): D_a^phi = sum of durations of (a, phi). */
  for (uint64_t e = 0; e < n; ++e) {
    AppAcc &acc = o->app[std::make_pair(app[e], (uint32_t)phase[e])];
    acc.total += (u128)(uint64_t)dur_ns[e];
    acc.count += 1;
  }
  /* Scale, Eq. (3): p_a / D_a^phi for each (a, phi) with any invocation. */
  for (const auto &kv : o->app) {
    uint64_t m;
    int32_t r;
    scale_entry(o->c[kv.first.first], o->C, kv.second.total, &m, &r);
    o->mant[kv.first] = m;
    o->rho[kv.first] = r;
  }
  /* Pass B, Eq. (2)-(3): per (key, phase) sum of p_a * d / D_a^phi. */
  for (uint64_t e = 0; e < n; ++e) {
    const std::pair<uint32_t, uint32_t> ap(app[e], (uint32_t)phase[e]);
    const u128 v = event_share(dur_ns[e], o->mant[ap], o->rho[ap]);
    if (v > ((u128)1 << 96)) std::abort(); /* v <= d * r <= 2^96 */
    GroupAcc &g = o->group[std::make_pair(key[e], (uint32_t)phase[e])];
    g.count += 1;
    g.wsum += v;
    g.raw += (u128)(uint64_t)dur_ns[e];
  }
  /* S_phi = sum_k W[k, phi]. */
  o->phase_total.assign(o->P, 0);
  for (const auto &kv : o->group) o->phase_total[kv.first.second] += kv.second.wsum;
  o->state = ST_AGGREGATED;
  *num_groups = o->group.size();
  return ATREX_ORACLE_OK;
}

/* The same group-by with the events split into `threads` contiguous ranges,
 * one thread each.  Every thread fills private maps for its range (pass A,
 * then, once the scale exists, pass B) and the maps are merged by exact
 * integer addition, so the result is the single-threaded one bit for bit:
 * every output is a sum over events, and integer addition is exact and
 * order-free. */
int atrex_oracle_aggregate_events_sharded(atrex_oracle *o, const uint32_t *key,
                                          const uint32_t *app, const uint8_t *phase,
                                          const int64_t *dur_ns, uint64_t n,
                                          uint32_t threads, uint64_t *num_groups) {
  if (!o || !num_groups || threads < 1) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state != ST_INIT) return ATREX_ORACLE_E_STATE;
  if (n >= ((uint64_t)1 << 31)) return ATREX_ORACLE_E_INVALID_ARG;
  if (n > 0 && (!key || !app || !phase || !dur_ns)) return ATREX_ORACLE_E_INVALID_ARG;
  typedef std::pair<uint32_t, uint32_t> Key;
  const uint64_t T = threads;
  auto lo_of = [&](uint64_t t) { return n * t / T; };
  std::vector<int> bad(T, 0);
  std::vector<std::map<Key, AppAcc> > apps(T);
  std::vector<std::thread> pool;
  /* O0 and pass A (Eq. (2)) per range. */
  for (uint64_t t = 0; t < T; ++t)
    pool.emplace_back([&, t]() {
      for (uint64_t e = lo_of(t); e < lo_of(t + 1); ++e) {
        if (app[e] >= o->A || phase[e] >= o->P || dur_ns[e] < 0) { bad[t] = 1; return; }
        AppAcc &acc = apps[t][Key(app[e], (uint32_t)phase[e])];
        acc.total += (u128)(uint64_t)dur_ns[e];
        acc.count += 1;
      }
    });
  for (auto &th : pool) th.join();
  pool.clear();
  for (uint64_t t = 0; t < T; ++t)
    if (bad[t]) { o->app.clear(); return ATREX_ORACLE_E_OUT_OF_RANGE; }
  for (uint64_t t = 0; t < T; ++t)
    for (const auto &kv : apps[t]) {
      AppAcc &acc = o->app[kv.first];
      acc.total += kv.second.total;
      acc.count += kv.second.count;
    }
  apps.clear();
  /* Scale, Eq. (3), as in the single-threaded group-by. */
  for (const auto &kv : o->app) {
    uint64_t m;
    int32_t r;
    scale_entry(o->c[kv.first.first], o->C, kv.second.total, &m, &r);
    o->mant[kv.first] = m;
    o->rho[kv.first] = r;
  }
  /* Pass B, Eq. (2)-(3), per range (the scale maps are only read). */
  std::vector<std::map<Key, GroupAcc> > groups(T);
  for (uint64_t t = 0; t < T; ++t)
    pool.emplace_back([&, t]() {
      for (uint64_t e = lo_of(t); e < lo_of(t + 1); ++e) {
        const Key ap(app[e], (uint32_t)phase[e]);
        const u128 v = event_share(dur_ns[e], o->mant.at(ap), o->rho.at(ap));
        if (v > ((u128)1 << 96)) std::abort(); /* v <= d * r <= 2^96 */
        GroupAcc &g = groups[t][Key(key[e], (uint32_t)phase[e])];
        g.count += 1;
        g.wsum += v;
        g.raw += (u128)(uint64_t)dur_ns[e];
      }
    });
  for (auto &th : pool) th.join();
  for (uint64_t t = 0; t < T; ++t)
    for (const auto &kv : groups[t]) {
      GroupAcc &g = o->group[kv.first];
      g.count += kv.second.count;
      g.wsum += kv.second.wsum;
      g.raw += kv.second.raw;
    }
  o->phase_total.assign(o->P, 0);
  for (const auto &kv : o->group) o->phase_total[kv.first.second] += kv.second.wsum;
  o->state = ST_AGGREGATED;
  *num_groups = o->group.size();
  return ATREX_ORACLE_OK;
}

int atrex_oracle_phase_normalize(atrex_oracle *o, uint32_t *key, uint8_t *phase,
                                 uint64_t *count, uint64_t *wsum_lohi,
                                 uint64_t *raw_ns_lohi, double *weight,
                                 uint64_t *phase_total_lohi) {
  if (!o) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  if (!o->group.empty() && (!key || !phase || !count || !wsum_lohi || !weight))
    return ATREX_ORACLE_E_INVALID_ARG;
  if (!phase_total_lohi) return ATREX_ORACLE_E_INVALID_ARG;
  size_t i = 0;
  for (const auto &kv : o->group) { /* std::map order: (key, phase) ascending */
    key[i] = kv.first.first;
    phase[i] = (uint8_t)kv.first.second;
    count[i] = kv.second.count;
    put128(wsum_lohi, i, kv.second.wsum);
    if (raw_ns_lohi) put128(raw_ns_lohi, i, kv.second.raw);
    /* Per-phase normalisation: each phase's weights sum to one. */
    const u128 S = o->phase_total[kv.first.second];
    weight[i] = S == 0 ? 0.0 : to_double(kv.second.wsum) / to_double(S);
    ++i;
  }
  for (uint32_t ph = 0; ph < o->P; ++ph) put128(phase_total_lohi, ph, o->phase_total[ph]);
  o->state = ST_NORMALIZED;
  return ATREX_ORACLE_OK;
}

int atrex_oracle_app_totals(const atrex_oracle *o, uint64_t *total_lohi,
                            uint64_t *count, uint64_t *mant, int32_t *rho) {
  if (!o || !total_lohi || !count || !mant || !rho) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  for (uint32_t a = 0; a < o->A; ++a)
    for (uint32_t ph = 0; ph < o->P; ++ph) {
      const size_t i = (size_t)a * o->P + ph;
      const std::pair<uint32_t, uint32_t> ap(a, ph);
      const auto it = o->app.find(ap);
      put128(total_lohi, i, it == o->app.end() ? 0 : it->second.total);
      count[i] = it == o->app.end() ? 0 : it->second.count;
      mant[i] = it == o->app.end() ? 0 : o->mant.at(ap);
      rho[i] = it == o->app.end() ? 0 : o->rho.at(ap);
    }
  return ATREX_ORACLE_OK;
}

int atrex_oracle_num_ops(const atrex_oracle *o, uint64_t *num_ops) {
  if (!o || !num_ops) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  *num_ops = eq3_units(o, [](uint32_t k) { return k >> 16; }).size();
  return ATREX_ORACLE_OK;
}

int atrex_oracle_op_weights(const atrex_oracle *o, uint32_t *op, uint64_t *U_lohi,
                            double *w) {
  if (!o || !op || !U_lohi || !w) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  const std::map<uint32_t, u128> U = eq3_units(o, [](uint32_t k) { return k >> 16; });
  u128 sum = 0;
  for (const auto &kv : U) sum += kv.second;
  size_t i = 0;
  for (const auto &kv : U) {
    op[i] = kv.first;
    put128(U_lohi, i, kv.second);
    w[i] = sum == 0 ? 0.0 : to_double(kv.second) / to_double(sum);
    ++i;
  }
  return ATREX_ORACLE_OK;
}

int atrex_oracle_num_keys(const atrex_oracle *o, uint64_t *num_keys) {
  if (!o || !num_keys) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  *num_keys = eq3_units(o, [](uint32_t k) { return k; }).size();
  return ATREX_ORACLE_OK;
}

int atrex_oracle_key_weights(const atrex_oracle *o, uint32_t *key, uint64_t *U_lohi,
                             double *omega) {
  if (!o || !key || !U_lohi || !omega) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state == ST_INIT) return ATREX_ORACLE_E_STATE;
  const std::map<uint32_t, u128> U = eq3_units(o, [](uint32_t k) { return k; });
  u128 sum = 0;
  for (const auto &kv : U) sum += kv.second;
  size_t i = 0;
  for (const auto &kv : U) {
    key[i] = kv.first;
    put128(U_lohi, i, kv.second);
    omega[i] = sum == 0 ? 0.0 : to_double(kv.second) / to_double(sum);
    ++i;
  }
  return ATREX_ORACLE_OK;
}

int atrex_oracle_weighted_score(atrex_oracle *o, const uint32_t *score_key,
                                const double *s, uint64_t n, uint64_t *num_ops,
                                uint32_t *op, double *op_weight, double *op_score,
                                double *s_agg) {
  if (!o || !s_agg) return ATREX_ORACLE_E_INVALID_ARG;
  if (o->state != ST_NORMALIZED) return ATREX_ORACLE_E_STATE;
  if (n == 0 || !score_key || !s) return ATREX_ORACLE_E_INVALID_ARG;
  /* Eq. (4): S_j lies in (0, 1]; above 1 is an evaluation error, not clipped;
   * NaN marks a unit that is not correct (S_j undefined). */
  for (uint64_t j = 0; j < n; ++j)
    if (!std::isnan(s[j]) && !(s[j] > 0.0 && s[j] <= 1.0)) return ATREX_ORACLE_E_OUT_OF_RANGE;
  /* Each (operator, shape) unit is scored once. */
  std::map<uint32_t, double> by_key;
  for (uint64_t j = 0; j < n; ++j)
    if (!by_key.insert(std::make_pair(score_key[j], s[j])).second)
      return ATREX_ORACLE_E_INVALID_ARG;
  /* Retained operators: those the score names.  Eq. (5): median of the
   * correct shapes' S_j, or 0 when the operator has none. */
  std::map<uint32_t, std::vector<double>> correct;
  for (const auto &kv : by_key) {
    std::vector<double> &v = correct[kv.first >> 16];
    if (!std::isnan(kv.second)) v.push_back(kv.second);
  }
  const std::map<uint32_t, u128> U = eq3_units(o, [](uint32_t k) { return k >> 16; });
  u128 sumU = 0;
  for (const auto &kv : correct) {
    const auto it = U.find(kv.first);
    if (it != U.end()) sumU += it->second;
  }
  if (sumU == 0) return ATREX_ORACLE_E_INVALID_ARG; /* no retained weight */
  /* Eq. (6): S_agg = sum_i w_i S_i, Neumaier-compensated, ascending op. */
  double sum = 0.0, comp = 0.0;
  size_t i = 0;
  for (auto &kv : correct) {
    std::vector<double> &v = kv.second;
    double Si = 0.0;
    if (!v.empty()) {
      std::sort(v.begin(), v.end());
      const size_t h = v.size() / 2;
      Si = (v.size() % 2) ? v[h] : (v[h - 1] + v[h]) / 2.0;
    }
    const auto it = U.find(kv.first);
    const u128 Ui = it == U.end() ? 0 : it->second;
    const double wi = to_double(Ui) / to_double(sumU);
    const double x = wi * Si;
    const double t = sum + x;
    if (std::fabs(sum) >= std::fabs(x)) comp += (sum - t) + x;
    else comp += (x - t) + sum;
    sum = t;
    if (op) op[i] = kv.first;
    if (op_weight) op_weight[i] = wi;
    if (op_score) op_score[i] = Si;
    ++i;
  }
  if (num_ops) *num_ops = correct.size();
  *s_agg = sum + comp;
  return ATREX_ORACLE_OK;
}

void atrex_oracle_destroy(atrex_oracle *o) { delete o; }

}  // extern "C"
