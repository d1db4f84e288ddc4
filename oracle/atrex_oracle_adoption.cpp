/*
 * atrex_oracle_adoption.cpp -- plain CPU oracle for the target-DSL device-time
 * share ("adoption", §4.1, Metrics).  TEST INFRASTRUCTURE ONLY (see
 * atrex_oracle.h): used by the tests, the smoke check and the benchmark's
 * CPU-baseline leg, never by the product path.
 *
 * What it computes, from the definition in §4.1 (Metrics):
 *   per (operator, shape) key k, over the kernel invocations of one profile:
 *     D_dsl[k] = sum of dur over invocations inside the target DSL,
 *     D_tot[k] = sum of dur over all invocations,
 *     share[k] = RN(D_dsl) / RN(D_tot)   (undefined, NaN, when D_tot = 0);
 *   a shape "runs" when D_tot > 0;
 *   per operator i: the mean of share[k] over its running shapes (NaN when it
 *     has none: the operator is then excluded, not scored 0);
 *   adoption: the mean of the operator means over the operators where it is
 *     defined (NaN when there are none).
 * Every mean here is the exact mean of its fp64 terms rounded once to the
 * nearest double (ties to even), so it does not depend on the order of the
 * terms.  Written for obviousness: std::map group-by, unsigned __int128 sums,
 * a plain big-integer exact sum and a schoolbook division.
 */
#include "atrex_oracle.h"

#include <cmath>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <map>
#include <new>
#include <vector>

typedef unsigned __int128 u128;

namespace {

/* Non-negative big integer, 32-bit limbs, least significant first. */
struct Big {
  std::vector<uint32_t> d;
  void trim() {
    while (!d.empty() && d.back() == 0) d.pop_back();
  }
  bool zero() const { return d.empty(); }
  int bitlen() const {
    if (d.empty()) return 0;
    return 32 * (int)(d.size() - 1) + 32 - __builtin_clz(d.back());
  }
  int bit(int i) const {
    const size_t w = (size_t)i / 32;
    return w < d.size() ? (int)((d[w] >> (i % 32)) & 1u) : 0;
  }
};

/* a += x * 2^s for a 64-bit x. */
void big_add_shifted(Big &a, uint64_t x, int s) {
  if (x == 0) return;
  const size_t w = (size_t)s / 32, b = (size_t)s % 32;
  /* x * 2^b spans at most three 32-bit limbs */
  const u128 v = (u128)x << b;
  const uint32_t parts[3] = {(uint32_t)v, (uint32_t)(v >> 32), (uint32_t)(v >> 64)};
  if (a.d.size() < w + 4) a.d.resize(w + 4, 0);
  uint64_t carry = 0;
  for (size_t i = 0; i < 3 || carry; ++i) {
    if (w + i >= a.d.size()) a.d.push_back(0);
    const uint64_t t = (uint64_t)a.d[w + i] + (i < 3 ? parts[i] : 0) + carry;
    a.d[w + i] = (uint32_t)t;
    carry = t >> 32;
  }
  a.trim();
}

/* a * 2^s */
Big big_shl(const Big &a, int s) {
  Big r;
  if (a.zero()) return r;
  const size_t w = (size_t)s / 32, b = (size_t)s % 32;
  r.d.assign(w, 0);
  uint32_t carry = 0;
  for (uint32_t x : a.d) {
    r.d.push_back(b ? (x << b) | carry : x);
    carry = b ? x >> (32 - b) : 0;
  }
  if (carry) r.d.push_back(carry);
  r.trim();
  return r;
}

/* floor(a / n) and a mod n for 0 < n < 2^32 (schoolbook, most significant
 * limb first). */
Big big_divmod(const Big &a, uint32_t n, uint32_t *rem) {
  Big q;
  q.d.assign(a.d.size(), 0);
  uint64_t r = 0;
  for (size_t i = a.d.size(); i-- > 0;) {
    const uint64_t cur = (r << 32) | a.d[i];
    q.d[i] = (uint32_t)(cur / n);
    r = cur % n;
  }
  q.trim();
  *rem = (uint32_t)r;
  return q;
}

/* The exact sum of finite non-negative doubles, kept as an integer count of
 * 2^-1074 (the smallest subnormal), so every double is an exact multiple. */
struct ExactSum {
  Big s;
  void add(double x) {
    if (!(x >= 0.0) || std::isinf(x)) std::abort(); /* only finite x >= 0 are summed */
    if (x == 0.0) return;
    int e;
    const double f = std::frexp(x, &e);                 /* x = f 2^e, f in [0.5, 1) */
    const uint64_t m = (uint64_t)std::ldexp(f, 53);      /* x = m 2^(e-53), exact */
    const int s_ = e - 53 + 1074;                        /* x = m 2^s_ * 2^-1074 */
    if (s_ >= 0) big_add_shifted(s, m, s_);
    else big_add_shifted(s, m >> (-s_), 0);  /* subnormal: the low bits of m are 0 */
  }
};

/* The exact mean sum / n (n >= 1) rounded to the nearest double, ties to
 * even.  The quotient is formed with at least 64 significant bits and a
 * sticky bit for the rest, then rounded once. */
double exact_mean(const ExactSum &acc, uint64_t n) {
  if (n == 0 || n >= ((uint64_t)1 << 32)) std::abort();
  if (acc.s.zero()) return 0.0;
  const int t = 64 + 33;
  uint32_t rem = 0;
  const Big q = big_divmod(big_shl(acc.s, t), (uint32_t)n, &rem);
  /* value = (q + rem / n) * 2^(-1074 - t), q >= 2^64 */
  const int L = q.bitlen();
  const int drop = L - 53;
  uint64_t mant = 0;
  for (int i = L - 1; i >= drop; --i) mant = (mant << 1) | (uint64_t)q.bit(i);
  /* the dropped bits against one half of the last kept bit */
  const bool half = q.bit(drop - 1) != 0;
  bool sticky = rem != 0;
  for (int i = drop - 2; i >= 0 && !sticky; --i) sticky = q.bit(i) != 0;
  if (half && (sticky || (mant & 1u))) ++mant;
  int exp2 = drop - 1074 - t;
  if (mant == ((uint64_t)1 << 53)) {
    mant >>= 1;
    ++exp2;
  }
  const double r = std::ldexp((double)mant, exp2);
  if (!(r >= std::numeric_limits<double>::min())) std::abort(); /* normal results only */
  return r;
}

struct KeyTime {
  uint64_t count = 0;
  u128 dsl = 0, total = 0;
};

void put128(uint64_t *dst, size_t i, u128 x) {
  dst[2 * i] = (uint64_t)x;
  dst[2 * i + 1] = (uint64_t)(x >> 64);
}

}  // namespace

struct atrex_oracle_share {
  std::map<uint32_t, KeyTime> keys;   /* key -> times, ascending */
  std::map<uint32_t, double> share;   /* key -> share (NaN when D_tot = 0) */
  struct Op {
    uint32_t shapes;   /* running shapes */
    double mean;       /* NaN when no shape runs */
  };
  std::map<uint32_t, Op> ops;         /* operator -> mean share */
  double adoption;
  uint64_t defined_ops;
};

extern "C" {

double atrex_oracle_exact_mean(const double *x, uint64_t n) {
  if (n == 0 || !x) return std::numeric_limits<double>::quiet_NaN();
  ExactSum acc;
  for (uint64_t i = 0; i < n; ++i) acc.add(x[i]);
  return exact_mean(acc, n);
}

int atrex_oracle_share_compute(const uint32_t *key, const uint8_t *is_dsl, const int64_t *dur_ns,
                               uint64_t n, atrex_oracle_share **out) {
  if (!out) return ATREX_ORACLE_E_INVALID_ARG;
  *out = nullptr;
  if (n >= ((uint64_t)1 << 31)) return ATREX_ORACLE_E_INVALID_ARG;
  if (n > 0 && (!key || !is_dsl || !dur_ns)) return ATREX_ORACLE_E_INVALID_ARG;
  /* every invocation is inside the target DSL (1) or not (0), with dur >= 0 */
  for (uint64_t e = 0; e < n; ++e)
    if (is_dsl[e] > 1 || dur_ns[e] < 0) return ATREX_ORACLE_E_OUT_OF_RANGE;
  atrex_oracle_share *r = new (std::nothrow) atrex_oracle_share();
  if (!r) return ATREX_ORACLE_E_INVALID_ARG;
  /* device time per (operator, shape): in the target DSL, and in total */
  for (uint64_t e = 0; e < n; ++e) {
    KeyTime &k = r->keys[key[e]];
    k.count += 1;
    k.total += (u128)(uint64_t)dur_ns[e];
    if (is_dsl[e]) k.dsl += (u128)(uint64_t)dur_ns[e];
  }
  /* per-shape share; per-operator mean over the shapes that ran */
  std::map<uint32_t, std::vector<double> > running;
  for (const auto &kv : r->keys) {
    const uint32_t op = kv.first >> 16;
    std::vector<double> &v = running[op];  /* every operator in the profile is listed */
    if (kv.second.total == 0) {
      r->share[kv.first] = std::numeric_limits<double>::quiet_NaN();
      continue;
    }
    const double s = (double)kv.second.dsl / (double)kv.second.total; /* RN, RN, one division */
    r->share[kv.first] = s;
    v.push_back(s);
  }
  std::vector<double> means;
  for (const auto &kv : running) {
    atrex_oracle_share::Op o;
    o.shapes = (uint32_t)kv.second.size();
    o.mean = kv.second.empty() ? std::numeric_limits<double>::quiet_NaN()
                               : atrex_oracle_exact_mean(kv.second.data(), kv.second.size());
    if (!kv.second.empty()) means.push_back(o.mean);
    r->ops[kv.first] = o;
  }
  /* the mean over the operators where the share is defined */
  r->defined_ops = means.size();
  r->adoption = means.empty() ? std::numeric_limits<double>::quiet_NaN()
                              : atrex_oracle_exact_mean(means.data(), means.size());
  *out = r;
  return ATREX_ORACLE_OK;
}

int atrex_oracle_share_sizes(const atrex_oracle_share *s, uint64_t *num_keys, uint64_t *num_ops) {
  if (!s || !num_keys || !num_ops) return ATREX_ORACLE_E_INVALID_ARG;
  *num_keys = s->keys.size();
  *num_ops = s->ops.size();
  return ATREX_ORACLE_OK;
}

int atrex_oracle_share_keys(const atrex_oracle_share *s, uint32_t *key, uint64_t *count,
                            uint64_t *dsl_lohi, uint64_t *total_lohi, double *share) {
  if (!s || (!s->keys.empty() && (!key || !count || !dsl_lohi || !total_lohi || !share)))
    return ATREX_ORACLE_E_INVALID_ARG;
  size_t i = 0;
  for (const auto &kv : s->keys) {
    key[i] = kv.first;
    count[i] = kv.second.count;
    put128(dsl_lohi, i, kv.second.dsl);
    put128(total_lohi, i, kv.second.total);
    share[i] = s->share.at(kv.first);
    ++i;
  }
  return ATREX_ORACLE_OK;
}

int atrex_oracle_share_ops(const atrex_oracle_share *s, uint32_t *op, uint32_t *shapes, double *op_share,
                           double *adoption, uint64_t *defined_ops) {
  if (!s || !adoption || !defined_ops || (!s->ops.empty() && (!op || !shapes || !op_share)))
    return ATREX_ORACLE_E_INVALID_ARG;
  size_t i = 0;
  for (const auto &kv : s->ops) {
    op[i] = kv.first;
    shapes[i] = kv.second.shapes;
    op_share[i] = kv.second.mean;
    ++i;
  }
  *adoption = s->adoption;
  *defined_ops = s->defined_ops;
  return ATREX_ORACLE_OK;
}

void atrex_oracle_share_destroy(atrex_oracle_share *s) { delete s; }

}  // extern "C"
