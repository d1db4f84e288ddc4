/*
 * atrex_oracle_stats.cpp -- plain CPU oracle for the observed runtime of each
 * (operator, shape) unit, the deployment baseline recorded for every retained
 * unit (§3.1, "Baselines and weights").  TEST INFRASTRUCTURE ONLY (see
 * atrex_oracle.h): used by the tests, the smoke check and the benchmark's
 * CPU-baseline leg, never by the product path.
 *
 * Per unit (a key, or a (key, phase) pair), over its invocations:
 *   count, total = sum of dur (u128), mean = RN(total) / RN(count),
 *   min, max, and nearest-rank quantiles: for q in (0, 1] given as an integer
 *   number of 1e-5 steps, the value of rank ceil(q count) in ascending order
 *   (the smallest duration with at least a fraction q of the invocations at
 *   or below it).
 * Written for obviousness: std::map of vectors, std::sort, integer ranks.
 */
#include "atrex_oracle.h"

#include <algorithm>
#include <map>
#include <new>
#include <utility>
#include <vector>

typedef unsigned __int128 u128;

struct atrex_oracle_stats {
  std::vector<uint32_t> key;
  std::vector<uint8_t> phase;
  std::vector<uint64_t> count;
  std::vector<u128> total;
  std::vector<double> mean;
  std::vector<int64_t> mn, mx;
  std::vector<int64_t> quant;  /* [units][nq] */
  uint32_t nq;
};

extern "C" {

int atrex_oracle_unit_stats(const uint32_t *key, const uint8_t *phase, const int64_t *dur_ns, uint64_t n,
                            uint32_t num_phases, int by_phase, const uint32_t *q_1e5, uint32_t nq,
                            atrex_oracle_stats **out) {
  if (!out) return ATREX_ORACLE_E_INVALID_ARG;
  *out = nullptr;
  if (n >= ((uint64_t)1 << 31) || num_phases < 1 || num_phases > 8 || nq > 8 || (nq && !q_1e5))
    return ATREX_ORACLE_E_INVALID_ARG;
  if (n > 0 && (!key || !phase || !dur_ns)) return ATREX_ORACLE_E_INVALID_ARG;
  for (uint32_t j = 0; j < nq; ++j)
    if (q_1e5[j] < 1 || q_1e5[j] > 100000) return ATREX_ORACLE_E_INVALID_ARG;
  for (uint64_t e = 0; e < n; ++e)
    if (phase[e] >= num_phases || dur_ns[e] < 0) return ATREX_ORACLE_E_OUT_OF_RANGE;
  /* the durations of every unit, in ascending unit order */
  std::map<std::pair<uint32_t, uint32_t>, std::vector<int64_t> > units;
  for (uint64_t e = 0; e < n; ++e)
    units[std::make_pair(key[e], by_phase ? (uint32_t)phase[e] : 0u)].push_back(dur_ns[e]);
  atrex_oracle_stats *r = new (std::nothrow) atrex_oracle_stats();
  if (!r) return ATREX_ORACLE_E_INVALID_ARG;
  r->nq = nq;
  for (auto &kv : units) {
    std::vector<int64_t> &v = kv.second;
    std::sort(v.begin(), v.end());
    const uint64_t c = v.size();
    u128 t = 0;
    for (int64_t d : v) t += (u128)(uint64_t)d;
    r->key.push_back(kv.first.first);
    r->phase.push_back((uint8_t)kv.first.second);
    r->count.push_back(c);
    r->total.push_back(t);
    r->mean.push_back((double)t / (double)c); /* RN, RN, one division */
    r->mn.push_back(v.front());
    r->mx.push_back(v.back());
    for (uint32_t j = 0; j < nq; ++j) {
      const uint64_t rank = ((uint64_t)q_1e5[j] * c + 99999) / 100000; /* ceil(q c), >= 1 */
      r->quant.push_back(v[rank - 1]);
    }
  }
  *out = r;
  return ATREX_ORACLE_OK;
}

int atrex_oracle_stats_size(const atrex_oracle_stats *s, uint64_t *num_units) {
  if (!s || !num_units) return ATREX_ORACLE_E_INVALID_ARG;
  *num_units = s->key.size();
  return ATREX_ORACLE_OK;
}

int atrex_oracle_stats_get(const atrex_oracle_stats *s, uint32_t *key, uint8_t *phase, uint64_t *count,
                           uint64_t *total_lohi, double *mean, int64_t *mn, int64_t *mx, int64_t *quant) {
  if (!s) return ATREX_ORACLE_E_INVALID_ARG;
  const size_t U = s->key.size();
  if (U && (!key || !phase || !count || !total_lohi || !mean || !mn || !mx || (s->nq && !quant)))
    return ATREX_ORACLE_E_INVALID_ARG;
  for (size_t i = 0; i < U; ++i) {
    key[i] = s->key[i];
    phase[i] = s->phase[i];
    count[i] = s->count[i];
    total_lohi[2 * i] = (uint64_t)s->total[i];
    total_lohi[2 * i + 1] = (uint64_t)(s->total[i] >> 64);
    mean[i] = s->mean[i];
    mn[i] = s->mn[i];
    mx[i] = s->mx[i];
  }
  for (size_t i = 0; i < s->quant.size(); ++i) quant[i] = s->quant[i];
  return ATREX_ORACLE_OK;
}

void atrex_oracle_stats_destroy(atrex_oracle_stats *s) { delete s; }

}  // extern "C"
