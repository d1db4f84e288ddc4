/*
 * atrex_oracle_join.cpp -- plain CPU oracle for the host/device correlation
 * join that labels device kernel records with the framework operation, shape
 * and serving phase that produced them (§3.1: host events -- Python-frame
 * context -- and device events -- runtime kernel records -- are matched by
 * correlation id when one is available, otherwise by graph anchor or by
 * timestamp).  TEST INFRASTRUCTURE ONLY (see atrex_oracle.h): used by the
 * tests, the smoke check and the benchmark's CPU-baseline leg, never by the
 * product path.
 *
 * Each kernel record (corr, anchor, stream, start, end) takes, in this order:
 *   1. the label of the launch record with its correlation id (corr != 0);
 *   2. else the label of the graph-anchor record with its anchor (anchor != 0);
 *   3. else the label of the interval record on its stream that contains its
 *      start time (begin <= start < end);
 *   4. else no label.
 * Labelled kernels become events (key, app, phase, dur = end - start) in the
 * order of the kernel records.  Written for obviousness: std::map lookups
 * (the intervals keyed by (stream, begin); they do not overlap, so the one
 * that can contain a start is the last one beginning at or before it).
 */
#include "atrex_oracle.h"

#include <cstddef>
#include <iterator>
#include <map>
#include <new>
#include <utility>
#include <vector>

struct atrex_oracle_join {
  std::vector<uint32_t> key, app;
  std::vector<uint8_t> phase;
  std::vector<int64_t> dur;
  std::vector<uint8_t> source; /* per kernel record: 0 corr, 1 anchor, 2 interval, 3 none */
  uint64_t by[4];
};

extern "C" {

int atrex_oracle_correlate(const uint64_t *k_corr, const uint64_t *k_anchor, const uint32_t *k_stream,
                           const int64_t *k_start, const int64_t *k_end, uint64_t n,
                           const uint8_t *h_kind, const uint64_t *h_id, const uint32_t *h_key,
                           const uint32_t *h_app, const uint8_t *h_phase, uint64_t m,
                           const uint32_t *i_stream, const int64_t *i_begin, const int64_t *i_end,
                           const uint32_t *i_key, const uint32_t *i_app, const uint8_t *i_phase, uint64_t mi,
                           atrex_oracle_join **out) {
  if (!out) return ATREX_ORACLE_E_INVALID_ARG;
  *out = nullptr;
  if (n >= ((uint64_t)1 << 31) || m >= ((uint64_t)1 << 31) || mi >= ((uint64_t)1 << 31))
    return ATREX_ORACLE_E_INVALID_ARG;
  if (n && (!k_corr || !k_anchor || !k_stream || !k_start || !k_end)) return ATREX_ORACLE_E_INVALID_ARG;
  if (m && (!h_kind || !h_id || !h_key || !h_app || !h_phase)) return ATREX_ORACLE_E_INVALID_ARG;
  if (mi && (!i_stream || !i_begin || !i_end || !i_key || !i_app || !i_phase)) return ATREX_ORACLE_E_INVALID_ARG;
  /* host records: one label per (kind, id); ids are nonzero */
  std::map<std::pair<uint32_t, uint64_t>, uint64_t> host;
  for (uint64_t j = 0; j < m; ++j) {
    if (h_kind[j] > 1 || h_id[j] == 0) return ATREX_ORACLE_E_INVALID_ARG;
    if (!host.insert(std::make_pair(std::make_pair((uint32_t)h_kind[j], h_id[j]), j)).second)
      return ATREX_ORACLE_E_INVALID_ARG; /* the same id twice */
  }
  /* intervals: ascending (stream, begin), begin <= end, no overlap on a stream */
  for (uint64_t j = 0; j < mi; ++j) {
    if (i_end[j] < i_begin[j]) return ATREX_ORACLE_E_INVALID_ARG;
    if (j > 0 && (i_stream[j] < i_stream[j - 1] ||
                  (i_stream[j] == i_stream[j - 1] && i_begin[j] < i_end[j - 1])))
      return ATREX_ORACLE_E_INVALID_ARG;
  }
  for (uint64_t e = 0; e < n; ++e)
    if (k_end[e] < k_start[e]) return ATREX_ORACLE_E_OUT_OF_RANGE;
  std::map<std::pair<uint32_t, int64_t>, uint64_t> ivl; /* (stream, begin) -> interval */
  for (uint64_t j = 0; j < mi; ++j) ivl[std::make_pair(i_stream[j], i_begin[j])] = j;
  atrex_oracle_join *r = new (std::nothrow) atrex_oracle_join();
  if (!r) return ATREX_ORACLE_E_INVALID_ARG;
  r->by[0] = r->by[1] = r->by[2] = r->by[3] = 0;
  for (uint64_t e = 0; e < n; ++e) {
    uint8_t src = 3;
    uint32_t key = 0, app = 0;
    uint8_t ph = 0;
    for (uint32_t kind = 0; kind < 2 && src == 3; ++kind) {
      const uint64_t id = kind == 0 ? k_corr[e] : k_anchor[e];
      if (id == 0) continue;
      const auto it = host.find(std::make_pair(kind, id));
      if (it == host.end()) continue;
      src = (uint8_t)kind;
      key = h_key[it->second];
      app = h_app[it->second];
      ph = h_phase[it->second];
    }
    if (src == 3) {
      /* the last interval of the stream beginning at or before the start */
      const auto it = ivl.upper_bound(std::make_pair(k_stream[e], k_start[e]));
      if (it != ivl.begin()) {
        const uint64_t j = std::prev(it)->second;
        if (i_stream[j] == k_stream[e] && k_start[e] < i_end[j]) {
          src = 2;
          key = i_key[j];
          app = i_app[j];
          ph = i_phase[j];
        }
      }
    }
    r->source.push_back(src);
    r->by[src] += 1;
    if (src != 3) {
      r->key.push_back(key);
      r->app.push_back(app);
      r->phase.push_back(ph);
      r->dur.push_back(k_end[e] - k_start[e]);
    }
  }
  *out = r;
  return ATREX_ORACLE_OK;
}

int atrex_oracle_join_counts(const atrex_oracle_join *j, uint64_t *labelled, uint64_t *by /* [4] */) {
  if (!j || !labelled || !by) return ATREX_ORACLE_E_INVALID_ARG;
  *labelled = j->key.size();
  for (int i = 0; i < 4; ++i) by[i] = j->by[i];
  return ATREX_ORACLE_OK;
}

int atrex_oracle_join_get(const atrex_oracle_join *j, uint32_t *key, uint32_t *app, uint8_t *phase, int64_t *dur,
                          uint8_t *source) {
  if (!j) return ATREX_ORACLE_E_INVALID_ARG;
  const size_t L = j->key.size(), N = j->source.size();
  if ((L && (!key || !app || !phase || !dur)) || (N && !source)) return ATREX_ORACLE_E_INVALID_ARG;
  for (size_t i = 0; i < L; ++i) {
    key[i] = j->key[i];
    app[i] = j->app[i];
    phase[i] = j->phase[i];
    dur[i] = j->dur[i];
  }
  for (size_t i = 0; i < N; ++i) source[i] = j->source[i];
  return ATREX_ORACLE_OK;
}

void atrex_oracle_join_destroy(atrex_oracle_join *j) { delete j; }

}  // extern "C"
