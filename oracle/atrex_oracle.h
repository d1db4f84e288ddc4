/*
 * atrex_oracle.h -- plain, slow, single-threaded CPU oracle for the
 * trace-event -> importance-weight path (paper §3.4 Eq. (2)-(3), §3.6
 * Eq. (4)-(6)).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link
 * or call this code: it exists so that the tests, the smoke check and the
 * benchmark's CPU-baseline leg have an independent answer to compare the GPU
 * library against.  It shares no header, helper, table or constant generator
 * with the GPU library; the status values below are restated here on purpose.
 *
 * All pointers are HOST pointers.  128-bit integers cross the ABI as two
 * uint64_t words, low word first ("lohi" arrays hold 2 words per element).
 *
 * Fixed-point definition computed here (the paper fixes no numerics; this is
 * the reading that makes every integer output the floor of an exact rational):
 *   C        = sum_a c_a                                   (c_a: Q16 card-hours)
 *   T[a,ph]  = sum of dur over events of app a in phase ph     (Eq. (2), D_a^ph)
 *   r[a,ph]  = 2^96 * c_a / (C * T[a,ph])                  (p_a / D_a^ph in Q96)
 *   rho      = floor(log2 r),  m = floor(r * 2^(55 - rho)) in [2^55, 2^56)
 *              (m = 0, rho = 0 when T = 0 or c_a = 0)
 *   v_e      = floor(dur_e * m * 2^(rho - 55))   (<= 2^96)
 *   W[k,ph]  = sum of v_e over events of key k in phase ph (Eq. (3) numerator)
 *   S[ph]    = sum_k W[k,ph];  weight[k,ph] = RN(W) / RN(S[ph])
 *   U_i      = (L_P / |Phi_i|) * sum_{ph in Phi_i} sum_{s} W[(i,s),ph],
 *              L_P = lcm(1..P), Phi_i = phases with >= 1 event of operator i
 *   w_i      = RN(U_i) / RN(sum_{j retained} U_j)             (Eq. (3))
 *   S_i      = median of correct S_j of operator i, else 0     (Eq. (5))
 *   S_agg    = sum_{i retained} w_i * S_i  (Neumaier, ascending op) (Eq. (6))
 * key = op << 16 | shape; the operator of a key is key >> 16.
 */
#ifndef ATREX_ORACLE_H
#define ATREX_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status values (same numbering as the GPU library's, restated independently). */
#define ATREX_ORACLE_OK               0
#define ATREX_ORACLE_E_INVALID_ARG   (-1)
#define ATREX_ORACLE_E_OUT_OF_RANGE  (-2)
#define ATREX_ORACLE_E_STATE         (-3)

typedef struct atrex_oracle atrex_oracle;

/* num_phases P in [1,8]; num_apps A >= 1; app_weight_q16[A] with sum > 0. */
int atrex_oracle_init(uint32_t num_phases, uint32_t num_apps,
                      const uint32_t *app_weight_q16, atrex_oracle **out);

/* Group-by of n events (n < 2^31).  Exactly once per context.  On error the
 * context is left as after init.  *num_groups = distinct (key, phase). */
int atrex_oracle_aggregate_events(atrex_oracle *o, const uint32_t *key,
                                  const uint32_t *app, const uint8_t *phase,
                                  const int64_t *dur_ns, uint64_t n,
                                  uint64_t *num_groups);

/* The same group-by with the events split into `threads` >= 1 contiguous
 * ranges, each summed by its own thread into private maps that are then merged
 * by exact integer addition: the outputs equal the single-threaded ones bit
 * for bit.  Used to time the oracle on every host core and to evaluate it on
 * the largest workloads. */
int atrex_oracle_aggregate_events_sharded(atrex_oracle *o, const uint32_t *key,
                                          const uint32_t *app, const uint8_t *phase,
                                          const int64_t *dur_ns, uint64_t n,
                                          uint32_t threads, uint64_t *num_groups);

/* Groups ascending by (key, phase); arrays sized num_groups (lohi: 2x). */
int atrex_oracle_phase_normalize(atrex_oracle *o, uint32_t *key, uint8_t *phase,
                                 uint64_t *count, uint64_t *wsum_lohi,
                                 uint64_t *raw_ns_lohi /* nullable */,
                                 double *weight, uint64_t *phase_total_lohi /* [2P] */);

/* Per (app, phase), index a*P + ph: T (lohi), event count, mantissa, exponent. */
int atrex_oracle_app_totals(const atrex_oracle *o, uint64_t *total_lohi,
                            uint64_t *count, uint64_t *mant, int32_t *rho);

/* Operators present in the trace, ascending; U (lohi) and w over all of them. */
int atrex_oracle_num_ops(const atrex_oracle *o, uint64_t *num_ops);
int atrex_oracle_op_weights(const atrex_oracle *o, uint32_t *op, uint64_t *U_lohi,
                            double *w);

/* Keys present in the trace, ascending; Eq. (3) at key granularity. */
int atrex_oracle_num_keys(const atrex_oracle *o, uint64_t *num_keys);
int atrex_oracle_key_weights(const atrex_oracle *o, uint32_t *key, uint64_t *U_lohi,
                             double *omega);

/* Eq. (4)-(6).  s[j] is S_j of score_key[j]: NaN = unit not correct,
 * otherwise it must lie in (0, 1].  Retained operators = those named by
 * score_key.  Outputs per retained operator (ascending) when non-null. */
int atrex_oracle_weighted_score(atrex_oracle *o, const uint32_t *score_key,
                                const double *s, uint64_t n, uint64_t *num_ops,
                                uint32_t *op, double *op_weight, double *op_score,
                                double *s_agg);

void atrex_oracle_destroy(atrex_oracle *o);

/* ---- Target-DSL device-time share ("adoption", §4.1 Metrics);
 * atrex_oracle_adoption.cpp.  Events of one profile: key, is_dsl (1 = the
 * invocation ran inside the target DSL, 0 = not; anything else is
 * OUT_OF_RANGE), dur >= 0; n < 2^31.
 *   D_dsl[k], D_tot[k] = sums of dur (u128);  share[k] = RN(D_dsl)/RN(D_tot),
 *   NaN when D_tot = 0 (the shape did not run);
 *   op_share[i] = exact mean of share over operator i's running shapes,
 *   rounded once (NaN when none runs);
 *   adoption = exact mean of op_share over the operators where it is
 *   defined, rounded once (NaN when none is). */
typedef struct atrex_oracle_share atrex_oracle_share;
int atrex_oracle_share_compute(const uint32_t *key, const uint8_t *is_dsl, const int64_t *dur_ns,
                               uint64_t n, atrex_oracle_share **out);
int atrex_oracle_share_sizes(const atrex_oracle_share *s, uint64_t *num_keys, uint64_t *num_ops);
/* keys ascending; count = invocations; dsl/total (lohi) */
int atrex_oracle_share_keys(const atrex_oracle_share *s, uint32_t *key, uint64_t *count,
                            uint64_t *dsl_lohi, uint64_t *total_lohi, double *share);
/* operators ascending (every operator with an invocation); shapes = running shapes */
int atrex_oracle_share_ops(const atrex_oracle_share *s, uint32_t *op, uint32_t *shapes, double *op_share,
                           double *adoption, uint64_t *defined_ops);
void atrex_oracle_share_destroy(atrex_oracle_share *s);
/* The exact mean of n >= 1 finite non-negative doubles whose mean is a normal
 * number, rounded to nearest, ties to even (NaN for n = 0). */
double atrex_oracle_exact_mean(const double *x, uint64_t n);

/* ---- Observed runtime of each unit, the deployment baseline (§3.1,
 * "Baselines and weights"); atrex_oracle_stats.cpp.  Units: keys
 * (by_phase = 0) or (key, phase) pairs (by_phase = 1), ascending.  Per unit:
 * count, total (u128, lohi), mean = RN(total)/RN(count), min, max, and for
 * each of nq <= 8 quantiles q_1e5[j] in [1, 100000] (q = q_1e5 / 1e5) the
 * nearest-rank value: rank ceil(q count) of the ascending durations.
 * OUT_OF_RANGE for phase >= num_phases or dur < 0; INVALID_ARG for a bad q. */
typedef struct atrex_oracle_stats atrex_oracle_stats;
int atrex_oracle_unit_stats(const uint32_t *key, const uint8_t *phase, const int64_t *dur_ns, uint64_t n,
                            uint32_t num_phases, int by_phase, const uint32_t *q_1e5, uint32_t nq,
                            atrex_oracle_stats **out);
int atrex_oracle_stats_size(const atrex_oracle_stats *s, uint64_t *num_units);
/* quant: [num_units][nq] */
int atrex_oracle_stats_get(const atrex_oracle_stats *s, uint32_t *key, uint8_t *phase, uint64_t *count,
                           uint64_t *total_lohi, double *mean, int64_t *mn, int64_t *mx, int64_t *quant);
void atrex_oracle_stats_destroy(atrex_oracle_stats *s);

/* ---- Host/device correlation join (§3.1); atrex_oracle_join.cpp.
 * Kernel records: corr, anchor (0 = none), stream, start, end (end < start:
 * OUT_OF_RANGE).  Host records: kind (0 launch, keyed by correlation id; 1
 * graph anchor), id (nonzero, unique per kind: INVALID_ARG otherwise), label
 * key/app/phase.  Interval records: stream, begin, end, label; ascending by
 * (stream, begin), begin <= end, not overlapping on a stream (INVALID_ARG
 * otherwise).  A kernel takes the label of its correlation id, else of its
 * anchor, else of the interval on its stream containing its start, else
 * none (source 0, 1, 2, 3).  Labelled kernels become events (key, app, phase,
 * dur = end - start) in kernel order.  n, m, mi < 2^31. */
typedef struct atrex_oracle_join atrex_oracle_join;
int atrex_oracle_correlate(const uint64_t *k_corr, const uint64_t *k_anchor, const uint32_t *k_stream,
                           const int64_t *k_start, const int64_t *k_end, uint64_t n,
                           const uint8_t *h_kind, const uint64_t *h_id, const uint32_t *h_key,
                           const uint32_t *h_app, const uint8_t *h_phase, uint64_t m,
                           const uint32_t *i_stream, const int64_t *i_begin, const int64_t *i_end,
                           const uint32_t *i_key, const uint32_t *i_app, const uint8_t *i_phase, uint64_t mi,
                           atrex_oracle_join **out);
int atrex_oracle_join_counts(const atrex_oracle_join *j, uint64_t *labelled, uint64_t *by /* [4] */);
int atrex_oracle_join_get(const atrex_oracle_join *j, uint32_t *key, uint32_t *app, uint8_t *phase, int64_t *dur,
                          uint8_t *source);
void atrex_oracle_join_destroy(atrex_oracle_join *j);

#ifdef __cplusplus
}
#endif
#endif
