/*
 * atrex.h -- C ABI of the MI355X (gfx950) trace-weighting library.
 *
 * It turns labelled kernel-invocation events into per-(operator/shape key,
 * serving phase) importance weights and the importance-weighted roofline
 * score of the paper:
 *   - §3.4, Eq. (2): per-(application, phase) device time D_a^phi and per
 *     (key, phase) device time, summed over every invocation;
 *   - §3.4, Eq. (3): each invocation's time divided by its application's phase
 *     total and weighted by the application's card-hour share p_a, averaged
 *     over the phases the operator runs in, normalised over operators;
 *   - §3.6, Eq. (4)-(6): per-unit roofline achievement S_j in (0, 1], per
 *     operator median over correct shapes (0 if none), weighted sum S_agg.
 *
 * Numerics (the paper fixes none; every integer output is the floor of an
 * exact rational, so it is reproducible bit for bit):
 *   C = sum_a c_a;  T[a,ph] = sum of dur (u128);
 *   r = 2^96 c_a / (C T),  rho = floor(log2 r),  m = floor(r 2^(55-rho)) in
 *   [2^55, 2^56)  (m = 0 when T = 0 or c_a = 0);
 *   v = floor(dur * m * 2^(rho-55)) <= 2^96 per event;  W[k,ph] = sum v (u128);
 *   S[ph] = sum_k W[k,ph] <= 2^96;  weight = RN(W)/RN(S[ph]) in fp64;
 *   U_i = (lcm(1..P)/|Phi_i|) sum_{ph in Phi_i} sum_shapes W, Phi_i = phases
 *   with >= 1 invocation of operator i;  w_i = RN(U_i)/RN(sum_{retained} U).
 * key = op << 16 | shape; the operator of a key is key >> 16.
 *
 * Conventions for every entry point:
 *   - returns atrex_status (0 = OK, < 0 = error); no exception crosses the ABI;
 *   - pointers marked DEVICE are HIP device pointers owned by the caller (for
 *     instance torch tensors); HOST pointers are ordinary host memory;
 *   - the library allocates no device memory: all scratch space lives in the
 *     caller's workspace (size from atrex_workspace_bytes);
 *   - all device work is enqueued on the stream given at init; each call
 *     synchronises that stream before returning, so device-detected errors
 *     come back as status codes;
 *   - a context is not thread-safe; use one context per host thread.
 * Call order: atrex_aggregate_init -> atrex_aggregate_events (once) ->
 * atrex_phase_normalize -> atrex_op_weights / atrex_key_weights /
 * atrex_weighted_score (any number of times) -> atrex_aggregate_destroy.
 * A call out of order returns ATREX_E_STATE.
 */
#ifndef ATREX_H
#define ATREX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATREX_OK = 0,
  ATREX_E_INVALID_ARG = -1,  /* bad parameter, null pointer, P not in [1,8], sum c_a = 0,
                                duplicate score key, no retained weight */
  ATREX_E_OUT_OF_RANGE = -2, /* event app >= A, phase >= P or dur < 0; score S not in (0,1] and not NaN */
  ATREX_E_STATE = -3,        /* call out of order */
  ATREX_E_CAPACITY = -4,     /* workspace too small, n > max_events, groups > max_groups */
  ATREX_E_DEVICE = -5        /* a HIP runtime error */
} atrex_status;

/* Group-by engine for the per-(key, phase) pass.  AUTO picks by capacity;
 * the others force one engine (all give identical results). */
typedef enum {
  ATREX_PATH_AUTO = 0,
  ATREX_PATH_LDS_HASH = 1,    /* per-workgroup LDS hash table, dense merge */
  ATREX_PATH_GLOBAL_HASH = 2, /* global hash table with device atomics */
  ATREX_PATH_RADIX_SORT = 3   /* partition by key digits, then LDS group-by per bucket */
} atrex_path;

/* Flags for atrex_init_params.flags */
#define ATREX_FLAG_TIMING 1u /* record per-kernel hipEvent times (atrex_kernel_times) */
#define ATREX_FLAG_RAW 2u    /* also accumulate the plain device time sum of dur per group */
#define ATREX_FLAG_APP_COUNT 4u /* also count the invocations n[a,ph] of every (app, phase) in
                                   pass A (Eq. (2)); read with atrex_get_app_totals */
#define ATREX_FLAG_DEVICE_TIME 8u /* plain device-time group-by: the events carry no application
                                     (atrex_events.app must be NULL), num_apps must be 1 and
                                     app_weight_q16 is ignored; every invocation's share is its
                                     duration, so W[k,ph] = sum of dur (u128) and
                                     atrex_get_app_totals gives T[ph] and n[ph] (counts always
                                     on).  Not with ATREX_FLAG_RAW (W is already the raw time).
                                     This is the input of atrex_target_share. */
#define ATREX_FLAG_INCREMENTAL 16u /* the events are an append-only log that grows between calls:
                                      the context keeps the per-(app, phase) totals (and counts) of
                                      the events folded so far, and each group-by runs pass A over
                                      the new events only (see atrex_refresh).  Implies
                                      ATREX_FLAG_APP_COUNT; not with ATREX_FLAG_DEVICE_TIME. */

typedef struct {
  uint64_t lo, hi; /* value = lo + hi * 2^64 */
} atrex_u128;

typedef struct atrex_ctx atrex_ctx;

typedef struct {
  uint32_t num_phases;            /* P in [1, 8] */
  uint32_t num_apps;              /* A >= 1; event app ids must be < A */
  const uint32_t *app_weight_q16; /* DEVICE [A]: card-hour weight c_a (Q16); sum must be > 0.
                                     Read during init only. */
  uint64_t max_events;            /* largest n passed to aggregate_events; n < 2^31 */
  uint64_t max_groups;            /* capacity for distinct (key, phase) groups (0: max_events) */
  uint64_t max_keys;              /* capacity for distinct keys (0: max_groups) */
  uint64_t max_score;             /* largest n passed to weighted_score (0: max_groups) */
  atrex_path path;                /* AUTO or a forced engine */
  void *workspace;                /* DEVICE, caller-owned, 256-byte aligned */
  size_t workspace_bytes;
  void *stream;                   /* hipStream_t; NULL = default stream */
  uint32_t flags;                 /* ATREX_FLAG_* */
} atrex_init_params;

typedef struct { /* DEVICE struct-of-arrays, caller-owned, read only, borrowed for the call */
  const uint32_t *key;   /* [n] op << 16 | shape */
  const uint32_t *app;   /* [n] application id < A; NULL with ATREX_FLAG_DEVICE_TIME */
  const uint8_t *phase;  /* [n] serving phase < P */
  const int64_t *dur_ns; /* [n] invocation duration, >= 0 */
  uint64_t n;            /* n <= max_events, n < 2^31 */
} atrex_events;

typedef struct {           /* DEVICE outputs, caller-allocated with num_groups rows */
  uint32_t *key;           /* [G] ascending (key, phase) */
  uint8_t *phase;          /* [G] */
  uint64_t *count;         /* [G] invocations */
  atrex_u128 *wsum;        /* [G] W[k,ph], Q96 */
  double *weight;          /* [G] RN(W)/RN(S[ph]); each phase sums to 1 */
  atrex_u128 *phase_total; /* [P] S[ph] */
  atrex_u128 *raw_ns;      /* [G] or NULL: plain device time sum of dur per group
                              (requires ATREX_FLAG_RAW at init) */
} atrex_groups;

/* Workspace size for the given parameters (workspace fields ignored).
 * HOST: p, bytes.  Fails with ATREX_E_INVALID_ARG on bad parameters. */
atrex_status atrex_workspace_bytes(const atrex_init_params *p, size_t *bytes);

/* Validates p, computes C = sum c_a on the device and prepares the context.
 * HOST: p, out.  On error *out is NULL.  Paper: §3.4 (p_a = c_a / C). */
atrex_status atrex_aggregate_init(const atrex_init_params *p, atrex_ctx **out);

/* Runs the group-by: pass A (Eq. (2), D_a^phi), the per-(app, phase) scale
 * (Eq. (3), p_a / D_a^phi), pass B (Eq. (2)-(3), per (key, phase) Q96 sums),
 * and orders the distinct groups.  Exactly once per context; after an error
 * the context returns to the initialised state.  HOST: ev (struct), num_groups.
 * Errors: OUT_OF_RANGE for a bad event (no partial results), CAPACITY when
 * n > max_events or the distinct groups exceed max_groups. */
atrex_status atrex_aggregate_events(atrex_ctx *ctx, const atrex_events *ev, uint64_t *num_groups);

/* Writes the groups (ascending key, phase) and the per-phase normalised
 * weights (§3.4, weights normalised within each serving phase), and prepares
 * Eq. (3) per operator and per key.  HOST: out (struct of DEVICE pointers),
 * num_ops and num_keys (nullable) receive the number of operators / keys. */
atrex_status atrex_phase_normalize(atrex_ctx *ctx, const atrex_groups *out, uint64_t *num_ops,
                                   uint64_t *num_keys);

/* Eq. (3) per operator over every operator in the trace, ascending op:
 * op [num_ops], U [num_ops] (u128), w [num_ops] (fp64, sums to 1). DEVICE. */
atrex_status atrex_op_weights(atrex_ctx *ctx, uint32_t *op, atrex_u128 *U, double *w);

/* Eq. (3) at key granularity, ascending key: key, U, omega [num_keys]. DEVICE. */
atrex_status atrex_key_weights(atrex_ctx *ctx, uint32_t *key, atrex_u128 *U, double *omega);

/* §3.6 Eq. (4)-(6).  score_key [n], s [n] (DEVICE): S_j of each scored
 * (operator, shape) unit; NaN = not correct, otherwise S_j must be in (0, 1]
 * (above 1 is an evaluation error, not clipped).  Retained operators = those
 * named by score_key; w_i is renormalised over them.  Outputs (DEVICE,
 * nullable, [n] capacity): op, op_weight (w_i), op_score (S_i: median of the
 * correct S_j, mean of the two middle values for an even count, else 0);
 * num_ops (HOST, nullable) = retained operators; s_agg (HOST) = sum w_i S_i.
 * Checks in order: S range (OUT_OF_RANGE), duplicate keys (INVALID_ARG), zero
 * retained weight (INVALID_ARG).  n <= max_score. */
atrex_status atrex_weighted_score(atrex_ctx *ctx, const uint32_t *score_key, const double *s,
                                  uint64_t n, uint32_t *op, double *op_weight, double *op_score,
                                  uint64_t *num_ops, double *s_agg);

typedef struct {
  uint64_t num_groups;     /* as atrex_aggregate_events returns it */
  uint64_t num_ops;        /* as atrex_phase_normalize returns them */
  uint64_t num_keys;
  uint64_t num_scored_ops; /* atrex_weighted_score's num_ops (0 without a score) */
  double s_agg;            /* atrex_weighted_score's s_agg (0 without a score) */
  uint32_t one_wait;       /* 1: the unit, weight and score kernels enqueued right behind the
                              group-by were kept, so the host waited once for the whole call;
                              0: they ran after the group-by's own wait (or not at all) */
} atrex_run_result;

/* One batch through the whole path in one call: atrex_aggregate_reset,
 * atrex_aggregate_events, atrex_phase_normalize and, when n_score > 0,
 * atrex_weighted_score, with the same outputs and the same errors in the same
 * order (§3.4 Eq. (2)-(3), §3.6 Eq. (4)-(6)).  out (DEVICE arrays as for
 * atrex_phase_normalize) holds out_capacity groups: CAPACITY when the trace
 * has more.  score_key, s, op, op_weight, op_score as for
 * atrex_weighted_score (n_score = 0: no score).  With n_score <= 8192 and
 * timing off, the normalisation and the score run back to back; when the
 * LDS engine orders the groups in one launch (the usual case for it) they
 * are enqueued right behind the group-by and the host waits once, at the
 * end; otherwise it also waits after the group-by, whose count sizes what
 * follows.  After an error the results of the stages before it stay valid as
 * with the separate calls.
 * HOST: ev (struct), out (struct), r. */
atrex_status atrex_run(atrex_ctx *ctx, const atrex_events *ev, const atrex_groups *out,
                       uint64_t out_capacity, const uint32_t *score_key, const double *s,
                       uint64_t n_score, uint32_t *op, double *op_weight, double *op_score,
                       atrex_run_result *r);

/* Per (app, phase), index a * P + ph (DEVICE, [A*P]): T = D_a^phi (u128),
 * the device time of Eq. (2) (§3.4); n (nullable) = the number of
 * invocations of (a, ph), i.e. the sum over kernels of m_{a,phi,r} in Eq. (2),
 * which needs ATREX_FLAG_APP_COUNT at init (INVALID_ARG otherwise);
 * mant / rho (nullable): the scale m, rho defined above (m = 0: no share).
 * Valid after atrex_aggregate_events (STATE before). */
atrex_status atrex_get_app_totals(atrex_ctx *ctx, atrex_u128 *T, uint64_t *n, uint64_t *mant,
                                  int32_t *rho);

/* ---- Incremental refresh of the weights (§3.4: the weights are recomputed
 * when the trace distribution is refreshed) -------------------------------
 * With ATREX_FLAG_INCREMENTAL the caller keeps the trace as an append-only
 * log of events in device memory (n < 2^31, at most max_events) and the
 * context keeps the per-(app, phase) totals of the first n_folded events.  A
 * refresh folds the new events log[n_folded, n) into those totals (pass A
 * over the new events only: D_a^phi is a plain sum), forms the Eq. (3) scale
 * from the totals of the whole log, runs pass B over the whole log (every
 * event's share depends on the new totals) and orders the groups, exactly as
 * atrex_aggregate_events over the whole log would: the results are identical
 * bit for bit.  The first n_folded events must not have changed since they
 * were folded (the library cannot check it).  On success n_folded becomes n;
 * after an error the totals and n_folded are as before.  Then
 * atrex_phase_normalize / atrex_weighted_score as usual; atrex_aggregate_reset
 * keeps the totals.  atrex_aggregate_events and atrex_run on such a context
 * fold log[n_folded, ev->n) the same way (INVALID_ARG when ev->n < n_folded).
 * Errors: INVALID_ARG unless the context has ATREX_FLAG_INCREMENTAL and
 * log->n = n_folded + n_new; as atrex_aggregate_events otherwise.
 * HOST: log (struct of DEVICE pointers), num_groups. */
atrex_status atrex_refresh(atrex_ctx *ctx, const atrex_events *log, uint64_t n_new, uint64_t *num_groups);

/* The incremental state, to checkpoint a context or to resume in another one
 * (same num_phases, num_apps and app weights): T (u128) and n (u64) per
 * (app, phase), index a * P + ph (DEVICE, [A*P]), and n_folded (HOST).
 * atrex_refresh_restore needs the initialised state (after init or reset);
 * INVALID_ARG without ATREX_FLAG_INCREMENTAL or with n_folded > max_events. */
atrex_status atrex_refresh_state(atrex_ctx *ctx, atrex_u128 *T, uint64_t *n, uint64_t *n_folded);
atrex_status atrex_refresh_restore(atrex_ctx *ctx, const atrex_u128 *T, const uint64_t *n, uint64_t n_folded);

/* ---- Observed runtime per unit (§3.1, "Baselines and weights": the runtime
 * observed in production for each retained (operator, shape) unit, kept as
 * its deployment baseline) ----------------------------------------------
 * Input: a context initialised with ATREX_FLAG_DEVICE_TIME whose
 * atrex_aggregate_events has run, and the same events again (ev->n must be
 * the aggregated count; INVALID_ARG when an event's unit is not among the
 * aggregated groups or the counts differ).  Units: every (key, phase) group
 * (by_phase != 0) or every key with its phases merged (by_phase = 0),
 * ascending.  Per unit u (DEVICE outputs of `capacity` rows; quantile_ns is
 * [capacity][nq]):
 *   count, total_ns = sum of dur (u128), mean_ns = RN(total) / count,
 *   min_ns, max_ns, and for each of nq <= 8 quantiles q_1e5[j] in [1, 100000]
 *   (HOST; q = q_1e5 / 1e5) the nearest-rank value: the duration of rank
 *   ceil(q count) in ascending order.
 * phase is 0 for merged units.  CAPACITY when the units exceed capacity
 * (*num_units still receives their number).  Valid after aggregate_events
 * (STATE before); leaves the context's state as it is.
 * HOST: ev (struct of DEVICE pointers), q_1e5, out (struct), num_units. */
typedef struct {
  uint32_t *key;
  uint8_t *phase;
  uint64_t *count;
  atrex_u128 *total_ns;
  double *mean_ns;
  int64_t *min_ns;
  int64_t *max_ns;
  int64_t *quantile_ns;
} atrex_stats_out;

atrex_status atrex_unit_stats(atrex_ctx *ctx, const atrex_events *ev, int by_phase, const uint32_t *q_1e5,
                              uint32_t nq, const atrex_stats_out *out, uint64_t capacity, uint64_t *num_units);

/* ---- Host/device correlation join (§3.1: the tracer matches host events --
 * the framework operation, its shape and serving phase from the Python frame
 * -- with device kernel records through correlation ids when available, and
 * through graph anchors or timestamps otherwise) --------------------------
 * Each kernel record takes, in this order: the label of the host launch
 * record with its correlation id (corr != 0); else of the host graph record
 * with its anchor (anchor != 0); else of the interval record on its stream
 * whose [begin, end) contains its start; else none.  Labelled records become
 * events (key, app, phase, dur = end - start) in kernel-record order: the
 * input of atrex_aggregate_events.  Context-free; all work on p->stream, which
 * the call synchronises.
 * Errors: INVALID_ARG for a host record of kind > 1, id 0 or an id repeated
 * within its kind, for intervals that are not ascending by (stream, begin),
 * have end < begin or overlap on a stream, and for bad parameters;
 * OUT_OF_RANGE for a kernel record with end < start; CAPACITY when n exceeds
 * the capacities, the workspace is too small, or more records are labelled
 * than out_capacity (r still receives the counts). */
typedef struct {            /* DEVICE, read only */
  const uint64_t *corr;     /* [n] correlation id of the launch, 0 = none */
  const uint64_t *anchor;   /* [n] graph anchor, 0 = none */
  const uint32_t *stream;   /* [n] */
  const int64_t *start_ns;  /* [n] device timestamps */
  const int64_t *end_ns;    /* [n] */
  uint64_t n;
} atrex_kernel_records;

typedef struct {            /* DEVICE, read only */
  const uint8_t *kind;      /* [n] 0 = launch (id is its correlation id), 1 = graph (id is its anchor) */
  const uint64_t *id;       /* [n] nonzero, unique within its kind */
  const uint32_t *key;      /* [n] labels: op << 16 | shape, app, serving phase */
  const uint32_t *app;
  const uint8_t *phase;
  uint64_t n;
} atrex_host_records;

typedef struct {            /* DEVICE, read only; ascending by (stream, begin_ns) */
  const uint32_t *stream;
  const int64_t *begin_ns;  /* [n] on the device timeline */
  const int64_t *end_ns;    /* [n] exclusive */
  const uint32_t *key;
  const uint32_t *app;
  const uint8_t *phase;
  uint64_t n;
} atrex_interval_records;

typedef struct {            /* DEVICE outputs, out_capacity rows */
  uint32_t *key;
  uint32_t *app;
  uint8_t *phase;
  int64_t *dur_ns;
} atrex_event_out;

/* Join methods (same results; they differ in how the host record of an id
 * is found):
 * HASH: the host records go into two open-addressing tables in device
 *   memory (one per id space), probed once per id of a kernel record;
 * PARTITION: host records and probes are scattered by the id's hash into
 *   buckets of about 2048 host records, each joined in LDS by one workgroup;
 *   for at most 2048 * 2^15 host records; it falls back to HASH when a
 *   bucket's table fills up (ids that crowd one bucket);
 * AUTO: PARTITION when max_host allows it, else HASH. */
#define ATREX_JOIN_AUTO 0u
#define ATREX_JOIN_HASH 1u
#define ATREX_JOIN_PARTITION 2u

typedef struct {
  uint64_t max_kernels;     /* kernel records per call, < 2^31 */
  uint64_t max_host;        /* host records per call, < 2^31 */
  void *workspace;          /* DEVICE, caller-owned, 256-byte aligned */
  size_t workspace_bytes;
  void *stream;             /* hipStream_t; NULL = default stream */
  uint32_t method;          /* ATREX_JOIN_*; PARTITION with max_host above its limit is INVALID_ARG */
} atrex_join_params;

typedef struct {
  uint64_t labelled;        /* events written (or wanted, on CAPACITY) */
  uint64_t by_source[4];    /* kernel records labelled by correlation id, by anchor, by interval; unlabelled */
  uint32_t method_used;     /* ATREX_JOIN_HASH or ATREX_JOIN_PARTITION */
} atrex_join_result;

/* Workspace size for p (workspace fields ignored).  HOST: p, bytes. */
atrex_status atrex_join_workspace_bytes(const atrex_join_params *p, size_t *bytes);

/* HOST: p, k, h, iv (nullable: no intervals), out (structs of DEVICE
 * pointers), r.  source (DEVICE [k->n], nullable): per kernel record 0, 1, 2
 * or 3 as above. */
atrex_status atrex_correlate(const atrex_join_params *p, const atrex_kernel_records *k, const atrex_host_records *h,
                             const atrex_interval_records *iv, const atrex_event_out *out, uint64_t out_capacity,
                             uint8_t *source, atrex_join_result *r);

/* ---- Target-DSL device-time share (§4.1, Metrics: "FlyDSL adoption") -------
 * Input: a context initialised with ATREX_FLAG_DEVICE_TIME and num_phases = 2
 * whose atrex_aggregate_events has run on one profile's kernel invocations,
 * with phase = 1 for an invocation inside the target DSL and 0 otherwise.
 * Per (operator, shape) key k:
 *   dsl_ns[k] = sum of dur inside the DSL, total_ns[k] = sum of dur (u128),
 *   share[k] = RN(dsl) / RN(total), NaN when total = 0 (the shape did not run);
 * per operator i (every operator with an invocation, ascending):
 *   op_shapes[i] = its running shapes (total > 0),
 *   op_share[i] = the exact mean of share over them, rounded once to the
 *   nearest double (NaN when none runs: the operator is then excluded);
 * adoption = the exact mean of op_share over the operators where it is
 *   defined, rounded once (NaN when none is); defined_ops = their number.
 * The means do not depend on the order of the terms.  Keys ascending. */
typedef struct {           /* DEVICE outputs, caller-allocated */
  uint32_t *key;           /* [key_capacity] */
  uint64_t *count;         /* [key_capacity] invocations */
  atrex_u128 *dsl_ns;      /* [key_capacity] */
  atrex_u128 *total_ns;    /* [key_capacity] */
  double *share;           /* [key_capacity] */
  uint32_t *op;            /* [op_capacity] */
  uint32_t *op_shapes;     /* [op_capacity] */
  double *op_share;        /* [op_capacity] */
} atrex_share_out;

typedef struct {   /* HOST result */
  uint64_t num_keys, num_ops, defined_ops;
  double adoption;
} atrex_share_result;

/* Valid once atrex_aggregate_events has run (STATE before), any number of
 * times; leaves the context's state as it is.  INVALID_ARG unless the
 * context has ATREX_FLAG_DEVICE_TIME and num_phases = 2.  CAPACITY when the
 * keys exceed key_capacity or the operators op_capacity (r still receives the
 * counts; the outputs then hold the first entries only).  HOST: out (struct of
 * DEVICE pointers), r. */
atrex_status atrex_target_share(atrex_ctx *ctx, const atrex_share_out *out, uint64_t key_capacity,
                                uint64_t op_capacity, atrex_share_result *r);

/* Per-kernel device times of the last aggregate_events / phase_normalize /
 * weighted_score call when ATREX_FLAG_TIMING was set (HOST arrays of cap
 * entries; names point to static strings).  *count = entries written. */
atrex_status atrex_kernel_times(atrex_ctx *ctx, const char **names, float *ms, uint64_t *items,
                                int cap, int *count);

/* Name of the engine the last aggregate_events used (static string). */
const char *atrex_path_used(atrex_ctx *ctx);

/* Returns the context to the initialised state so that the next batch of
 * events can be aggregated with the same workspace (previous results are
 * discarded).  HOST: ctx. */
atrex_status atrex_aggregate_reset(atrex_ctx *ctx);

atrex_status atrex_aggregate_destroy(atrex_ctx *ctx);

const char *atrex_status_str(atrex_status s);

/* ---- Allocation-free variant of atrex_run --------------------------------
 * For callers that cannot allocate device memory or create a context: tight
 * serving loops and harnesses that forbid hipMalloc.  It takes no context and
 * no workspace and calls no hipMalloc, hipFree or other allocating routine:
 * its scratch is a static device array of ATREX_NOALLOC_SCRATCH_BYTES that
 * every GPU the library is loaded on holds until the process ends.  Calls that
 * overlap on one GPU (from two host threads, or on two streams) race on that
 * array and must be serialised by the caller.  Each call clears what must
 * start at zero; nothing carries over between calls.  It synchronises the
 * stream, so it cannot be captured into a HIP graph.
 * Same outputs, statuses and order of checks as atrex_run (the per-(key,
 * phase) group-by uses the global-hash engine, whose scratch does not grow
 * with the number of events; results are identical).  CAPACITY when n,
 * out_capacity, n_score or num_apps * num_phases exceeds the limits below, or
 * the call's scratch does not fit the array. */
#define ATREX_NOALLOC_SCRATCH_BYTES (64ull << 20)
#define ATREX_NOALLOC_MAX_EVENTS (1ull << 24)
#define ATREX_NOALLOC_MAX_GROUPS (1ull << 16) /* out_capacity */
#define ATREX_NOALLOC_MAX_PAIRS (1ull << 13)  /* num_apps * num_phases */
#define ATREX_NOALLOC_MAX_SCORE 8192ull       /* n_score */

typedef struct {
  uint32_t num_phases;            /* P in [1, 8] */
  uint32_t num_apps;              /* A >= 1; event app ids must be < A */
  const uint32_t *app_weight_q16; /* DEVICE [A]: card-hour weight c_a (Q16); sum must be > 0 */
  void *stream;                   /* hipStream_t; NULL = default stream */
} atrex_noalloc_params;

/* HOST: p, ev (struct of DEVICE pointers), out (struct of DEVICE pointers), r;
 * score_key, s, op, op_weight, op_score as for atrex_run (DEVICE). */
atrex_status atrex_run_noalloc(const atrex_noalloc_params *p, const atrex_events *ev,
                               const atrex_groups *out, uint64_t out_capacity,
                               const uint32_t *score_key, const double *s, uint64_t n_score,
                               uint32_t *op, double *op_weight, double *op_score,
                               atrex_run_result *r);

#ifdef __cplusplus
}
#endif
#endif
