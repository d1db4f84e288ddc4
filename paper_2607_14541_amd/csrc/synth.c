/*
 * synth.c -- seeded synthetic trace generator (host, OpenMP).
 *
 * Produces labelled kernel-invocation events (key = op << 16 | shape, app,
 * phase, duration in ns) shaped like production inference traces: Zipf or
 * uniform (operator, shape) popularity, lognormal durations, a skewed
 * application mix.  It holds none of the aggregation arithmetic; both the GPU
 * library's tests/benchmark and the CPU oracle consume the arrays it writes.
 *
 * Random numbers: SplitMix64 (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) used as a counter-based
 * generator -- the i-th output of the stream seeded with mix(seed, stream) is
 * mix(state0 + (i + 1) * gamma), so any event can be generated independently.
 * Normals: Box-Muller.  Zipf: inverse CDF by binary search in a caller-built
 * cumulative table.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* Stream start state for (seed, stream). */
static inline uint64_t sm_state(uint64_t seed, uint64_t stream) {
  return sm_mix(seed * GAMMA + sm_mix(stream + 0x632BE59BD9B4E019ULL));
}

/* i-th 64-bit output of a stream. */
static inline uint64_t sm_at(uint64_t state, uint64_t i) { return sm_mix(state + (i + 1) * GAMMA); }

/* uniform in [0, 1) with 53 random bits */
static inline double u01(uint64_t x) { return (double)(x >> 11) * 0x1.0p-53; }
/* uniform in (0, 1] */
static inline double u01_open0(uint64_t x) { return (double)((x >> 11) + 1) * 0x1.0p-53; }

/* uniform integer in [0, n) (multiply-shift; n < 2^32) */
static inline uint32_t below(uint64_t x, uint32_t n) { return (uint32_t)(((x >> 32) * (uint64_t)n) >> 32); }

static inline double std_normal(uint64_t x1, uint64_t x2) {
  const double r = sqrt(-2.0 * log(u01_open0(x1)));
  return r * cos(6.283185307179586 * u01(x2));
}

/* first index r with cdf[r] > u (cdf ascending, cdf[n-1] >= 1 > u) */
static inline uint32_t inv_cdf(const double *cdf, uint32_t n, double u) {
  uint32_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const uint32_t mid = lo + (hi - lo) / 2;
    if (cdf[mid] > u) hi = mid; else lo = mid + 1;
  }
  return lo;
}

typedef struct {
  uint64_t seed;
  uint32_t key_mode;      /* 0 uniform op x shape, 1 Zipf ids, 2 hot key + uniform tail */
  uint32_t num_ops;       /* mode 0 */
  uint32_t num_shapes;    /* mode 0 */
  uint32_t zipf_n;        /* mode 1: number of ids; cdf/perm have zipf_n entries */
  uint32_t shape_bits;    /* mode 1/2: op = id >> shape_bits (+ op_base), shape = id & mask */
  uint32_t op_base;       /* mode 2: tail ops start here */
  uint32_t tail_n;        /* mode 2: tail ids */
  double hot_p;           /* mode 2: probability of the hot key (op 0, shape 0) */
  uint32_t num_phases;
  double phase0_frac;     /* > 0 and num_phases == 2: P(phase 0); else uniform */
  uint32_t num_apps;
  uint32_t dur_mode;      /* 0 lognormal(mu, sigma) clamped to [0, 2^62]; 1 uniform int [lo, hi] */
  double mu, sigma;
  int64_t dur_lo, dur_hi;
} atrex_synth_cfg;

enum { S_KEY = 1, S_KEY2 = 2, S_APP = 3, S_PHASE = 4, S_DUR1 = 5, S_DUR2 = 6 };

void atrex_synth_events(const atrex_synth_cfg *cfg, const double *cdf, const uint32_t *perm,
                        uint64_t begin, uint64_t n, uint32_t *key, uint32_t *app,
                        uint8_t *phase, int64_t *dur) {
  const uint64_t stK = sm_state(cfg->seed, S_KEY), stK2 = sm_state(cfg->seed, S_KEY2);
  const uint64_t stA = sm_state(cfg->seed, S_APP), stP = sm_state(cfg->seed, S_PHASE);
  const uint64_t stD1 = sm_state(cfg->seed, S_DUR1), stD2 = sm_state(cfg->seed, S_DUR2);
  const uint32_t smask = (1u << cfg->shape_bits) - 1u;
#pragma omp parallel for schedule(static, 65536)
  for (int64_t j = 0; j < (int64_t)n; ++j) {
    const uint64_t i = begin + (uint64_t)j;
    uint32_t op, shape;
    const uint64_t rk = sm_at(stK, i);
    if (cfg->key_mode == 0) {
      op = below(rk, cfg->num_ops);
      shape = below(sm_at(stK2, i), cfg->num_shapes);
    } else if (cfg->key_mode == 1) {
      const uint32_t id = perm[inv_cdf(cdf, cfg->zipf_n, u01(rk))];
      op = id >> cfg->shape_bits;
      shape = id & smask;
    } else {
      if (u01(rk) < cfg->hot_p) {
        op = 0;
        shape = 0;
      } else {
        const uint32_t id = below(sm_at(stK2, i), cfg->tail_n);
        op = cfg->op_base + (id >> cfg->shape_bits);
        shape = id & smask;
      }
    }
    key[j] = (op << 16) | (shape & 0xFFFFu);
    app[j] = below(sm_at(stA, i), cfg->num_apps);
    const uint64_t rp = sm_at(stP, i);
    if (cfg->num_phases == 2 && cfg->phase0_frac > 0.0)
      phase[j] = u01(rp) < cfg->phase0_frac ? 0 : 1;
    else
      phase[j] = (uint8_t)below(rp, cfg->num_phases);
    if (cfg->dur_mode == 0) {
      const double z = std_normal(sm_at(stD1, i), sm_at(stD2, i));
      double d = exp(cfg->mu + cfg->sigma * z);
      if (d > 4611686018427387904.0) d = 4611686018427387904.0; /* 2^62 */
      dur[j] = llround(d);
    } else {
      const uint64_t span = (uint64_t)(cfg->dur_hi - cfg->dur_lo) + 1u;
      dur[j] = cfg->dur_lo + (int64_t)(sm_at(stD1, i) % span);
    }
  }
}

/* n raw 64-bit outputs of stream `stream` starting at index `begin`. */
void atrex_synth_u64(uint64_t seed, uint64_t stream, uint64_t begin, uint64_t n, uint64_t *out) {
  const uint64_t st = sm_state(seed, stream);
#pragma omp parallel for schedule(static, 65536)
  for (int64_t j = 0; j < (int64_t)n; ++j) out[j] = sm_at(st, begin + (uint64_t)j);
}

/* n standard normals (Box-Muller on two sub-streams). */
void atrex_synth_normal(uint64_t seed, uint64_t stream, uint64_t n, double *out) {
  const uint64_t s1 = sm_state(seed, stream), s2 = sm_state(seed, stream + 1000003u);
  for (uint64_t j = 0; j < n; ++j) out[j] = std_normal(sm_at(s1, j), sm_at(s2, j));
}
