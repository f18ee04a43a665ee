/*
 * Seeded synthetic workload generator (host, plain C).
 *
 * This module produces the *inputs* of the serving simulator: request arrival
 * traces and the uniform draws the problem builders turn into model latencies,
 * weights and placement permutations.  It holds none of the simulator's
 * arithmetic (dispatch, pipeline recurrence, admission, counting), so the
 * simulator and its CPU checker can both consume what it writes.
 *
 * Arrival model (paper, Sec. 3.1 and Sec. 6.2/6.5): each model receives an
 * independent Gamma renewal process parameterised by a rate lambda and a
 * coefficient of variation cv.  Inter-arrival X ~ Gamma(shape = 1/cv^2,
 * scale = cv^2/lambda), so E[X] = 1/lambda and sd(X)/E[X] = cv; cv = 1 is the
 * Poisson process the paper uses in Sec. 3.1 and Sec. 3.4.  The first arrival
 * of a model is at X_1, the j-th at t_{j-1} + X_j (left-to-right fp64 sum),
 * and only arrivals with t < duration are kept.  All models are merged into one
 * trace ordered by (t, model id, per-model index), so equal timestamps (common
 * when cv >= 3 because many gaps fall below half an ulp of t) have a defined
 * order.
 *
 * Random numbers: a counter-based generator.  Stream key k and counter c give
 * u64 = mix64(k + (c + 1) * 0x9E3779B97F4A7C15), where mix64 is the 64-bit
 * finaliser of SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  Uniforms are
 * ((u64 >> 11) + 0.5) * 2^-53, strictly inside (0, 1).
 *
 * Gamma variates: Marsaglia and Tsang, "A simple method for generating gamma
 * variables", ACM TOMS 26(3), 2000: for shape a >= 1 with d = a - 1/3,
 * c = 1/sqrt(9d), draw a standard normal x and v = (1 + c x)^3, accept d*v
 * when v > 0 and either u < 1 - 0.0331 x^4 or log u < x^2/2 + d(1 - v + log v).
 * For a < 1 the boost from the same paper, Gamma(a) = Gamma(a + 1) * U^(1/a),
 * is used.
 * Standard normals come from Marsaglia's polar method (one value per
 * accepted pair; the second is discarded so every draw consumes a fixed
 * pattern of counters).
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC (no FMA
 * contraction, so results do not depend on the host's vector ISA).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/alpaserve_gen.h"

#define GOLDEN 0x9E3779B97F4A7C15ULL

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

typedef struct {
  uint64_t key;
  uint64_t ctr;
} stream_t;

static uint64_t next_u64(stream_t* s) {
  uint64_t r = mix64(s->key + (s->ctr + 1) * GOLDEN);
  s->ctr++;
  return r;
}

static double next_uniform(stream_t* s) {
  return ((double)(next_u64(s) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

uint64_t as_gen_key(uint64_t seed, uint64_t purpose, uint64_t index) {
  /* Three chained finaliser rounds: distinct (seed, purpose, index) triples
   * give unrelated stream keys. */
  uint64_t k = mix64(seed + GOLDEN);
  k = mix64(k ^ (purpose + 0x632BE59BD9B4E019ULL));
  k = mix64(k ^ (index + 0x8CB92BA72F3D8DD7ULL));
  return k;
}

int as_gen_uniforms(uint64_t key, int64_t n, double* out) {
  if (n < 0 || (n > 0 && out == NULL)) return AS_GEN_E_INVALID_ARG;
  stream_t s = {key, 0};
  for (int64_t i = 0; i < n; ++i) out[i] = next_uniform(&s);
  return AS_GEN_OK;
}

static double std_normal(stream_t* s) {
  for (;;) {
    double a = 2.0 * next_uniform(s) - 1.0;
    double b = 2.0 * next_uniform(s) - 1.0;
    double q = a * a + b * b;
    if (q > 0.0 && q < 1.0) return a * sqrt(-2.0 * log(q) / q);
  }
}

/* Gamma(shape a, scale 1) for a >= 1. */
static double gamma_mt(stream_t* s, double a) {
  const double d = a - 1.0 / 3.0;
  const double c = 1.0 / sqrt(9.0 * d);
  for (;;) {
    double x = std_normal(s);
    double v = 1.0 + c * x;
    if (v <= 0.0) continue;
    v = v * v * v;
    double u = next_uniform(s);
    double x2 = x * x;
    if (u < 1.0 - 0.0331 * (x2 * x2)) return d * v;
    if (log(u) < 0.5 * x2 + d * (1.0 - v + log(v))) return d * v;
  }
}

double as_gen_gamma(uint64_t key, uint64_t counter, double shape, uint64_t* counter_out) {
  stream_t s = {key, counter};
  double x;
  if (shape >= 1.0) {
    x = gamma_mt(&s, shape);
  } else {
    double g = gamma_mt(&s, shape + 1.0);
    double u = next_uniform(&s);
    x = g * pow(u, 1.0 / shape);
  }
  if (counter_out) *counter_out = s.ctr;
  return x;
}

typedef struct {
  double t;
  int32_t model;
  int64_t idx;
} arrival_t;

static int cmp_arrival(const void* pa, const void* pb) {
  const arrival_t* a = (const arrival_t*)pa;
  const arrival_t* b = (const arrival_t*)pb;
  if (a->t < b->t) return -1;
  if (a->t > b->t) return 1;
  if (a->model != b->model) return a->model < b->model ? -1 : 1;
  if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
  return 0;
}

/* Per-model arrivals for one model: appends to a growing array. */
static int gen_model(uint64_t seed, int32_t m, double rate, double cv, double duration,
                     arrival_t** buf, int64_t* len, int64_t* cap) {
  if (rate <= 0.0) return AS_GEN_OK;
  const double shape = 1.0 / (cv * cv);
  const double scale = (cv * cv) / rate;
  uint64_t key = as_gen_key(seed, AS_GEN_PURPOSE_ARRIVAL, (uint64_t)m);
  uint64_t ctr = 0;
  double t = 0.0;
  int64_t j = 0;
  for (;;) {
    double x = as_gen_gamma(key, ctr, shape, &ctr) * scale;
    t = t + x;
    if (!(t < duration)) break;
    if (*len == *cap) {
      int64_t ncap = *cap ? *cap * 2 : 4096;
      arrival_t* nb = (arrival_t*)realloc(*buf, (size_t)ncap * sizeof(arrival_t));
      if (!nb) return AS_GEN_E_NOMEM;
      *buf = nb;
      *cap = ncap;
    }
    (*buf)[*len].t = t;
    (*buf)[*len].model = m;
    (*buf)[*len].idx = j++;
    (*len)++;
  }
  return AS_GEN_OK;
}

/* Appends one arrival; grows the buffer. */
static int push_arrival(arrival_t** buf, int64_t* len, int64_t* cap, double t, int32_t m, int64_t j) {
  if (*len == *cap) {
    int64_t ncap = *cap ? *cap * 2 : 4096;
    arrival_t* nb = (arrival_t*)realloc(*buf, (size_t)ncap * sizeof(arrival_t));
    if (!nb) return AS_GEN_E_NOMEM;
    *buf = nb;
    *cap = ncap;
  }
  (*buf)[*len].t = t;
  (*buf)[*len].model = m;
  (*buf)[*len].idx = j;
  (*len)++;
  return AS_GEN_OK;
}

/* Sort the collected arrivals and copy them out (shared by both traces). */
static int emit_trace(arrival_t* buf, int64_t len, int64_t capacity, double* t_out, int32_t* m_out,
                      int64_t* n_out) {
  *n_out = len;
  if (len > capacity || (len > 0 && (t_out == NULL || m_out == NULL))) {
    free(buf);
    return AS_GEN_E_CAPACITY;
  }
  if (len > 0) qsort(buf, (size_t)len, sizeof(arrival_t), cmp_arrival);
  for (int64_t i = 0; i < len; ++i) {
    t_out[i] = buf[i].t;
    m_out[i] = buf[i].model;
  }
  free(buf);
  return AS_GEN_OK;
}

int as_gen_trace_windowed(uint64_t seed, int32_t n_models, int32_t n_windows, double window,
                          const double* rate, const double* cv, int64_t capacity, double* t_out,
                          int32_t* m_out, int64_t* n_out) {
  if (n_models < 0 || n_windows < 0 || n_out == NULL || capacity < 0) return AS_GEN_E_INVALID_ARG;
  if (!(window > 0.0) || !isfinite(window)) return AS_GEN_E_INVALID_ARG;
  const int64_t cells = (int64_t)n_models * n_windows;
  if (cells > 0 && (rate == NULL || cv == NULL)) return AS_GEN_E_INVALID_ARG;
  for (int64_t i = 0; i < cells; ++i)
    if (!(rate[i] >= 0.0) || !isfinite(rate[i]) || !(cv[i] > 0.0) || !isfinite(cv[i]))
      return AS_GEN_E_INVALID_ARG;
  arrival_t* buf = NULL;
  int64_t len = 0, cap = 0;
  for (int32_t m = 0; m < n_models; ++m) {
    int64_t j = 0;  /* per-model arrival index, across windows */
    for (int32_t w = 0; w < n_windows; ++w) {
      const double r = rate[(int64_t)m * n_windows + w];
      if (r <= 0.0) continue;
      const double c = cv[(int64_t)m * n_windows + w];
      const double shape = 1.0 / (c * c);
      const double scale = (c * c) / r;
      const double start = (double)w * window;
      const double end = (double)(w + 1) * window;
      const uint64_t key =
          as_gen_key(seed, AS_GEN_PURPOSE_WINDOW, (uint64_t)m * (uint64_t)n_windows + (uint64_t)w);
      uint64_t ctr = 0;
      double t = start;
      for (;;) {
        t = t + as_gen_gamma(key, ctr, shape, &ctr) * scale;
        if (!(t < end)) break;
        const int rc = push_arrival(&buf, &len, &cap, t, m, j++);
        if (rc != AS_GEN_OK) {
          free(buf);
          return rc;
        }
      }
    }
  }
  return emit_trace(buf, len, capacity, t_out, m_out, n_out);
}

int as_gen_trace(uint64_t seed, int32_t n_models, const double* rate, double cv,
                 double duration, int64_t capacity, double* t_out, int32_t* m_out,
                 int64_t* n_out) {
  if (n_models < 0 || (n_models > 0 && rate == NULL) || n_out == NULL) return AS_GEN_E_INVALID_ARG;
  if (!(cv > 0.0) || !isfinite(cv) || !(duration >= 0.0) || !isfinite(duration) || capacity < 0)
    return AS_GEN_E_INVALID_ARG;
  for (int32_t m = 0; m < n_models; ++m)
    if (!(rate[m] >= 0.0) || !isfinite(rate[m])) return AS_GEN_E_INVALID_ARG;
  arrival_t* buf = NULL;
  int64_t len = 0, cap = 0;
  for (int32_t m = 0; m < n_models; ++m) {
    int rc = gen_model(seed, m, rate[m], cv, duration, &buf, &len, &cap);
    if (rc != AS_GEN_OK) {
      free(buf);
      return rc;
    }
  }
  *n_out = len;
  if (len > capacity || (len > 0 && (t_out == NULL || m_out == NULL))) {
    free(buf);
    return AS_GEN_E_CAPACITY;
  }
  if (len > 0) qsort(buf, (size_t)len, sizeof(arrival_t), cmp_arrival);
  for (int64_t i = 0; i < len; ++i) {
    t_out[i] = buf[i].t;
    m_out[i] = buf[i].model;
  }
  free(buf);
  return AS_GEN_OK;
}

int as_gen_permutations(uint64_t seed, uint64_t purpose, uint64_t first_index, int64_t count,
                        int32_t n, int32_t* out) {
  if (count < 0 || n < 0 || (count > 0 && n > 0 && out == NULL)) return AS_GEN_E_INVALID_ARG;
  for (int64_t r = 0; r < count; ++r) {
    int32_t* p = out + r * (int64_t)n;
    stream_t s = {as_gen_key(seed, purpose, first_index + (uint64_t)r), 0};
    for (int32_t i = 0; i < n; ++i) p[i] = i;
    /* Fisher-Yates (Durstenfeld): for i = n-1 .. 1 swap p[i] with p[j],
     * j uniform in [0, i]. */
    for (int32_t i = n - 1; i >= 1; --i) {
      int32_t j = (int32_t)(next_uniform(&s) * (double)(i + 1));
      if (j > i) j = i;
      int32_t tmp = p[i];
      p[i] = p[j];
      p[j] = tmp;
    }
  }
  return AS_GEN_OK;
}
