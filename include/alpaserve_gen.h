/*
 * alpaserve_gen.h -- seeded synthetic workload generator (host library
 * libas_gen.so, plain C, no GPU code).
 *
 * The generator writes the inputs of the serving simulator: merged Gamma
 * arrival traces (the arrival model of Sec. 3.1, Sec. 3.2 and Sec. 6.2: a
 * Gamma process per model, parameterised by rate and coefficient of
 * variation, "CV") and keyed uniform draws for the problem builders.
 * It holds none of the simulator's arithmetic.
 *
 * Every pointer is a HOST pointer owned by the caller.  Functions return
 * AS_GEN_OK (0) or a negative AS_GEN_E_* code and never abort.
 * Determinism: outputs depend only on the arguments (and on the host libm's
 * log, sqrt and pow, which are used by the Gamma sampler).
 */
#ifndef ALPASERVE_GEN_H
#define ALPASERVE_GEN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AS_GEN_OK 0
#define AS_GEN_E_INVALID_ARG (-1)
#define AS_GEN_E_CAPACITY (-2) /* output buffer too small; *n_out holds the needed length */
#define AS_GEN_E_NOMEM (-3)

/* Purposes used to derive independent streams from one configuration seed. */
#define AS_GEN_PURPOSE_ARRIVAL 1u  /* per-model arrival gaps (index = model id)     */
#define AS_GEN_PURPOSE_LATENCY 2u  /* model single-device latencies                 */
#define AS_GEN_PURPOSE_WEIGHT 3u   /* model weight sizes                            */
#define AS_GEN_PURPOSE_PERMUTE 4u  /* placement permutations (index = candidate id) */
#define AS_GEN_PURPOSE_WINDOW 5u   /* windowed arrival gaps (index = m * n_windows + w) */
#define AS_GEN_PURPOSE_WPARAM 6u   /* window parameters of the problem builders      */

/* Stream key for (configuration seed, purpose, index).  Pure function. */
uint64_t as_gen_key(uint64_t seed, uint64_t purpose, uint64_t index);

/* n uniforms in (0, 1) from stream `key`, counters 0..n-1, into out[n]. */
int as_gen_uniforms(uint64_t key, int64_t n, double* out);

/* One Gamma(shape, scale 1) variate from stream `key` starting at `counter`;
 * the first unused counter is stored to *counter_out when it is not NULL.
 * shape must be > 0. */
double as_gen_gamma(uint64_t key, uint64_t counter, double shape, uint64_t* counter_out);

/* count permutations of 0..n-1, row r from stream as_gen_key(seed, purpose,
 * first_index + r), by Fisher-Yates with j = floor(u * (i + 1)).
 * out[count][n] (int32, host). */
int as_gen_permutations(uint64_t seed, uint64_t purpose, uint64_t first_index, int64_t count,
                        int32_t n, int32_t* out);

/*
 * Merged arrival trace of n_models independent Gamma renewal processes.
 *   seed      configuration seed; model m uses stream as_gen_key(seed, ARRIVAL, m)
 *   rate[m]   arrivals per second of model m (>= 0, finite; 0 = no arrivals)
 *   cv        coefficient of variation of the gaps (> 0; 1 = Poisson)
 *   duration  keep arrivals with t < duration (seconds, >= 0)
 *   capacity  length of t_out / m_out
 *   t_out[n]  arrival times in seconds, nondecreasing
 *   m_out[n]  model id of each arrival, in [0, n_models)
 *   *n_out    number of arrivals (always written on success and on
 *             AS_GEN_E_CAPACITY, so the caller can size a second call)
 * Order: ascending (t, model id, per-model arrival index).
 */
int as_gen_trace(uint64_t seed, int32_t n_models, const double* rate, double cv,
                 double duration, int64_t capacity, double* t_out, int32_t* m_out,
                 int64_t* n_out);

/*
 * Non-stationary trace: time is cut into n_windows windows of `window`
 * seconds, and in window w model m receives a Gamma renewal process with its
 * own rate and CV, restarted at the window's start (Sec. 6.1 fits the
 * arrivals of each time window of a production trace with a Gamma process
 * by rate and CV and resamples from the fitted processes; Sec. 6.4 evaluates
 * placements on a trace other than the one they were chosen for).
 *   seed        configuration seed; window w of model m uses stream
 *               as_gen_key(seed, WINDOW, m * n_windows + w)
 *   rate, cv    [n_models][n_windows] row-major (rate >= 0 finite, 0 = no
 *               arrivals; cv > 0 finite)
 *   window      window length in seconds (> 0, finite)
 * Arrivals of window w are w*window + X_1, + X_2, ... kept while
 * t < (w + 1)*window (both bounds are one fp64 product).  The per-model
 * arrival index runs across windows.  Outputs, order and capacity handling
 * as for as_gen_trace.
 */
int as_gen_trace_windowed(uint64_t seed, int32_t n_models, int32_t n_windows, double window,
                          const double* rate, const double* cv, int64_t capacity, double* t_out,
                          int32_t* m_out, int64_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* ALPASERVE_GEN_H */
