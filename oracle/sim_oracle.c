/*
 * ORACLE -- test infrastructure only.  Nothing in the product path may link,
 * load or call this file; only tests, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or constant generator with
 * the GPU simulator.
 *
 * A plain, slow, single-threaded CPU simulator of AlpaServe's serving model,
 * written from the paper's definitions:
 *   - Sec. 4.3 (runtime scheduling): a central controller sends each request
 *     to the group with the shortest queue among the groups that host the
 *     requested model; every group runs one first-come-first-served queue and
 *     rejects a request it cannot finish within the SLO, which is possible
 *     because execution times are predictable.
 *   - Sec. 3.2 (SLO experiment): requests that would miss the deadline even if
 *     scheduled immediately are dropped; SLO attainment is the fraction of all
 *     requests finished within the deadline; the deadline is a multiple
 *     ("SLO scale") of the model's single-device latency.
 *   - Sec. 3.4 (queueing analysis): a pipelined group is a chain of stages, each
 *     a single server; one request's latency is the sum of its stage latencies
 *     and the throughput is limited by the slowest stage.
 *   - Sec. 4.2 (placement): a placement partitions the devices into groups,
 *     each group has one shared parallel configuration (pipeline depth S,
 *     intra-op degree k) and hosts a subset of the models; a model may be
 *     replicated on several groups.
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - "shortest queue" is the group whose stage-0 free time (finish time at
 *     stage 0 of the last request it accepted; 0 before any) is smallest, ties
 *     to the lowest group index;
 *   - the SLO check happens when the request arrives: the projected finish
 *     f_{S-1} is accepted iff f_{S-1} <= t + slo (a finish exactly at the
 *     deadline is on time); a rejected request changes no state and is not
 *     retried on another group;
 *   - requests of a model that no group hosts are misses (they stay in the
 *     denominator of the attainment);
 *   - requests are handled in array order (the trace order breaks ties of
 *     equal arrival times); slo_m = slo_scale * d_single[m], one fp64 product.
 *
 * Per accepted request and stage s of the chosen group g (f_{-1} = t):
 *     f_s = max(f_{s-1}, F[g][s]) + L[m][c_g][s],   then F[g][s] := f_s.
 * All arithmetic is IEEE binary64, round to nearest even, no FMA
 * contraction (build with -ffp-contract=off), no reassociation.
 *
 * Verification digest (not part of the paper; it lets a checker compare two
 * simulators without the full per-request output): accept bits are packed 64
 * per word (bit i mod 64 of word i div 64), each finished word w folds into
 * h = (h XOR w) * 0x9E3779B97F4A7C15 mod 2^64 (the last partial word too), and
 * fin_sum is the sum mod 2^64 of the IEEE bit patterns of accepted finish
 * times.  Per-request output: finish time if accepted, -1 if rejected, -2 if
 * no group hosts the model.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_E_ARG (-1)
#define ORACLE_E_NOMEM (-2)

static double oracle_max(double a, double b) { return a < b ? b : a; }

static uint64_t bits_of(double x) {
  uint64_t u;
  memcpy(&u, &x, sizeof u);
  return u;
}

/*
 * Simulate one job: one trace, one placement, one SLO scale.
 *   t[n], model[n]          trace (seconds; model ids in [0, n_models))
 *   d_single[n_models]      single-device latency of each model (SLO base)
 *   cfg_stages[n_configs]   pipeline depth S of each parallel configuration
 *   stage_lat               [n_models][n_configs][max_stages] stage latencies
 *   group_cfg[n_groups]     configuration of each group (-1 = unused group)
 *   host_mask[n_models]     bit g set <=> group g hosts the model
 *   slo_scale               SLO multiple of d_single
 * Outputs: *served_out, digest_out[2] = {h, fin_sum}, finish_out[n] (may be NULL).
 */
/*
 * The same simulation with two more outputs, for the fast placement
 * heuristic of Sec. 4.2 (simulate once, then place the model with the most
 * unserved requests on the available group with the lowest utilization):
 *   model_served_out[n_models]  served requests of each model (may be NULL)
 *   group_busy_out[n_groups]    busy time of each group: for every request the
 *                               group serves, in trace order, the latency of
 *                               its slowest stage for that model (the stage
 *                               that bounds the group's throughput, Sec. 3.4)
 *                               is added to a running fp64 sum; 0 for groups
 *                               that serve nothing (may be NULL)
 */
int oracle_simulate_job_stats(int64_t n, const double* t, const int32_t* model, int32_t n_models,
                              const double* d_single, int32_t n_configs, const int32_t* cfg_stages,
                              int32_t max_stages, const double* stage_lat, int32_t n_groups,
                              const int32_t* group_cfg, const uint64_t* host_mask, double slo_scale,
                              int64_t* served_out, uint64_t* digest_out, double* finish_out,
                              int64_t* model_served_out, double* group_busy_out) {
  if (n < 0 || n_models <= 0 || n_configs <= 0 || max_stages <= 0 || n_groups <= 0 ||
      n_groups > 64 || !served_out || !digest_out)
    return ORACLE_E_ARG;

  double* F = (double*)calloc((size_t)n_groups * (size_t)max_stages, sizeof(double));
  double* slo = (double*)malloc((size_t)n_models * sizeof(double));
  double* f = (double*)malloc((size_t)max_stages * sizeof(double));
  if (!F || !slo || !f) {
    free(F);
    free(slo);
    free(f);
    return ORACLE_E_NOMEM;
  }
  /* inputs the definitions above do not cover are refused, not guessed */
  for (int32_t c = 0; c < n_configs; ++c)
    if (cfg_stages[c] < 1 || cfg_stages[c] > max_stages) goto bad_arg;
  for (int32_t m = 0; m < n_models; ++m)
    for (int32_t g = 0; g < 64; ++g)
      if ((host_mask[m] >> g) & 1u)
        if (g >= n_groups || group_cfg[g] < 0 || group_cfg[g] >= n_configs) goto bad_arg;
  for (int64_t i = 0; i < n; ++i)
    if (model[i] < 0 || model[i] >= n_models) goto bad_arg;

  for (int32_t m = 0; m < n_models; ++m) slo[m] = slo_scale * d_single[m];
  if (model_served_out)
    for (int32_t m = 0; m < n_models; ++m) model_served_out[m] = 0;
  if (group_busy_out)
    for (int32_t g = 0; g < n_groups; ++g) group_busy_out[g] = 0.0;

  int64_t served = 0;
  uint64_t h = 0, word = 0, fin_sum = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int32_t m = model[i];
    const double ti = t[i];
    const uint64_t mask = host_mask[m];
    double out;
    if (mask == 0) {
      out = -2.0;
    } else {
      /* dispatch: least stage-0 free time among hosting groups, lowest index on ties */
      int32_t gs = -1;
      for (int32_t g = 0; g < n_groups; ++g) {
        if (!((mask >> g) & 1u)) continue;
        if (gs < 0 || F[g * max_stages + 0] < F[gs * max_stages + 0]) gs = g;
      }
      const int32_t c = group_cfg[gs];
      const int32_t S = cfg_stages[c];
      /* projection through the stage chain */
      double prev = ti;
      for (int32_t s = 0; s < S; ++s) {
        const double lat = stage_lat[((int64_t)m * n_configs + c) * max_stages + s];
        f[s] = oracle_max(prev, F[gs * max_stages + s]) + lat;
        prev = f[s];
      }
      /* admission */
      const double deadline = ti + slo[m];
      if (prev > deadline) {
        out = -1.0;
      } else {
        for (int32_t s = 0; s < S; ++s) F[gs * max_stages + s] = f[s];
        if (model_served_out) model_served_out[m] += 1;
        if (group_busy_out) {
          double slowest = 0.0;
          for (int32_t s = 0; s < S; ++s)
            slowest = oracle_max(slowest, stage_lat[((int64_t)m * n_configs + c) * max_stages + s]);
          group_busy_out[gs] += slowest;
        }
        served += 1;
        fin_sum += bits_of(prev);
        word |= (uint64_t)1 << (i & 63);
        out = prev;
      }
    }
    if (finish_out) finish_out[i] = out;
    if ((i & 63) == 63 || i == n - 1) {
      h = (h ^ word) * 0x9E3779B97F4A7C15ULL;
      word = 0;
    }
  }
  *served_out = served;
  digest_out[0] = h;
  digest_out[1] = fin_sum;
  free(F);
  free(slo);
  free(f);
  return ORACLE_OK;

bad_arg:
  free(F);
  free(slo);
  free(f);
  return ORACLE_E_ARG;
}

int oracle_simulate_job(int64_t n, const double* t, const int32_t* model, int32_t n_models,
                        const double* d_single, int32_t n_configs, const int32_t* cfg_stages,
                        int32_t max_stages, const double* stage_lat, int32_t n_groups,
                        const int32_t* group_cfg, const uint64_t* host_mask, double slo_scale,
                        int64_t* served_out, uint64_t* digest_out, double* finish_out) {
  return oracle_simulate_job_stats(n, t, model, n_models, d_single, n_configs, cfg_stages, max_stages,
                                   stage_lat, n_groups, group_cfg, host_mask, slo_scale, served_out,
                                   digest_out, finish_out, NULL, NULL);
}

/*
 * Dynamic batching (Sec. 6.5).  The paper's batching strategy: a request
 * that arrives while a device group hosting its model is available runs at
 * once; otherwise it waits in a per-model queue; a group that becomes idle
 * picks a model it hosts and runs as many of that model's queued requests
 * as possible in one batch while the SLO holds.  A batch's execution latency
 * grows linearly with its size.
 *
 * Readings (each one also stated in the design notes):
 *   - a group is available, and becomes idle, when its stage 0 is free: at
 *     time x it is available iff F[g][0] <= x; among available hosting
 *     groups the one with the smallest F[g][0] runs an arriving request
 *     (lowest index on ties);
 *   - stage latencies of a batch of b requests of model m on configuration c:
 *     L[m][c][s] * (1 + beta * (b - 1)), the factor rounded once, then the
 *     product (beta >= 0; beta = 1: no throughput gain from batching);
 *   - a batch starting at x runs through the group's stages like one request:
 *     f_{-1} = x, f_s = max(f_{s-1}, F[g][s]) + lat_s; every request of the
 *     batch finishes at f_{S-1}; F[g][s] := f_s;
 *   - an arriving request that runs at once is served iff its finish is
 *     within its deadline t + slo_m; otherwise it is dropped;
 *   - a group becomes idle at tau = F[g][0]; if a model it hosts has queued
 *     requests it starts a batch at tau: the model whose queue head arrived
 *     first (lowest trace index); the batch takes the largest b <=
 *     min(max_batch, queue length) whose finish is within the head's deadline
 *     (the tightest of the model's queue, which is FIFO); if even b = 1 misses
 *     it, the head is dropped and the choice is made again; with no queued
 *     work the group stays idle;
 *   - before an arrival at t, every idle event at tau <= t is handled, in
 *     order of tau, lowest group first on ties; after the last arrival the
 *     remaining idle events are handled until no queued work remains.
 * Outputs as for the unbatched simulation, except the digest, which cannot
 * fold accept words in trace order because queued requests are decided
 * later: h = sum mod 2^64 over served requests i of mix(i), where mix is the
 * SplitMix64 finaliser of i; fin_sum as before.  batch_out[i] (may be NULL):
 * size of the batch request i ran in, 0 if not served.
 */
static uint64_t oracle_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

typedef struct {
  int64_t* idx; /* queued trace indices, FIFO from head */
  int64_t head, tail, cap;
} oracle_queue;

static int oracle_queue_push(oracle_queue* q, int64_t i) {
  if (q->tail == q->cap) {
    int64_t cap = q->cap ? 2 * q->cap : 16;
    int64_t* p = (int64_t*)realloc(q->idx, (size_t)cap * sizeof(int64_t));
    if (!p) return ORACLE_E_NOMEM;
    q->idx = p;
    q->cap = cap;
  }
  q->idx[q->tail++] = i;
  return ORACLE_OK;
}

int oracle_simulate_job_batched(int64_t n, const double* t, const int32_t* model, int32_t n_models,
                                const double* d_single, int32_t n_configs, const int32_t* cfg_stages,
                                int32_t max_stages, const double* stage_lat, int32_t n_groups,
                                const int32_t* group_cfg, const uint64_t* host_mask, double slo_scale,
                                int32_t max_batch, double beta, int64_t* served_out, uint64_t* digest_out,
                                double* finish_out, int32_t* batch_out) {
  if (n < 0 || n_models <= 0 || n_configs <= 0 || max_stages <= 0 || n_groups <= 0 || n_groups > 64 ||
      max_batch < 1 || !(beta >= 0.0) || !served_out || !digest_out)
    return ORACLE_E_ARG;
  for (int32_t c = 0; c < n_configs; ++c)
    if (cfg_stages[c] < 1 || cfg_stages[c] > max_stages) return ORACLE_E_ARG;
  for (int32_t m = 0; m < n_models; ++m)
    for (int32_t g = 0; g < 64; ++g)
      if ((host_mask[m] >> g) & 1u)
        if (g >= n_groups || group_cfg[g] < 0 || group_cfg[g] >= n_configs) return ORACLE_E_ARG;
  for (int64_t i = 0; i < n; ++i)
    if (model[i] < 0 || model[i] >= n_models) return ORACLE_E_ARG;

  double* F = (double*)calloc((size_t)n_groups * (size_t)max_stages, sizeof(double));
  double* slo = (double*)malloc((size_t)n_models * sizeof(double));
  double* f = (double*)malloc((size_t)max_stages * sizeof(double));
  oracle_queue* q = (oracle_queue*)calloc((size_t)n_models, sizeof(oracle_queue));
  int rc = ORACLE_OK;
  if (!F || !slo || !f || !q) {
    rc = ORACLE_E_NOMEM;
    goto done;
  }
  for (int32_t m = 0; m < n_models; ++m) slo[m] = slo_scale * d_single[m];
  int64_t served = 0;
  uint64_t h = 0, fin_sum = 0;
  if (finish_out)
    for (int64_t i = 0; i < n; ++i) finish_out[i] = (host_mask[model[i]] == 0) ? -2.0 : -1.0;
  if (batch_out)
    for (int64_t i = 0; i < n; ++i) batch_out[i] = 0;

/* finish of a batch of b requests of model m started at x on group g, into f[] */
#define ORACLE_BATCH_FINISH(g, m, b, x)                                                   \
  do {                                                                                    \
    const int32_t c_ = group_cfg[g];                                                      \
    const double fac_ = 1.0 + beta * (double)((b) - 1);                                  \
    double prev_ = (x);                                                                   \
    for (int32_t s_ = 0; s_ < cfg_stages[c_]; ++s_) {                                     \
      const double lat_ = stage_lat[((int64_t)(m) * n_configs + c_) * max_stages + s_] * fac_; \
      f[s_] = oracle_max(prev_, F[(g) * max_stages + s_]) + lat_;                         \
      prev_ = f[s_];                                                                      \
    }                                                                                     \
  } while (0)

  for (int64_t i = 0; i <= n; ++i) {
    /* idle events up to the next arrival (all of them after the last one) */
    const double horizon = i < n ? t[i] : 0.0;
    for (;;) {
      int32_t gs = -1;
      for (int32_t g = 0; g < n_groups; ++g) {
        if (group_cfg[g] < 0) continue;
        int work = 0;
        for (int32_t m = 0; m < n_models && !work; ++m)
          work = ((host_mask[m] >> g) & 1u) && q[m].head < q[m].tail;
        if (!work) continue;
        if (gs < 0 || F[g * max_stages] < F[gs * max_stages]) gs = g;
      }
      if (gs < 0) break;
      const double tau = F[gs * max_stages];
      if (i < n && !(tau <= horizon)) break;
      /* the group starts a batch at tau, or drops expired heads until it can */
      for (;;) {
        int32_t mc = -1;
        for (int32_t m = 0; m < n_models; ++m)
          if (((host_mask[m] >> gs) & 1u) && q[m].head < q[m].tail &&
              (mc < 0 || q[m].idx[q[m].head] < q[mc].idx[q[mc].head]))
            mc = m;
        if (mc < 0) break; /* nothing left for this group: it stays idle */
        const int64_t hd = q[mc].idx[q[mc].head];
        const double dl = t[hd] + slo[mc];
        const int64_t avail = q[mc].tail - q[mc].head;
        const int32_t bmax = avail < max_batch ? (int32_t)avail : max_batch;
        int32_t b = 0;
        for (int32_t bb = 1; bb <= bmax; ++bb) {
          ORACLE_BATCH_FINISH(gs, mc, bb, tau);
          if (f[cfg_stages[group_cfg[gs]] - 1] > dl) break;
          b = bb;
        }
        if (b == 0) {
          q[mc].head += 1; /* the head cannot meet its deadline: dropped */
          continue;
        }
        ORACLE_BATCH_FINISH(gs, mc, b, tau);
        const int32_t S = cfg_stages[group_cfg[gs]];
        for (int32_t s = 0; s < S; ++s) F[gs * max_stages + s] = f[s];
        const double fin = f[S - 1];
        for (int32_t k = 0; k < b; ++k) {
          const int64_t r = q[mc].idx[q[mc].head + k];
          served += 1;
          h += oracle_mix64((uint64_t)r);
          fin_sum += bits_of(fin);
          if (finish_out) finish_out[r] = fin;
          if (batch_out) batch_out[r] = b;
        }
        q[mc].head += b;
        break;
      }
    }
    if (i == n) break;
    /* the arrival */
    const int32_t m = model[i];
    const uint64_t mask = host_mask[m];
    if (mask == 0) continue;
    int32_t ga = -1;
    for (int32_t g = 0; g < n_groups; ++g)
      if (((mask >> g) & 1u) && F[g * max_stages] <= t[i] && (ga < 0 || F[g * max_stages] < F[ga * max_stages]))
        ga = g;
    if (ga >= 0) {
      ORACLE_BATCH_FINISH(ga, m, 1, t[i]);
      const int32_t S = cfg_stages[group_cfg[ga]];
      if (!(f[S - 1] > t[i] + slo[m])) {
        for (int32_t s = 0; s < S; ++s) F[ga * max_stages + s] = f[s];
        served += 1;
        h += oracle_mix64((uint64_t)i);
        fin_sum += bits_of(f[S - 1]);
        if (finish_out) finish_out[i] = f[S - 1];
        if (batch_out) batch_out[i] = 1;
      }
    } else if ((rc = oracle_queue_push(&q[m], i)) != ORACLE_OK) {
      goto done;
    }
  }
#undef ORACLE_BATCH_FINISH
  *served_out = served;
  digest_out[0] = h;
  digest_out[1] = fin_sum;
done:
  if (q)
    for (int32_t m = 0; m < n_models; ++m) free(q[m].idx);
  free(q);
  free(F);
  free(slo);
  free(f);
  return rc;
}
