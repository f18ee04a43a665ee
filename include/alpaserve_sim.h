/*
 * alpaserve_sim.h -- C-ABI of libalpaserve_sim.so, the batched serving
 * simulator for AlpaServe-style placement search on AMD MI355X (gfx950).
 *
 * What is computed (AlpaServe, Sec. 4.3, Sec. 3.2, Sec. 3.4, Sec. 4.2):
 * one "job" is a (trace, placement, SLO scale) triple.  A placement splits the
 * devices into groups; group g has one parallel configuration c_g with S pipeline
 * stages and hosts a subset of the models (a model may be hosted by several
 * groups).  Requests are processed in trace order.  A request for model m at
 * time t goes to the hosting group with the smallest stage-0 free time (ties to
 * the lowest group index); its projected finish is
 *     f_{-1} = t,  f_s = max(f_{s-1}, F[g][s]) + L[m][c_g][s]   (s = 0..S-1)
 * where F[g][s] is the finish time at stage s of the last request the group
 * accepted (0 initially).  It is served iff f_{S-1} <= t + scale * d_single[m]
 * (the product rounded once); then F[g][s] := f_s.  Otherwise it is rejected
 * and nothing changes (no retry on another group).  A request for a model no
 * group hosts is a miss.  All arithmetic is IEEE binary64, round to nearest,
 * no fused multiply-add, in exactly this order, so results are reproducible
 * bit for bit on any conforming implementation.
 *
 * Outputs per job: served = number of served requests; attain = served / n
 * (0 when n = 0); digest[2] = {h, fin_sum}: accept bits packed 64 per word (bit
 * i mod 64 of word i div 64, the last word possibly partial), each word w folded
 * as h = (h XOR w) * 0x9E3779B97F4A7C15 mod 2^64 starting from h = 0, and
 * fin_sum = sum mod 2^64 of the IEEE-754 bit patterns of served finish times.
 * Optional per-request output for selected jobs: the finish time of a served
 * request, -1.0 for a rejected one, -2.0 for a miss.
 *
 * Conventions shared by every entry point:
 *   - Pointers are DEVICE pointers unless marked HOST.  The caller owns every
 *     buffer; outputs are caller-allocated and fully written.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream); outputs are valid after the stream synchronises.
 *   - Return 0 (AS_OK) or a negative AS_E_* code; as_last_error() then holds a
 *     message.  Nothing aborts and no C++ exception crosses this boundary.
 *   - Scalar arguments and HOST arrays are always checked.  Device data are not
 *     read by the checks; call as_validate() (synchronous) to check them.
 *     Invalid device data give unspecified results but never an access outside
 *     the buffers described here.
 */
#ifndef ALPASERVE_SIM_H
#define ALPASERVE_SIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AS_OK 0
#define AS_E_INVALID_ARG (-1) /* null pointer, negative size, bad host array    */
#define AS_E_LIMITS (-2)      /* a size beyond the limits below                  */
#define AS_E_HIP (-3)         /* a HIP runtime call or kernel launch failed      */
#define AS_E_NOMEM (-4)       /* device allocation failed                        */
#define AS_E_INVALID_DATA (-5) /* as_validate found a device-data precondition broken */

#define AS_MAX_MODELS 64   /* M: per-group hosted-model bitmaps are 64 bits wide */
#define AS_MAX_GROUPS 64   /* G: host_mask rows are 64-bit group bitmaps         */
#define AS_MAX_STAGES 8    /* S per configuration                                */
#define AS_MAX_CONFIGS 32  /* C                                                  */
#define AS_MAX_FINISH 256  /* jobs with per-request output per call              */

/* One arrival trace. */
typedef struct {
  int64_t n;            /* number of requests, >= 0                                 */
  const double* t;      /* [n] arrival times in seconds: finite, >= 0, nondecreasing */
  const int32_t* model; /* [n] model ids in [0, n_models)                          */
} as_trace_t;

/* Models and parallel configurations (Sec. 4.1 produces per-configuration
 * stage latencies; here they are inputs). */
typedef struct {
  int32_t n_models;          /* M, 1..AS_MAX_MODELS                               */
  int32_t n_configs;         /* C, 1..AS_MAX_CONFIGS                              */
  int32_t max_stages;        /* row length of stage_lat, >= every cfg_stages[c]   */
  const double* d_single;    /* [M] single-device latency, the SLO base: finite, > 0 */
  const int32_t* cfg_stages; /* HOST [C] pipeline depth S_c, 1..AS_MAX_STAGES     */
  const double* stage_lat;   /* [M][C][max_stages] stage latencies in seconds:
                                finite, >= 0; entries s >= S_c are ignored        */
} as_models_t;

/* Candidate placements (Sec. 4.2: group partition + model selection + config). */
typedef struct {
  int32_t n_placements;      /* P, >= 0                                           */
  int32_t max_groups;        /* G, 1..AS_MAX_GROUPS                               */
  const int32_t* group_cfg;  /* [P][G] configuration of group g, -1 = no group    */
  const uint64_t* host_mask; /* [P][M] bit g set <=> group g hosts model m; only
                                groups with group_cfg >= 0 may be set            */
} as_placements_t;

/*
 * Score every placement at every SLO scale over one shared trace
 * (Alg. 1's simulate(sel, W) call, batched; Sec. 4.2).
 *   slo_scale[K]     SLO multiples of d_single: >= 0 (+inf allowed, NaN not)
 *   jobs             J = P * K, job j = p * K + k (row-major [P][K])
 *   out_served[J]    served counts
 *   out_attain[J]    served / n, or NULL
 *   out_digest[J][2] {h, fin_sum}, or NULL
 *   finish_jobs      HOST [n_finish] distinct job ids in [0, J), or NULL
 *   out_finish       [n_finish][trace->n] per-request outputs of those jobs
 * Each job's state lives in one wavefront: lanes hold the groups of a job
 * (several jobs per wavefront when the group count allows), arrivals are
 * staged through LDS in chunks shared by the workgroup.
 */
int as_simulate_placements(const as_trace_t* trace, const as_models_t* models,
                           const as_placements_t* placements, const double* slo_scale,
                           int32_t n_scales, int64_t* out_served, double* out_attain,
                           uint64_t* out_digest, const int32_t* finish_jobs, int32_t n_finish,
                           double* out_finish, void* stream);

/* Bytes of device memory that as_simulate_placements_noalloc may use. */
#define AS_NOALLOC_SCRATCH_BYTES (256u << 20)

/*
 * as_simulate_placements for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid
 * allocation): the same arguments, kernels and results, bit for bit, but no
 * hipMalloc, hipFree or other allocating call is made.  Where the speculative
 * kernels take the call (long traces), their workspace (accept bits and saved
 * states, about 0.19 bytes per request x job) comes from an array of
 * AS_NOALLOC_SCRATCH_BYTES in device memory that the library holds on every
 * device it runs on until the process ends; a call whose workspace would be
 * larger returns AS_E_LIMITS without launching anything (as_simulate_placements
 * takes such calls).  Every call on one device shares that device's array, and
 * the array keeps the last call's contents (each call initialises what it
 * reads), so calls that overlap on one device -- on different streams, or
 * from different threads without ordering -- race and give unspecified
 * results; calls ordered on one stream do not.
 */
int as_simulate_placements_noalloc(const as_trace_t* trace, const as_models_t* models,
                                   const as_placements_t* placements, const double* slo_scale,
                                   int32_t n_scales, int64_t* out_served, double* out_attain,
                                   uint64_t* out_digest, const int32_t* finish_jobs, int32_t n_finish,
                                   double* out_finish, void* stream);

/* A job of the segmented variant. */
typedef struct {
  int32_t placement; /* index into the placements                       */
  int32_t segment;   /* trace segment, index into seg_offsets           */
  double slo_scale;  /* SLO multiple: >= 0, +inf allowed                */
} as_job_t;

/*
 * Jobs that each bring their own trace segment: the same simulation (Sec.
 * 4.3, Sec. 3.2, Sec. 3.4) per job, for the SLO-attainment curves of Sec. 3.2
 * and Sec. 6 that vary the SLO scale, the rate and the burstiness (CV) of the
 * workload for one placement, each grid point with its own generated
 * workload.  Segment s is requests
 * [seg_offsets[s], seg_offsets[s+1]) of t/model, each segment nondecreasing in
 * t on its own.
 *   t, model         concatenated segments (device)
 *   seg_offsets      [n_segments + 1], nondecreasing, seg_offsets[0] = 0 (device)
 *   jobs             [n_jobs] (device)
 *   out_*            as above, indexed by job; attain = served / segment length
 *   out_finish       [n_finish][finish_stride]; row f receives job
 *                    finish_jobs[f]'s outputs for requests i < min(segment
 *                    length, finish_stride)
 * Asynchronous on `stream`.  With more than 32 groups (one job per
 * wavefront at a time) and 2..4096 jobs, the jobs are sorted by segment
 * length on the device: up to two wavefronts per SIMD they run one per
 * wavefront, longest and shortest segment alternating; beyond, two
 * wavefronts per SIMD take them in turn, longest first, from a counter.
 * Neither changes any result.  The order array and the counter (4 bytes per
 * job, plus 4) come from the library's memory pool and are released
 * stream-ordered.
 */
int as_simulate_jobs(const double* t, const int32_t* model, const int64_t* seg_offsets,
                     int32_t n_segments, const as_models_t* models,
                     const as_placements_t* placements, const as_job_t* jobs, int32_t n_jobs,
                     int64_t* out_served, double* out_attain, uint64_t* out_digest,
                     const int32_t* finish_jobs, int32_t n_finish, double* out_finish,
                     int64_t finish_stride, void* stream);

/*
 * Check the device-data preconditions of as_simulate_placements (trace
 * sorted, finite and >= 0; model ids in range; group configurations in
 * [-1, C); host_mask bits only on existing groups; latencies finite and >= 0;
 * d_single finite and > 0; scales >= 0 and not NaN).  Synchronous: returns
 * AS_OK, AS_E_INVALID_DATA with a message naming the first failed check, or
 * another AS_E_* code.  Allocates a few bytes of device memory per call.
 */
int as_validate(const as_trace_t* trace, const as_models_t* models,
                const as_placements_t* placements, const double* slo_scale, int32_t n_scales,
                void* stream);

/*
 * Alg. 1 of the paper (simulator-guided greedy model selection, Sec. 4.2)
 * with beam size 1 on one group partition.  Starting from the empty selection,
 * every step scores each feasible addition -- a (model m, group g) pair with g
 * not yet hosting m whose weight still fits in g's memory -- by simulating the
 * selection plus that replica over the trace (one batched launch per step),
 * commits the candidate with the most served requests (lowest candidate index
 * in (m, g) order on ties), and repeats until no addition fits.  The result is
 * the best selection seen (replaced only by a strictly better one; the empty
 * selection serves 0).
 *   trace, models     device data as for as_simulate_placements
 *   weight_mib        HOST [M] model weights (integer MiB, >= 0)
 *   n_groups          G, 1..AS_MAX_GROUPS
 *   group_cfg         HOST [G] configuration of each group (-1 = no group)
 *   group_mem_mib     HOST [G] memory of each group (sum of its devices', MiB):
 *                     a selection fits iff every group's hosted weights sum to
 *                     at most its memory (each device of a group stores 1/(S*k)
 *                     of every hosted model)
 *   slo_scale         one SLO multiple for every model (>= 0, +inf allowed)
 *   best_mask         HOST out [M] bit g set <=> group g hosts model m
 *   best_served       HOST out served requests of best_mask
 *   step_model/_group/_served  HOST out [max_steps] trajectory (may be NULL
 *                     when max_steps = 0); *n_steps = steps taken (steps beyond
 *                     max_steps are taken but not recorded)
 * Synchronous on `stream`; allocates device memory for the candidate batch.
 */
int as_greedy_placement(const as_trace_t* trace, const as_models_t* models,
                        const int64_t* weight_mib, int32_t n_groups, const int32_t* group_cfg,
                        const int64_t* group_mem_mib, double slo_scale, uint64_t* best_mask,
                        int64_t* best_served, int32_t* step_model, int32_t* step_group,
                        int64_t* step_served, int32_t max_steps, int32_t* n_steps,
                        void* stream);

/*
 * Alg. 1 with beam size `beam` >= 1 (Sec. 4.2): every step expands each
 * selection of the beam, in beam order, by every feasible (m, g) addition in
 * (m, g) order, drops a new selection equal to one produced earlier in the
 * same step, scores all of them in one batched launch, keeps the `beam` most
 * served (the earlier candidate first on ties) as the next beam and compares
 * the best of them with the best selection so far (replaced only by a
 * strictly better one).  Arguments as for as_greedy_placement (beam = 1 is
 * as_greedy_placement); step i records the best selection of step i: the
 * replica (step_model, step_group) that its parent gained and its served
 * count.
 */
int as_beam_placement(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                      int32_t n_groups, const int32_t* group_cfg, const int64_t* group_mem_mib,
                      double slo_scale, int32_t beam, uint64_t* best_mask, int64_t* best_served,
                      int32_t* step_model, int32_t* step_group, int64_t* step_served, int32_t max_steps,
                      int32_t* n_steps, void* stream);

/*
 * The fast heuristic of Sec. 4.2 for very large workloads: simulate the
 * current selection once (as_simulate_stats), then add the model with the
 * most unserved requests (its requests in the trace minus the served ones;
 * among models that still fit on some group; lowest id on ties) to the
 * available group with the lowest utilization (least busy time; among the
 * groups where the replica fits; lowest index on ties); repeat until no
 * replica fits.  Every simulated selection, the last one included, competes
 * for the result (replaced only by a strictly better one).  Arguments as for
 * as_greedy_placement; step i records the replica added and the served count
 * of the selection it was added to.
 */
int as_fast_placement(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                      int32_t n_groups, const int32_t* group_cfg, const int64_t* group_mem_mib,
                      double slo_scale, uint64_t* best_mask, int64_t* best_served, int32_t* step_model,
                      int32_t* step_group, int64_t* step_served, int32_t max_steps, int32_t* n_steps,
                      void* stream);

/*
 * Reduced Alg. 2 (Sec. 4.2): run as_greedy_placement on each of n_partitions
 * partitions and keep the strictly best (first on ties).  The partitions'
 * searches advance in lockstep: one launch per step scores the candidates of
 * all of them.  Partition p has
 * part_groups[p] groups whose configurations and memories are
 * part_cfg[off_p ..] and part_mem_mib[off_p ..], off_p = sum of earlier
 * part_groups (HOST arrays).  Outputs: *best_partition, best_mask[M] (HOST),
 * *best_served, part_served[n_partitions] (HOST, each partition's best).
 */
int as_partition_search(const as_trace_t* trace, const as_models_t* models,
                        const int64_t* weight_mib, int32_t n_partitions, const int32_t* part_groups,
                        const int32_t* part_cfg, const int64_t* part_mem_mib, double slo_scale,
                        int32_t* best_partition, uint64_t* best_mask, int64_t* best_served,
                        int64_t* part_served, void* stream);

/*
 * The simulation of as_simulate_placements with the statistics that the fast
 * placement heuristic of Sec. 4.2 reads after simulating a selection once
 * (place the model with the most unserved requests on the available group
 * with the lowest utilization).  Jobs and scales as for
 * as_simulate_placements (job j = p * K + k); every pointer is a device
 * pointer.
 *   out_served[J]             served counts (required)
 *   out_digest[J][2]          {h, fin_sum} as above, or NULL
 *   out_model_served[J][M]    served requests of each model, or NULL
 *   out_group_busy[J][G]      busy time of each group, or NULL: for every
 *                             request group g serves, in trace order, the
 *                             largest stage latency of that model in g's
 *                             configuration (the stage that bounds the
 *                             group's throughput, Sec. 3.4) is added to an
 *                             fp64 sum starting at 0
 * With one scale the jobs run on the shared-trace kernel (lanes = groups,
 * several jobs per wavefront); with several, one job per wavefront.  The
 * stage-latency table must fit in the LDS of a workgroup (AS_E_LIMITS
 * otherwise).
 */
int as_simulate_stats(const as_trace_t* trace, const as_models_t* models,
                      const as_placements_t* placements, const double* slo_scale, int32_t n_scales,
                      int64_t* out_served, uint64_t* out_digest, int64_t* out_model_served,
                      double* out_group_busy, void* stream);

/*
 * Dynamic batching (Sec. 6.5).  The same jobs as as_simulate_placements (job
 * j = p * K + k), simulated with the paper's batching strategy: a request
 * that arrives while a group hosting its model is available runs at once,
 * otherwise it waits in a per-model queue; a group that becomes idle picks a
 * model it hosts and runs as many of its queued requests as possible in one
 * batch while the SLO holds.  Exact rules:
 *   - a group is available, and becomes idle, when its stage 0 is free: at
 *     time x iff F[g][0] <= x.  An arriving request (time t, model m) runs on
 *     the available hosting group with the smallest F[g][0] (lowest index on
 *     ties) as a batch of one starting at t, and is served iff its finish is
 *     <= t + scale * d_single[m]; otherwise it is dropped.  With no available
 *     hosting group it joins the tail of m's queue;
 *   - a batch of b requests of model m on group g with configuration c
 *     starting at x: stage latencies lat_s = L[m][c][s] * (1 + beta*(b-1))
 *     (the factor rounded once, then the product), f_{-1} = x, f_s =
 *     max(f_{s-1}, F[g][s]) + lat_s; all b requests finish at f_{S-1}, and
 *     F[g][s] := f_s;
 *   - a group becomes idle at tau = F[g][0].  If models it hosts have queued
 *     requests it starts a batch at tau: of the model whose queue head has
 *     the lowest trace index, the largest b <= min(max_batch, queue length)
 *     whose finish is <= the head's deadline (the tightest in that FIFO
 *     queue).  If b = 1 misses it, the head is dropped and the choice is made
 *     again.  With no queued work the group stays idle;
 *   - before each arrival at t every idle event at tau <= t is handled, in
 *     order of tau, lowest group first on ties; after the last arrival the
 *     remaining ones are handled until no queued work remains.
 *   beta            latency slope, finite, >= 0 (1: a batch of b takes b times
 *                   as long as one request, as for GPUs a small batch saturates)
 *   max_batch       >= 1
 *   queue_cap       the longest queue a model may reach in a job, a power of
 *                   two in 1..2^20; if a queue would grow past it the call
 *                   returns AS_E_LIMITS and its results are incomplete (the
 *                   queues take no memory of their own: a queue is always a
 *                   run of its model's arrivals, kept as two positions in a
 *                   per-model arrival list the call builds once for all jobs).
 *                   The stage-latency table must fit in a workgroup's LDS
 *                   (M * pow2ceil(C) * Smax * 8 bytes), else AS_E_LIMITS
 *   out_served[J]   served counts
 *   out_digest[J][2] {h, fin_sum} or NULL, where h = sum mod 2^64 over served
 *                   requests i of mix(i), mix the SplitMix64 finaliser
 *                   (queued requests are decided out of trace order, so the
 *                   accept-word fold of the other entry points does not apply)
 *   finish_jobs, n_finish, out_finish as for as_simulate_placements (finish
 *                   time of a served request, -1 dropped, -2 no hosting group)
 * Synchronous on `stream` (it reads back a flags word); allocates about
 * 24 bytes of device memory per request of the trace per call (the arrival
 * lists) and frees it before returning.  AS_E_INVALID_DATA if a queue is ever
 * found not to be such a run (the rules rule it out; the check guards the
 * results).  One job per wavefront: lanes = groups for the free times,
 * lanes = models for the queues.
 */
int as_simulate_batched(const as_trace_t* trace, const as_models_t* models,
                        const as_placements_t* placements, const double* slo_scale, int32_t n_scales,
                        int32_t max_batch, double beta, int32_t queue_cap, int64_t* out_served,
                        uint64_t* out_digest, const int32_t* finish_jobs, int32_t n_finish,
                        double* out_finish, void* stream);

#define AS_MAX_BUCKETS 8 /* model buckets of one placement (Alg. 2) */

/* Options of as_placement_search (Alg. 2).  HOST struct. */
typedef struct {
  int32_t n_devices;          /* devices of the cluster, a multiple of device_unit        */
  int32_t device_unit;        /* device counts of buckets are multiples of this, >= 1     */
  int64_t device_mem_mib;     /* memory of one device (MiB), >= 0                         */
  const int32_t* cfg_devices; /* HOST [C] devices of a group of configuration c (S_c*k_c) */
  double bucket_threshold;    /* largest latency span (s) inside a model bucket, >= 0     */
  double balance_ratio;       /* largest max/min ratio of bucket loads kept, >= 1 (+inf:
                                 keep every split)                                         */
  double slo_scale;           /* SLO multiple of d_single for every model, >= 0           */
  int32_t max_buckets;        /* 1..AS_MAX_BUCKETS                                        */
  int32_t beam;               /* Alg. 1 beam size (>= 1), or 0 for the fast heuristic     */
} as_search_opts_t;

/* Result of as_placement_search.  HOST struct, written by the call.  Bucket b
 * has bucket_groups[b] groups with configurations bucket_group_cfg[b][0..],
 * each holding (number of its devices) x device_mem_mib MiB; bit g of
 * bucket_mask[b][m] is set iff its group g hosts model m. */
typedef struct {
  int64_t served;                 /* requests the placement serves (sum over buckets)  */
  int32_t n_buckets;              /* 0 when no placement serves anything               */
  int32_t n_bucket_configs;       /* model-bucket cuts enumerated                      */
  int32_t n_device_splits;        /* device splits enumerated                          */
  int32_t n_kept_splits;          /* splits kept by the balance rule                   */
  int32_t n_problems;             /* Alg. 1 problems solved (bucket x devices x config) */
  int64_t launches;               /* batched simulator launches of the search          */
  int64_t jobs_simulated;         /* simulations run (each over the whole trace)       */
  int32_t model_bucket[AS_MAX_MODELS];                 /* bucket of each model       */
  int32_t bucket_devices[AS_MAX_BUCKETS];              /* devices of each bucket     */
  int32_t bucket_cfg[AS_MAX_BUCKETS];                  /* configuration of its equal
                                                          groups; -1 if it serves nothing */
  int32_t bucket_groups[AS_MAX_BUCKETS];
  int32_t bucket_group_cfg[AS_MAX_BUCKETS][AS_MAX_GROUPS];
  int64_t bucket_served[AS_MAX_BUCKETS];
  uint64_t bucket_mask[AS_MAX_BUCKETS][AS_MAX_MODELS];
} as_search_result_t;

/*
 * Alg. 2 of Sec. 4.2: enumerate model buckets, device buckets, group
 * partitions and parallel configurations, run Alg. 1 (beam >= 1) or the fast
 * heuristic (beam = 0) for every bucket option, keep each bucket's strictly
 * best option and the strictly best concatenation (first on ties; the empty
 * placement serves 0).
 *   model buckets   models sorted by d_single (ties by id) cut into 1..
 *                   max_buckets contiguous runs, each spanning at most
 *                   bucket_threshold seconds (every such cut is tried)
 *   device buckets  every split of n_devices into the buckets in multiples
 *                   of device_unit (lexicographic), dropped when the largest
 *                   bucket load exceeds balance_ratio times the smallest; a
 *                   bucket's load is the sum over its models of (requests in
 *                   the trace x d_single) per device
 *   partitions      per bucket and configuration c with cfg_devices[c] <=
 *                   the bucket's devices: equal groups of configuration c and
 *                   one last group with the remaining devices, whose
 *                   configuration is the one of that device count with the
 *                   deepest pipeline not deeper than c's (lowest index on
 *                   ties; c is skipped if none exists or if the bucket would
 *                   have more than AS_MAX_GROUPS groups)
 *   selection       Alg. 1 places only the bucket's models, over the whole
 *                   trace (other models' requests are never served there)
 * trace, models, weight_mib as for as_greedy_placement.  Every Alg. 1 problem
 * is solved once and all of them advance in lockstep (one launch per step).
 * Synchronous on `stream`; allocates device memory for the candidate batches.
 */
int as_placement_search(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                        const as_search_opts_t* opts, as_search_result_t* result, void* stream);

/* Message of the last failed call on this thread ("" if none); valid until
 * the next call on this thread. */
const char* as_last_error(void);

/* Library version string. */
const char* as_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ALPASERVE_SIM_H */
