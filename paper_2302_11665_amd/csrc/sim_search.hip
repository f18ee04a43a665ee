// Placement search drivers over the batched simulator (Sec. 4.2): Alg. 1
// (simulator-guided greedy selection) and Alg. 2 (enumeration of group
// partitions and parallel configurations).  Every candidate of a step is a
// job of one batched launch on the caller's stream; the host keeps only the
// selection state and the argmax.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"

namespace as_host {
namespace {

// ------------------------------------------------------------ greedy search
// Candidate placements of one greedy step: row p is the current selection with
// model cand[2p] added to group cand[2p+1].
__global__ void expand_candidates(const uint64_t* __restrict__ base, const int32_t* __restrict__ cand,
                                  int P, int M, uint64_t* __restrict__ masks) {
  const int64_t n = (int64_t)P * M;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int p = (int)(i / M), m = (int)(i % M);
    masks[i] = base[m] | (cand[2 * p] == m ? (1ull << cand[2 * p + 1]) : 0ull);
  }
}

// Device buffers of a greedy search, sized for M x G candidates per step.
struct GreedyBufs {
  int32_t* gcfg = nullptr;   // [Pmax][G] the partition, repeated per candidate
  uint64_t* masks = nullptr; // [Pmax][M]
  int32_t* cand = nullptr;   // [Pmax][2]
  uint64_t* base = nullptr;  // [M]
  int64_t* served = nullptr; // [Pmax]
  double* scale = nullptr;   // [1]
  void release() {
    hipFree(gcfg);
    hipFree(masks);
    hipFree(cand);
    hipFree(base);
    hipFree(served);
    hipFree(scale);
  }
};

int greedy_one(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
               int32_t G, const int32_t* group_cfg, const int64_t* group_mem_mib, double slo_scale,
               uint64_t* best_mask, int64_t* best_served, int32_t* step_model, int32_t* step_group,
               int64_t* step_served, int32_t max_steps, int32_t* n_steps, hipStream_t s) {
  if (!trace || !models || !weight_mib || !group_cfg || !group_mem_mib || !best_mask ||
      !best_served || !n_steps)
    return fail(AS_E_INVALID_ARG, "greedy: NULL argument");
  if (trace->n < 0 || (trace->n > 0 && (!trace->t || !trace->model)))
    return fail(AS_E_INVALID_ARG, "greedy: bad trace");
  if (max_steps < 0 || (max_steps > 0 && (!step_model || !step_group || !step_served)))
    return fail(AS_E_INVALID_ARG, "greedy: bad trajectory buffers");
  if (!(slo_scale >= 0.0)) return fail(AS_E_INVALID_ARG, "greedy: slo_scale must be >= 0");
  if (G < 1 || G > AS_MAX_GROUPS) return fail(AS_E_LIMITS, "greedy: n_groups=%d outside 1..%d", G, AS_MAX_GROUPS);
  // shape checks shared with the simulate entry points (placements filled later)
  // shape checks shared with the simulate entry points; the placement arrays
  // are the driver's own device buffers, set below (placeholders here)
  as_placements_t pl{1, G, group_cfg, reinterpret_cast<const uint64_t*>(group_cfg)};
  KArgs a;
  std::memset(&a, 0, sizeof a);
  int W = 1, smax = 1;
  {
    const int rc = check_common(models, &pl, a, W, smax);
    if (rc != AS_OK) return rc;
  }
  const int M = models->n_models;
  // the partition's configurations decide the padded stage count
  int smax_used = 1;
  for (int g = 0; g < G; ++g) {
    const int c = group_cfg[g];
    if (c < -1 || c >= models->n_configs)
      return fail(AS_E_INVALID_ARG, "greedy: group_cfg[%d]=%d outside [-1, %d)", g, c, models->n_configs);
    if (c >= 0 && models->cfg_stages[c] > smax_used) smax_used = models->cfg_stages[c];
    if (group_mem_mib[g] < 0) return fail(AS_E_INVALID_ARG, "greedy: group_mem_mib[%d] < 0", g);
  }
  for (int m = 0; m < M; ++m)
    if (weight_mib[m] < 0) return fail(AS_E_INVALID_ARG, "greedy: weight_mib[%d] < 0", m);
  smax = pow2ceil(smax_used);

  const int Pmax = M * G;
  GreedyBufs b;
  hipError_t e = hipSuccess;
  if ((e = hipMalloc((void**)&b.gcfg, (size_t)Pmax * G * 4)) != hipSuccess ||
      (e = hipMalloc((void**)&b.masks, (size_t)Pmax * M * 8)) != hipSuccess ||
      (e = hipMalloc((void**)&b.cand, (size_t)Pmax * 2 * 4)) != hipSuccess ||
      (e = hipMalloc((void**)&b.base, (size_t)M * 8)) != hipSuccess ||
      (e = hipMalloc((void**)&b.served, (size_t)Pmax * 8)) != hipSuccess ||
      (e = hipMalloc((void**)&b.scale, 8)) != hipSuccess) {
    b.release();
    return fail(AS_E_NOMEM, "greedy: device allocation failed: %s", hipGetErrorString(e));
  }
  std::vector<int32_t> rep((size_t)Pmax * G);
  for (int p = 0; p < Pmax; ++p)
    for (int g = 0; g < G; ++g) rep[(size_t)p * G + g] = group_cfg[g];
  e = hipMemcpyAsync(b.gcfg, rep.data(), rep.size() * 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipMemcpyAsync(b.scale, &slo_scale, 8, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    b.release();
    return fail(AS_E_HIP, "greedy: upload failed: %s", hipGetErrorString(e));
  }

  a.t = trace->t;
  a.model = trace->model;
  a.n = trace->n;
  a.group_cfg = b.gcfg;
  a.host_mask = b.masks;
  a.slo_scale = b.scale;
  a.K = 1;
  a.out_served = b.served;

  std::vector<uint64_t> hosted(M, 0), best(M, 0);
  std::vector<int64_t> used(G, 0);
  std::vector<int32_t> cand;
  std::vector<int64_t> served;
  int64_t best_s = 0;
  int32_t steps = 0;
  int rc = AS_OK;
  for (;;) {
    cand.clear();
    for (int m = 0; m < M; ++m)
      for (int g = 0; g < G; ++g)
        if (group_cfg[g] >= 0 && !((hosted[m] >> g) & 1u) && used[g] + weight_mib[m] <= group_mem_mib[g]) {
          cand.push_back(m);
          cand.push_back(g);
        }
    const int P = (int)(cand.size() / 2);
    if (P == 0) break;
    e = hipMemcpyAsync(b.cand, cand.data(), cand.size() * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(b.base, hosted.data(), (size_t)M * 8, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) {
      int blocks = (int)(((int64_t)P * M + 255) / 256);
      if (blocks > 4096) blocks = 4096;
      hipLaunchKernelGGL(expand_candidates, dim3(blocks), dim3(256), 0, s, b.base, b.cand, P, M, b.masks);
      e = hipGetLastError();
    }
    if (e != hipSuccess) {
      rc = fail(AS_E_HIP, "greedy: step %d: %s", steps, hipGetErrorString(e));
      break;
    }
    a.P = P;
    a.J = P;
    rc = run_shared_trace(a, G, smax, s);
    if (rc != AS_OK) break;
    served.resize(P);
    e = hipMemcpyAsync(served.data(), b.served, (size_t)P * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      rc = fail(AS_E_HIP, "greedy: step %d: %s", steps, hipGetErrorString(e));
      break;
    }
    int bi = 0;
    for (int i = 1; i < P; ++i)
      if (served[i] > served[bi]) bi = i;
    const int m = cand[2 * bi], g = cand[2 * bi + 1];
    hosted[m] |= 1ull << g;
    used[g] += weight_mib[m];
    if (steps < max_steps) {
      step_model[steps] = m;
      step_group[steps] = g;
      step_served[steps] = served[bi];
    }
    ++steps;
    if (served[bi] > best_s) {
      best_s = served[bi];
      best = hosted;
    }
  }
  b.release();
  if (rc != AS_OK) return rc;
  for (int m = 0; m < M; ++m) best_mask[m] = best[m];
  *best_served = best_s;
  *n_steps = steps;
  return ok();
}

}  // namespace
}  // namespace as_host

using namespace as_host;

extern "C" {

int as_greedy_placement(const as_trace_t* trace, const as_models_t* models,
                        const int64_t* weight_mib, int32_t n_groups, const int32_t* group_cfg,
                        const int64_t* group_mem_mib, double slo_scale, uint64_t* best_mask,
                        int64_t* best_served, int32_t* step_model, int32_t* step_group,
                        int64_t* step_served, int32_t max_steps, int32_t* n_steps,
                        void* stream) {
  return greedy_one(trace, models, weight_mib, n_groups, group_cfg, group_mem_mib, slo_scale,
                    best_mask, best_served, step_model, step_group, step_served, max_steps, n_steps,
                    (hipStream_t)stream);
}

int as_partition_search(const as_trace_t* trace, const as_models_t* models,
                        const int64_t* weight_mib, int32_t n_partitions, const int32_t* part_groups,
                        const int32_t* part_cfg, const int64_t* part_mem_mib, double slo_scale,
                        int32_t* best_partition, uint64_t* best_mask, int64_t* best_served,
                        int64_t* part_served, void* stream) {
  if (n_partitions < 1 || !part_groups || !part_cfg || !part_mem_mib || !best_partition ||
      !best_mask || !best_served || !part_served || !models)
    return fail(AS_E_INVALID_ARG, "partition search: bad arguments");
  const int M = models->n_models;
  if (M < 1 || M > AS_MAX_MODELS) return fail(AS_E_LIMITS, "n_models=%d outside 1..%d", M, AS_MAX_MODELS);
  std::vector<uint64_t> mask(M);
  int64_t off = 0;
  int32_t best_p = -1;
  int64_t best_s = -1;
  for (int p = 0; p < n_partitions; ++p) {
    int64_t s_p = 0;
    int32_t steps = 0;
    int rc = greedy_one(trace, models, weight_mib, part_groups[p], part_cfg + off, part_mem_mib + off,
                        slo_scale, mask.data(), &s_p, nullptr, nullptr, nullptr, 0, &steps,
                        (hipStream_t)stream);
    if (rc != AS_OK) return rc;
    part_served[p] = s_p;
    if (s_p > best_s) {
      best_s = s_p;
      best_p = p;
      for (int m = 0; m < M; ++m) best_mask[m] = mask[m];
    }
    off += part_groups[p];
  }
  *best_partition = best_p;
  *best_served = best_s;
  return ok();
}

}  // extern "C"
