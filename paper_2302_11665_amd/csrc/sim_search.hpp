// Lockstep placement searches (Alg. 1 with any beam, the fast heuristic of
// Sec. 4.2) shared by the search entry points.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"

namespace as_host {

// One Alg. 1 problem: a group partition with one configuration per group,
// the memory of each group (MiB) and the models that may be placed (bit m).
struct Problem {
  int G = 0;
  std::vector<int32_t> cfg;  // [G], -1 = no group
  std::vector<int64_t> mem;  // [G]
  uint64_t models = 0;
};

// Outcome of one search: the best selection seen (replaced only by a strictly
// better one; the empty selection serves 0) and one record per step.
struct Result {
  std::vector<uint64_t> best_mask;  // [M]
  int64_t best_served = 0;
  int32_t steps = 0;
  std::vector<int32_t> step_model, step_group, step_parent, step_candidates;
  std::vector<int64_t> step_served;
};

// Work done by a search call: batched launches and jobs (each job simulates
// the whole trace once).
struct SearchCount {
  int64_t launches = 0;
  int64_t jobs = 0;
};

// Alg. 1 with beam size `beam` on every problem; all candidates of all
// active problems of a step are one batched launch.  max_steps < 0: no limit.
int beam_search(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                double slo_scale, int beam, const std::vector<Problem>& probs, std::vector<Result>& res,
                int max_steps, hipStream_t s, SearchCount* count = nullptr);

// The fast heuristic on every problem; one job per active problem per step.
int fast_search(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                double slo_scale, const std::vector<Problem>& probs, std::vector<Result>& res,
                int max_steps, hipStream_t s, SearchCount* count = nullptr);

}  // namespace as_host
