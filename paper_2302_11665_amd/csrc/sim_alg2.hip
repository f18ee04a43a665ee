// Alg. 2 of the paper (Sec. 4.2): enumeration-based group partition and
// model-parallel configuration selection around Alg. 1.
//
//   model buckets   the models sorted by single-device latency (ties by id)
//                   are cut into at most max_buckets contiguous runs, each
//                   spanning at most bucket_threshold seconds of latency, so
//                   models whose latencies differ by more than the threshold
//                   never share a bucket; every such cut is enumerated
//   device buckets  the devices are split among the buckets in multiples of
//                   device_unit; a split is dropped when the buckets' loads
//                   (requests x latency of their models per device) differ
//                   by more than balance_ratio, since buckets should serve
//                   their requests at a similar pace
//   groups/configs  per bucket and parallel configuration c: equal groups of
//                   c's device count, plus one last group with the remaining
//                   devices (the configuration of that size with the deepest
//                   pipeline not deeper than c's)
//   selection       Alg. 1 (or the fast heuristic) on each bucket's options
//                   over the whole trace; requests of other buckets' models
//                   are never served there, so a bucket's served count is its
//                   own; the bucket keeps its strictly best option, the
//                   placement is the concatenation, the search keeps the
//                   strictly best placement.
// Every (bucket, device count, configuration) problem that any kept split
// needs is solved once, and all of them advance in lockstep: one launch per
// step scores the candidates of every problem.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <map>
#include <numeric>
#include <tuple>
#include <vector>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_search.hpp"

namespace as_host {
namespace {

__global__ void count_requests(const int32_t* __restrict__ model, int64_t n, int M,
                               unsigned long long* __restrict__ counts) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t m = model[i];
    if (m >= 0 && m < M) atomicAdd(&counts[m], 1ull);
  }
}

// Contiguous cuts of the sorted model list into 1..K runs whose latency span
// is at most theta, by run count, then cut positions in lexicographic order.
void enum_buckets(const std::vector<double>& dsorted, int K, double theta,
                  std::vector<std::vector<int>>& out) {
  const int M = (int)dsorted.size();
  std::vector<int> starts;
  // recursive over run starts: a partition is the list of run start indices
  std::function<void(int, int)> rec = [&](int pos, int left) {
    if (pos == M) {
      if (left == 0) out.push_back(starts);
      return;
    }
    if (left == 0) return;
    for (int end = pos + 1; end <= M; ++end) {
      if (dsorted[end - 1] - dsorted[pos] > theta) break;
      starts.push_back(pos);
      rec(end, left - 1);
      starts.pop_back();
    }
  };
  for (int k = 1; k <= K && k <= M; ++k) rec(0, k);
}

// Compositions of `units` into k positive parts, lexicographic.
void enum_splits(int units, int k, std::vector<std::vector<int>>& out) {
  std::vector<int> a;
  std::function<void(int, int)> rec = [&](int left, int parts) {
    if (parts == 1) {
      a.push_back(left);
      out.push_back(a);
      a.pop_back();
      return;
    }
    for (int x = 1; x <= left - (parts - 1); ++x) {
      a.push_back(x);
      rec(left - x, parts - 1);
      a.pop_back();
    }
  };
  if (units >= k) rec(units, k);
}

}  // namespace
}  // namespace as_host

using namespace as_host;

extern "C" int as_placement_search(const as_trace_t* trace, const as_models_t* models,
                                   const int64_t* weight_mib, const as_search_opts_t* opts,
                                   as_search_result_t* result, void* stream) {
  if (!trace || !models || !weight_mib || !opts || !result)
    return fail(AS_E_INVALID_ARG, "placement search: NULL argument");
  const as_search_opts_t& o = *opts;
  const int M = models->n_models, C = models->n_configs;
  if (M < 1 || M > AS_MAX_MODELS) return fail(AS_E_LIMITS, "n_models=%d outside 1..%d", M, AS_MAX_MODELS);
  if (C < 1 || C > AS_MAX_CONFIGS) return fail(AS_E_LIMITS, "n_configs=%d outside 1..%d", C, AS_MAX_CONFIGS);
  if (!models->cfg_stages || !o.cfg_devices)
    return fail(AS_E_INVALID_ARG, "placement search: cfg_stages and cfg_devices must not be NULL");
  if (o.n_devices < 1 || o.device_unit < 1 || o.n_devices % o.device_unit != 0)
    return fail(AS_E_INVALID_ARG, "placement search: n_devices=%d must be a positive multiple of device_unit=%d",
                o.n_devices, o.device_unit);
  if (o.max_buckets < 1 || o.max_buckets > AS_MAX_BUCKETS)
    return fail(AS_E_LIMITS, "placement search: max_buckets=%d outside 1..%d", o.max_buckets, AS_MAX_BUCKETS);
  if (!(o.bucket_threshold >= 0.0)) return fail(AS_E_INVALID_ARG, "placement search: bucket_threshold must be >= 0");
  if (!(o.balance_ratio >= 1.0)) return fail(AS_E_INVALID_ARG, "placement search: balance_ratio must be >= 1");
  if (o.beam < 0) return fail(AS_E_INVALID_ARG, "placement search: beam=%d < 0", o.beam);
  if (o.device_mem_mib < 0) return fail(AS_E_INVALID_ARG, "placement search: device_mem_mib < 0");
  if (!(o.slo_scale >= 0.0)) return fail(AS_E_INVALID_ARG, "placement search: slo_scale must be >= 0");
  for (int c = 0; c < C; ++c)
    if (o.cfg_devices[c] < 1) return fail(AS_E_INVALID_ARG, "placement search: cfg_devices[%d] < 1", c);
  if (trace->n < 0 || (trace->n > 0 && (!trace->t || !trace->model)))
    return fail(AS_E_INVALID_ARG, "placement search: bad trace");
  hipStream_t s = (hipStream_t)stream;

  // d_single lives on the device: one copy to the host for the enumeration
  std::vector<double> d(M);
  std::vector<unsigned long long> nreq(M, 0);
  {
    unsigned long long* dc = nullptr;
    hipError_t e = hipMalloc((void**)&dc, (size_t)M * 8);
    if (e != hipSuccess) return fail(AS_E_NOMEM, "placement search: %s", hipGetErrorString(e));
    e = hipMemsetAsync(dc, 0, (size_t)M * 8, s);
    if (e == hipSuccess && trace->n > 0) {
      const int blocks = (int)std::min<int64_t>((trace->n + 255) / 256, 2048);
      hipLaunchKernelGGL(count_requests, dim3(blocks), dim3(256), 0, s, trace->model, trace->n, M, dc);
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpyAsync(nreq.data(), dc, (size_t)M * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(d.data(), models->d_single, (size_t)M * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    hipFree(dc);
    if (e != hipSuccess) return fail(AS_E_HIP, "placement search: %s", hipGetErrorString(e));
  }
  std::vector<int> order(M);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return d[a] < d[b]; });
  std::vector<double> dsorted(M);
  for (int i = 0; i < M; ++i) dsorted[i] = d[order[i]];
  // load of a sorted range [lo, hi): requests x single-device latency
  auto load = [&](int lo, int hi) {
    double x = 0.0;
    for (int i = lo; i < hi; ++i) x += (double)nreq[order[i]] * d[order[i]];
    return x;
  };

  std::vector<std::vector<int>> cuts;
  enum_buckets(dsorted, o.max_buckets, o.bucket_threshold, cuts);
  const int units = o.n_devices / o.device_unit;
  // kept (cut, split) pairs and the distinct (lo, hi, devices) subproblems
  std::vector<std::pair<int, std::vector<int>>> kept;
  std::map<std::tuple<int, int, int>, int> sub_index;
  std::vector<std::tuple<int, int, int>> subs;
  int n_splits = 0;
  for (int ci = 0; ci < (int)cuts.size(); ++ci) {
    const std::vector<int>& st = cuts[ci];
    const int k = (int)st.size();
    std::vector<std::vector<int>> splits;
    enum_splits(units, k, splits);
    for (const std::vector<int>& sp : splits) {
      ++n_splits;
      if (!std::isinf(o.balance_ratio)) {
        double lmin = 0.0, lmax = 0.0;
        for (int b = 0; b < k; ++b) {
          const int lo = st[b], hi = b + 1 < k ? st[b + 1] : M;
          const double rho = load(lo, hi) / (double)(sp[b] * o.device_unit);
          if (b == 0 || rho < lmin) lmin = rho;
          if (b == 0 || rho > lmax) lmax = rho;
        }
        if (!(lmax <= o.balance_ratio * lmin)) continue;
      }
      std::vector<int> ids;
      for (int b = 0; b < k; ++b) {
        const int lo = st[b], hi = b + 1 < k ? st[b + 1] : M;
        const auto key = std::make_tuple(lo, hi, sp[b] * o.device_unit);
        auto it = sub_index.find(key);
        if (it == sub_index.end()) {
          it = sub_index.emplace(key, (int)subs.size()).first;
          subs.push_back(key);
        }
        ids.push_back(it->second);
      }
      kept.emplace_back(ci, ids);
    }
  }

  // the Alg. 1 problems: every configuration option of every subproblem
  std::vector<Problem> probs;
  std::vector<int> prob_sub, prob_cfg;
  for (int q = 0; q < (int)subs.size(); ++q) {
    const int lo = std::get<0>(subs[q]), hi = std::get<1>(subs[q]), H = std::get<2>(subs[q]);
    uint64_t mset = 0;
    for (int i = lo; i < hi; ++i) mset |= 1ull << order[i];
    for (int c = 0; c < C; ++c) {
      const int sz = o.cfg_devices[c];
      if (sz > H) continue;
      const int nfull = H / sz, rem = H % sz;
      int clast = -1;
      if (rem > 0) {
        for (int c2 = 0; c2 < C; ++c2)
          if (o.cfg_devices[c2] == rem && models->cfg_stages[c2] <= models->cfg_stages[c] &&
              (clast < 0 || models->cfg_stages[c2] > models->cfg_stages[clast]))
            clast = c2;
        if (clast < 0) continue;
      }
      const int G = nfull + (rem > 0 ? 1 : 0);
      if (G > AS_MAX_GROUPS) continue;
      Problem pr;
      pr.G = G;
      pr.models = mset;
      for (int g = 0; g < nfull; ++g) {
        pr.cfg.push_back(c);
        pr.mem.push_back((int64_t)sz * o.device_mem_mib);
      }
      if (rem > 0) {
        pr.cfg.push_back(clast);
        pr.mem.push_back((int64_t)rem * o.device_mem_mib);
      }
      probs.push_back(pr);
      prob_sub.push_back(q);
      prob_cfg.push_back(c);
    }
  }
  std::vector<Result> res;
  SearchCount count;
  if (!probs.empty()) {
    const int rc = o.beam == 0 ? fast_search(trace, models, weight_mib, o.slo_scale, probs, res, -1, s, &count)
                               : beam_search(trace, models, weight_mib, o.slo_scale, o.beam, probs, res, -1, s,
                                             &count);
    if (rc != AS_OK) return rc;
  }
  // each subproblem keeps its strictly best option (none: serves nothing)
  std::vector<int> sub_best(subs.size(), -1);
  for (int p = 0; p < (int)probs.size(); ++p) {
    int& b = sub_best[prob_sub[p]];
    const int64_t cur = b < 0 ? 0 : res[b].best_served;
    if (res[p].best_served > cur) b = p;
  }
  // the strictly best concatenation
  std::memset(result, 0, sizeof *result);
  for (int m = 0; m < AS_MAX_MODELS; ++m) result->model_bucket[m] = -1;
  for (int b = 0; b < AS_MAX_BUCKETS; ++b) {
    result->bucket_cfg[b] = -1;
    for (int g = 0; g < AS_MAX_GROUPS; ++g) result->bucket_group_cfg[b][g] = -1;
  }
  int best_k = -1;
  int64_t best = 0;
  for (int kk = 0; kk < (int)kept.size(); ++kk) {
    int64_t tot = 0;
    for (int q : kept[kk].second)
      if (sub_best[q] >= 0) tot += res[sub_best[q]].best_served;
    if (tot > best) {
      best = tot;
      best_k = kk;
    }
  }
  result->n_bucket_configs = (int32_t)cuts.size();
  result->n_device_splits = n_splits;
  result->n_kept_splits = (int32_t)kept.size();
  result->n_problems = (int32_t)probs.size();
  result->launches = count.launches;
  result->jobs_simulated = count.jobs;
  result->served = best;
  if (best_k >= 0) {
    const std::vector<int>& st = cuts[kept[best_k].first];
    const std::vector<int>& ids = kept[best_k].second;
    const int k = (int)st.size();
    result->n_buckets = k;
    for (int b = 0; b < k; ++b) {
      const int lo = st[b], hi = b + 1 < k ? st[b + 1] : M;
      for (int i = lo; i < hi; ++i) result->model_bucket[order[i]] = b;
      const int q = ids[b];
      result->bucket_devices[b] = std::get<2>(subs[q]);
      const int p = sub_best[q];
      result->bucket_cfg[b] = p < 0 ? -1 : prob_cfg[p];
      result->bucket_groups[b] = p < 0 ? 0 : probs[p].G;
      for (int g = 0; g < AS_MAX_GROUPS; ++g)
        result->bucket_group_cfg[b][g] = (p >= 0 && g < probs[p].G) ? probs[p].cfg[g] : -1;
      result->bucket_served[b] = p < 0 ? 0 : res[p].best_served;
      for (int m = 0; m < M; ++m) result->bucket_mask[b][m] = p < 0 ? 0 : res[p].best_mask[m];
    }
  }
  return ok();
}
