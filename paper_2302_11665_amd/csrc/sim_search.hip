// Placement search drivers over the batched simulator (Sec. 4.2): Alg. 1
// (simulator-guided greedy selection, any beam size), the fast heuristic that
// Sec. 4.2 proposes for very large workloads, and Alg. 2 (enumeration of
// group partitions and parallel configurations).
//
// Several independent searches (the partitions of Alg. 2, the buckets of a
// bucket configuration) advance in lockstep: every candidate of every active
// search in one step is a job of one batched launch on the caller's stream,
// so a step fills the GPU with all of them at once.  The host keeps only the
// selection states, the feasibility checks and the argmax.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <string>
#include <unordered_set>
#include <vector>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_search.hpp"

namespace as_host {
namespace {

// Candidate placements of one step: row p is base row cand[4p] with model
// cand[4p+1] added to group cand[4p+2], in the group layout of search
// cand[4p+3] (its row of cfg_tab, Gtab entries); rows have G groups.
__global__ void expand_candidates(const uint64_t* __restrict__ base, const int32_t* __restrict__ cand,
                                  const int32_t* __restrict__ cfg_tab, int Gtab, int P, int M, int G,
                                  uint64_t* __restrict__ masks, int32_t* __restrict__ gcfg) {
  const int64_t nm = (int64_t)P * M, ng = (int64_t)P * G;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nm + ng; i += stride) {
    if (i < nm) {
      const int p = (int)(i / M), m = (int)(i % M);
      const int32_t* c = cand + 4 * (int64_t)p;
      masks[i] = base[(int64_t)c[0] * M + m] | (c[1] == m ? (1ull << c[2]) : 0ull);
    } else {
      const int64_t k = i - nm;
      const int p = (int)(k / G), g = (int)(k % G);
      gcfg[k] = g < Gtab ? cfg_tab[(int64_t)cand[4 * (int64_t)p + 3] * Gtab + g] : -1;
    }
  }
}

// Side streams and events of one search call (default priority), created on
// first use and destroyed with the call.
struct StreamPool {
  std::vector<hipStream_t> st;
  std::vector<hipEvent_t> ev;
  hipError_t get(size_t k) {
    while (st.size() <= k) {
      hipStream_t x = nullptr;
      hipEvent_t y = nullptr;
      hipError_t e = hipStreamCreateWithFlags(&x, hipStreamNonBlocking);
      if (e != hipSuccess) return e;
      st.push_back(x);
      e = hipEventCreateWithFlags(&y, hipEventDisableTiming);
      if (e != hipSuccess) return e;
      ev.push_back(y);
    }
    return hipSuccess;
  }
  ~StreamPool() {
    for (hipStream_t x : st) (void)hipStreamDestroy(x);
    for (hipEvent_t y : ev) (void)hipEventDestroy(y);
  }
};

// Requests of each model in the trace (the fast heuristic's unserved counts
// are these minus the served ones).
__global__ void count_models(const int32_t* __restrict__ model, int64_t n, int M,
                             unsigned long long* __restrict__ counts) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t m = model[i];
    if (m >= 0 && m < M) atomicAdd(&counts[m], 1ull);
  }
}

// Device buffers, grown on demand and freed at the end of a search call.
struct DevBufs {
  void* p[8] = {nullptr};
  size_t cap[8] = {0};
  hipError_t need(int k, size_t bytes) {
    if (bytes <= cap[k]) return hipSuccess;
    if (p[k]) (void)hipFree(p[k]);
    p[k] = nullptr;
    cap[k] = 0;
    const hipError_t e = hipMalloc(&p[k], bytes < 256 ? 256 : bytes);
    if (e == hipSuccess) cap[k] = bytes;
    return e;
  }
  ~DevBufs() {
    for (void* q : p)
      if (q) (void)hipFree(q);
  }
};

struct MaskHash {
  size_t operator()(const std::vector<uint64_t>& v) const {
    uint64_t h = 0x9E3779B97F4A7C15ULL;
    for (uint64_t x : v) h = (h ^ x) * 0xBF58476D1CE4E5B9ULL;
    return (size_t)h;
  }
};

// One selection of a search: hosting masks and memory used per group.
struct Sel {
  std::vector<uint64_t> mask;  // [M]
  std::vector<int64_t> used;   // [G]
};

bool fits(const Problem& pr, const Sel& s, const int64_t* w, int m, int g) {
  return pr.cfg[g] >= 0 && !((s.mask[m] >> g) & 1u) && s.used[g] + w[m] <= pr.mem[g];
}

}  // namespace

int check_search_common(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                        double slo_scale, const std::vector<Problem>& probs, KArgs& a, int& smax) {
  if (!trace || !models || !weight_mib) return fail(AS_E_INVALID_ARG, "search: NULL argument");
  if (trace->n < 0 || (trace->n > 0 && (!trace->t || !trace->model)))
    return fail(AS_E_INVALID_ARG, "search: bad trace");
  if (!(slo_scale >= 0.0)) return fail(AS_E_INVALID_ARG, "search: slo_scale must be >= 0");
  int Gmax = 1;
  for (const Problem& pr : probs) Gmax = std::max(Gmax, pr.G);
  if (Gmax > AS_MAX_GROUPS) return fail(AS_E_LIMITS, "search: %d groups > %d", Gmax, AS_MAX_GROUPS);
  // placement arrays are the driver's own device buffers, set per launch
  as_placements_t pl{1, Gmax, reinterpret_cast<const int32_t*>(weight_mib),
                     reinterpret_cast<const uint64_t*>(weight_mib)};
  std::memset(&a, 0, sizeof a);
  int W = 1;
  const int rc = check_common(models, &pl, a, W, smax);
  if (rc != AS_OK) return rc;
  int smax_used = 1;
  for (const Problem& pr : probs) {
    if (pr.G < 1) return fail(AS_E_INVALID_ARG, "search: a partition has no group");
    for (int g = 0; g < pr.G; ++g) {
      const int c = pr.cfg[g];
      if (c < -1 || c >= models->n_configs)
        return fail(AS_E_INVALID_ARG, "search: group configuration %d outside [-1, %d)", c, models->n_configs);
      if (c >= 0) smax_used = std::max(smax_used, models->cfg_stages[c]);
      if (pr.mem[g] < 0) return fail(AS_E_INVALID_ARG, "search: negative group memory");
    }
  }
  for (int m = 0; m < models->n_models; ++m)
    if (weight_mib[m] < 0) return fail(AS_E_INVALID_ARG, "search: weight_mib[%d] < 0", m);
  smax = pow2ceil(smax_used);
  a.G = Gmax;
  return AS_OK;
}

// Alg. 1 with beam size `beam` on every problem, in lockstep.
int beam_search(const as_trace_t* trace, const as_models_t* models, const int64_t* w, double slo_scale,
                int beam, const std::vector<Problem>& probs, std::vector<Result>& res, int max_steps,
                hipStream_t s, SearchCount* count) {
  if (beam < 1) return fail(AS_E_INVALID_ARG, "search: beam=%d < 1", beam);
  KArgs a;
  int smax = 1;
  int rc = check_search_common(trace, models, w, slo_scale, probs, a, smax);
  if (rc != AS_OK) return rc;
  const int M = models->n_models, G = a.G, R = (int)probs.size();
  res.assign(R, Result());
  std::vector<std::vector<Sel>> beams(R);
  std::vector<char> active(R, 1);
  for (int r = 0; r < R; ++r) {
    Sel e{std::vector<uint64_t>(M, 0), std::vector<int64_t>(probs[r].G, 0)};
    beams[r].push_back(e);
    res[r].best_mask.assign(M, 0);
  }
  std::vector<int32_t> cfg_tab((size_t)R * G, -1);
  for (int r = 0; r < R; ++r)
    for (int g = 0; g < probs[r].G; ++g) cfg_tab[(size_t)r * G + g] = probs[r].cfg[g];

  DevBufs d;
  hipError_t e = d.need(0, cfg_tab.size() * 4);
  if (e == hipSuccess) e = d.need(1, 8);
  if (e != hipSuccess) return fail(AS_E_NOMEM, "search: device allocation failed: %s", hipGetErrorString(e));
  e = hipMemcpyAsync(d.p[0], cfg_tab.data(), cfg_tab.size() * 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipMemcpyAsync(d.p[1], &slo_scale, 8, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(AS_E_HIP, "search: upload failed: %s", hipGetErrorString(e));

  a.t = trace->t;
  a.model = trace->model;
  a.n = trace->n;
  a.slo_scale = static_cast<const double*>(d.p[1]);
  a.K = 1;
  // kernel shape of each search: lanes per job (its group count rounded up
  // to a power of two) and padded stage count (its deepest configuration)
  std::vector<int> shape_of(R), shape_w, shape_s;
  for (int r = 0; r < R; ++r) {
    int sm = 1;
    for (int g = 0; g < probs[r].G; ++g)
      if (probs[r].cfg[g] >= 0) sm = std::max(sm, models->cfg_stages[probs[r].cfg[g]]);
    const int wr = pow2ceil(probs[r].G), sr = pow2ceil(sm);
    int k = 0;
    while (k < (int)shape_w.size() && !(shape_w[k] == wr && shape_s[k] == sr)) ++k;
    if (k == (int)shape_w.size()) {
      shape_w.push_back(wr);
      shape_s.push_back(sr);
    }
    shape_of[r] = k;
  }
  StreamPool pool;

  // candidate c of a step: (base row, model, group, search), and the new
  // selection it makes (kept on the host for dedup and the next beam)
  std::vector<int32_t> cand;
  std::vector<uint64_t> bases;
  std::vector<Sel> news;
  std::vector<int> cand_search;
  std::vector<int64_t> served;
  for (int step = 0; max_steps < 0 || step < max_steps; ++step) {
    cand.clear();
    bases.clear();
    news.clear();
    cand_search.clear();
    std::vector<int> first(R + 1, 0);
    int nbase = 0;
    for (int r = 0; r < R; ++r) {
      first[r] = (int)news.size();
      if (!active[r]) continue;
      const Problem& pr = probs[r];
      std::unordered_set<std::vector<uint64_t>, MaskHash> seen;
      for (size_t b = 0; b < beams[r].size(); ++b) {
        const Sel& sel = beams[r][b];
        const int base_row = nbase++;
        bases.insert(bases.end(), sel.mask.begin(), sel.mask.end());
        for (int m = 0; m < M; ++m) {
          if (!((pr.models >> m) & 1u)) continue;
          for (int g = 0; g < pr.G; ++g) {
            if (!fits(pr, sel, w, m, g)) continue;
            Sel nsel = sel;
            nsel.mask[m] |= 1ull << g;
            if (beam > 1 && !seen.insert(nsel.mask).second) continue;
            nsel.used[g] += w[m];
            cand.insert(cand.end(), {base_row, m, g, r});
            news.push_back(std::move(nsel));
            cand_search.push_back((int)b);
          }
        }
      }
      if ((int)news.size() == first[r]) active[r] = 0;
    }
    first[R] = (int)news.size();
    const int P = (int)news.size();
    if (P == 0) break;
    // one launch per kernel shape (lanes per job, padded stages), the shapes'
    // launches running side by side on their own streams: a search's jobs are
    // laid out for its own group count and pipeline depth, not the widest
    std::vector<int> order(P);
    for (int i = 0; i < P; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
      return shape_of[cand[4 * (size_t)x + 3]] < shape_of[cand[4 * (size_t)y + 3]];
    });
    std::vector<int32_t> cand_sorted((size_t)P * 4);
    for (int i = 0; i < P; ++i)
      for (int k = 0; k < 4; ++k) cand_sorted[4 * (size_t)i + k] = cand[4 * (size_t)order[i] + k];
    struct Launch {
      int shape, begin, end;
      size_t gofs;
    };
    std::vector<Launch> launches;
    size_t gtotal = 0;
    for (int i = 0; i < P;) {
      const int sh = shape_of[cand_sorted[4 * (size_t)i + 3]];
      int j = i;
      while (j < P && shape_of[cand_sorted[4 * (size_t)j + 3]] == sh) ++j;
      launches.push_back({sh, i, j, gtotal});
      gtotal += (size_t)(j - i) * shape_w[sh];
      i = j;
    }
    e = d.need(2, bases.size() * 8);
    if (e == hipSuccess) e = d.need(3, cand_sorted.size() * 4);
    if (e == hipSuccess) e = d.need(4, (size_t)P * M * 8);
    if (e == hipSuccess) e = d.need(5, gtotal * 4);
    if (e == hipSuccess) e = d.need(6, (size_t)P * 8);
    if (e != hipSuccess) return fail(AS_E_NOMEM, "search: device allocation failed: %s", hipGetErrorString(e));
    e = hipMemcpyAsync(d.p[2], bases.data(), bases.size() * 8, hipMemcpyHostToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(d.p[3], cand_sorted.data(), cand_sorted.size() * 4, hipMemcpyHostToDevice, s);
    for (const Launch& L : launches) {
      if (e != hipSuccess) break;
      const int Pc = L.end - L.begin, Gc = shape_w[L.shape];
      const int64_t work = (int64_t)Pc * (M + Gc);
      const int blocks = (int)std::min<int64_t>((work + 255) / 256, 4096);
      hipLaunchKernelGGL(expand_candidates, dim3(blocks), dim3(256), 0, s,
                         static_cast<const uint64_t*>(d.p[2]),
                         static_cast<const int32_t*>(d.p[3]) + 4 * (size_t)L.begin,
                         static_cast<const int32_t*>(d.p[0]), G, Pc, M, Gc,
                         static_cast<uint64_t*>(d.p[4]) + (size_t)L.begin * M,
                         static_cast<int32_t*>(d.p[5]) + L.gofs);
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = d.need(7, sizeof(KArgs));
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    // every shape in one dispatch; else one launch per shape, side by side
    // on streams of their own
    std::vector<ShapeJobs> shj;
    for (const Launch& L : launches) {
      ShapeJobs x;
      x.W = shape_w[L.shape];
      x.smax = shape_s[L.shape];
      x.v = as_dev::JobSet{L.end - L.begin, shape_w[L.shape], static_cast<const int32_t*>(d.p[5]) + L.gofs,
                           static_cast<const uint64_t*>(d.p[4]) + (size_t)L.begin * M,
                           static_cast<int64_t*>(d.p[6]) + L.begin, nullptr, nullptr, nullptr, nullptr};
      shj.push_back(x);
    }
    rc = run_shared_multi(a, d.p[7], shj.data(), (int)shj.size(), false, s);
    if (rc != AS_E_LIMITS && rc != AS_OK) return rc;
    const bool multi = rc == AS_OK;
    if (multi && count) {
      count->launches += 1;
      count->jobs += P;
    }
    if (!multi && e == hipSuccess) e = pool.get(launches.size());
    // the last event of the pool marks the expanded inputs on the caller's stream
    if (!multi && e == hipSuccess) e = hipEventRecord(pool.ev[launches.size()], s);
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    for (size_t k = 0; !multi && k < launches.size(); ++k) {
      const Launch& L = launches[k];
      hipStream_t sk = launches.size() == 1 ? s : pool.st[k];
      if (sk != s && (e = hipStreamWaitEvent(sk, pool.ev[launches.size()], 0)) != hipSuccess)
        return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
      KArgs ak = a;
      ak.group_cfg = static_cast<const int32_t*>(d.p[5]) + L.gofs;
      ak.host_mask = static_cast<const uint64_t*>(d.p[4]) + (size_t)L.begin * M;
      ak.out_served = static_cast<int64_t*>(d.p[6]) + L.begin;
      ak.P = L.end - L.begin;
      ak.J = ak.P;
      ak.G = shape_w[L.shape];
      rc = run_shared_trace(ak, ak.G, shape_s[L.shape], sk);
      if (rc != AS_OK) return rc;
      if (sk != s) {
        if ((e = hipEventRecord(pool.ev[k], sk)) != hipSuccess || (e = hipStreamWaitEvent(s, pool.ev[k], 0)) != hipSuccess)
          return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
      }
      if (count) {
        count->launches += 1;
        count->jobs += ak.P;
      }
    }
    std::vector<int64_t> served_sorted(P);
    e = hipMemcpyAsync(served_sorted.data(), d.p[6], (size_t)P * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    served.assign(P, 0);
    for (int i = 0; i < P; ++i) served[order[i]] = served_sorted[i];
    for (int r = 0; r < R; ++r) {
      if (first[r] == first[r + 1]) continue;
      // top-k by served count, the earlier candidate first on ties
      std::vector<int> idx;
      for (int i = first[r]; i < first[r + 1]; ++i) idx.push_back(i);
      std::stable_sort(idx.begin(), idx.end(), [&](int x, int y) { return served[x] > served[y]; });
      if ((int)idx.size() > beam) idx.resize(beam);
      std::vector<Sel> nb;
      for (int i : idx) nb.push_back(news[i]);
      beams[r].swap(nb);
      const int i0 = idx[0];
      Result& out = res[r];
      out.step_parent.push_back(cand_search[i0]);
      out.step_model.push_back(cand[4 * (size_t)i0 + 1]);
      out.step_group.push_back(cand[4 * (size_t)i0 + 2]);
      out.step_served.push_back(served[i0]);
      out.step_candidates.push_back(first[r + 1] - first[r]);
      ++out.steps;
      if (served[i0] > out.best_served) {
        out.best_served = served[i0];
        out.best_mask = beams[r][0].mask;
      }
    }
  }
  return ok();
}

// The fast heuristic of Sec. 4.2 on every problem, in lockstep: simulate each
// current selection once (one job per search), then place the model with the
// most unserved requests on its available group with the least busy time.
int fast_search(const as_trace_t* trace, const as_models_t* models, const int64_t* w, double slo_scale,
                const std::vector<Problem>& probs, std::vector<Result>& res, int max_steps,
                hipStream_t s, SearchCount* count) {
  KArgs a;
  int smax = 1;
  int rc = check_search_common(trace, models, w, slo_scale, probs, a, smax);
  if (rc != AS_OK) return rc;
  const int M = models->n_models, G = a.G, R = (int)probs.size();
  res.assign(R, Result());
  std::vector<Sel> cur(R);
  std::vector<char> active(R, 1);
  for (int r = 0; r < R; ++r) {
    cur[r] = Sel{std::vector<uint64_t>(M, 0), std::vector<int64_t>(probs[r].G, 0)};
    res[r].best_mask.assign(M, 0);
  }
  // kernel shape of each problem: lanes per job (its group count rounded up
  // to a power of two) and padded stage count (its deepest configuration);
  // each step runs one statistics launch per shape, side by side, so a job's
  // per-request chain is only as wide and as deep as its own partition
  std::vector<int> shape_of(R), shape_w, shape_s;
  for (int r = 0; r < R; ++r) {
    int sm = 1;
    for (int g = 0; g < probs[r].G; ++g)
      if (probs[r].cfg[g] >= 0) sm = std::max(sm, models->cfg_stages[probs[r].cfg[g]]);
    const int wr = pow2ceil(probs[r].G), sr = pow2ceil(sm);
    int k = 0;
    while (k < (int)shape_w.size() && !(shape_w[k] == wr && shape_s[k] == sr)) ++k;
    if (k == (int)shape_w.size()) {
      shape_w.push_back(wr);
      shape_s.push_back(sr);
    }
    shape_of[r] = k;
  }
  const int Gp = pow2ceil(G);  // the widest row stride of a shape
  StreamPool pool;

  DevBufs d;
  hipError_t e = d.need(0, (size_t)R * Gp * 4);     // group configurations of the jobs
  if (e == hipSuccess) e = d.need(1, 8);            // the scale
  if (e == hipSuccess) e = d.need(2, (size_t)M * 8);  // per-model request counts
  if (e == hipSuccess) e = d.need(3, (size_t)R * M * 8);  // masks
  if (e == hipSuccess) e = d.need(4, (size_t)R * 8);      // served
  if (e == hipSuccess) e = d.need(5, (size_t)R * M * 8);  // per-model served
  if (e == hipSuccess) e = d.need(6, (size_t)R * Gp * 8);  // busy
  if (e != hipSuccess) return fail(AS_E_NOMEM, "search: device allocation failed: %s", hipGetErrorString(e));
  std::vector<unsigned long long> n_req(M, 0);
  e = hipMemcpyAsync(d.p[1], &slo_scale, 8, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipMemsetAsync(d.p[2], 0, (size_t)M * 8, s);
  if (e == hipSuccess && trace->n > 0) {
    const int blocks = (int)std::min<int64_t>((trace->n + 255) / 256, 2048);
    hipLaunchKernelGGL(count_models, dim3(blocks), dim3(256), 0, s, trace->model, trace->n, M,
                       static_cast<unsigned long long*>(d.p[2]));
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpyAsync(n_req.data(), d.p[2], (size_t)M * 8, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(AS_E_HIP, "search: setup failed: %s", hipGetErrorString(e));

  std::vector<int> live;
  std::vector<int32_t> gcfg;
  std::vector<uint64_t> masks;
  std::vector<int64_t> served, ms;
  std::vector<double> busy;
  struct Launch {
    int shape, begin, end;
    size_t gofs;  // first row entry of the shape's configuration and busy rows
  };
  std::vector<Launch> launches;
  std::vector<size_t> brow;  // live job q: its busy row's first entry
  for (int step = 0;; ++step) {
    live.clear();
    for (int r = 0; r < R; ++r)
      if (active[r]) live.push_back(r);
    if (live.empty()) break;
    std::stable_sort(live.begin(), live.end(), [&](int x, int y) { return shape_of[x] < shape_of[y]; });
    const int P = (int)live.size();
    launches.clear();
    brow.assign(P, 0);
    size_t gtotal = 0;
    for (int q = 0; q < P;) {
      const int sh = shape_of[live[q]];
      int q1 = q;
      while (q1 < P && shape_of[live[q1]] == sh) ++q1;
      launches.push_back({sh, q, q1, gtotal});
      for (int x = q; x < q1; ++x) brow[x] = gtotal + (size_t)(x - q) * shape_w[sh];
      gtotal += (size_t)(q1 - q) * shape_w[sh];
      q = q1;
    }
    gcfg.assign(gtotal, -1);
    masks.clear();
    for (int q = 0; q < P; ++q) {
      const int r = live[q];
      std::copy(probs[r].cfg.begin(), probs[r].cfg.end(), gcfg.begin() + brow[q]);
      masks.insert(masks.end(), cur[r].mask.begin(), cur[r].mask.end());
    }
    e = hipMemcpyAsync(d.p[0], gcfg.data(), gcfg.size() * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(d.p[3], masks.data(), masks.size() * 8, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = d.need(7, sizeof(KArgs));
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    // every shape in one dispatch; else one launch per shape, side by side
    // on streams of their own
    KArgs am = a;
    am.t = trace->t;
    am.model = trace->model;
    am.n = trace->n;
    am.slo_scale = static_cast<const double*>(d.p[1]);
    am.K = 1;
    am.n_finish = 0;
    std::vector<ShapeJobs> shj;
    for (const Launch& L : launches)
      shj.push_back(ShapeJobs{shape_w[L.shape], shape_s[L.shape],
                              as_dev::JobSet{L.end - L.begin, shape_w[L.shape],
                                             static_cast<const int32_t*>(d.p[0]) + L.gofs,
                                             static_cast<const uint64_t*>(d.p[3]) + (size_t)L.begin * M,
                                             static_cast<int64_t*>(d.p[4]) + L.begin, nullptr, nullptr,
                                             static_cast<int64_t*>(d.p[5]) + (size_t)L.begin * M,
                                             static_cast<double*>(d.p[6]) + L.gofs}});
    rc = run_shared_multi(am, d.p[7], shj.data(), (int)shj.size(), true, s);
    if (rc != AS_E_LIMITS && rc != AS_OK) return rc;
    const bool multi = rc == AS_OK;
    if (multi && count) {
      count->launches += 1;
      count->jobs += P;
    }
    if (!multi && e == hipSuccess) e = pool.get(launches.size());
    if (!multi && e == hipSuccess) e = hipEventRecord(pool.ev[launches.size()], s);
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    for (size_t k = 0; !multi && k < launches.size(); ++k) {
      const Launch& L = launches[k];
      hipStream_t sk = launches.size() == 1 ? s : pool.st[k];
      if (sk != s && (e = hipStreamWaitEvent(sk, pool.ev[launches.size()], 0)) != hipSuccess)
        return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
      const int Pk = L.end - L.begin, Gk = shape_w[L.shape];
      const int32_t* gk = static_cast<const int32_t*>(d.p[0]) + L.gofs;
      const uint64_t* mk = static_cast<const uint64_t*>(d.p[3]) + (size_t)L.begin * M;
      int64_t* sv = static_cast<int64_t*>(d.p[4]) + L.begin;
      int64_t* msv = static_cast<int64_t*>(d.p[5]) + (size_t)L.begin * M;
      double* bz = static_cast<double*>(d.p[6]) + L.gofs;
      KArgs ak = a;
      ak.t = trace->t;
      ak.model = trace->model;
      ak.n = trace->n;
      ak.slo_scale = static_cast<const double*>(d.p[1]);
      ak.K = 1;
      ak.P = Pk;
      ak.J = Pk;
      ak.G = Gk;
      ak.group_cfg = gk;
      ak.host_mask = mk;
      ak.out_served = sv;
      ak.out_digest = nullptr;
      ak.out_model_served = msv;
      ak.out_group_busy = bz;
      ak.n_finish = 0;
      rc = run_shared_stats(ak, shape_s[L.shape], sk);
      if (rc == AS_E_LIMITS) {
        // the shared-trace kernel does not take it: the general statistics kernel
        as_placements_t pl{Pk, Gk, gk, mk};
        rc = as_simulate_stats(trace, models, &pl, static_cast<const double*>(d.p[1]), 1, sv, nullptr, msv, bz,
                               sk);
      }
      if (rc != AS_OK) return rc;
      if (sk != s) {
        if ((e = hipEventRecord(pool.ev[k], sk)) != hipSuccess || (e = hipStreamWaitEvent(s, pool.ev[k], 0)) != hipSuccess)
          return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
      }
      if (count) {
        count->launches += 1;
        count->jobs += Pk;
      }
    }
    served.resize(P);
    ms.resize((size_t)P * M);
    busy.resize(gtotal);
    e = hipMemcpyAsync(served.data(), d.p[4], (size_t)P * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(ms.data(), d.p[5], (size_t)P * M * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipMemcpyAsync(busy.data(), d.p[6], gtotal * 8, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(AS_E_HIP, "search: step %d: %s", step, hipGetErrorString(e));
    for (int q = 0; q < P; ++q) {
      const int r = live[q];
      const Problem& pr = probs[r];
      Result& out = res[r];
      Sel& sel = cur[r];
      if (served[q] > out.best_served) {
        out.best_served = served[q];
        out.best_mask = sel.mask;
      }
      if (max_steps >= 0 && out.steps >= max_steps) {
        active[r] = 0;
        continue;
      }
      // the model with the most unserved requests among those that still fit somewhere
      int mstar = -1;
      int64_t umax = 0;
      for (int m = 0; m < M; ++m) {
        if (!((pr.models >> m) & 1u)) continue;
        bool any = false;
        for (int g = 0; g < pr.G && !any; ++g) any = fits(pr, sel, w, m, g);
        if (!any) continue;
        const int64_t u = (int64_t)n_req[m] - ms[(size_t)q * M + m];
        if (mstar < 0 || u > umax) {
          mstar = m;
          umax = u;
        }
      }
      if (mstar < 0) {
        active[r] = 0;
        continue;
      }
      int gstar = -1;
      for (int g = 0; g < pr.G; ++g)
        if (fits(pr, sel, w, mstar, g) && (gstar < 0 || busy[brow[q] + g] < busy[brow[q] + gstar]))
          gstar = g;
      sel.mask[mstar] |= 1ull << gstar;
      sel.used[gstar] += w[mstar];
      out.step_model.push_back(mstar);
      out.step_group.push_back(gstar);
      out.step_served.push_back(served[q]);
      out.step_parent.push_back(0);
      out.step_candidates.push_back(1);
      ++out.steps;
    }
  }
  return ok();
}

namespace {

// One problem from the C-ABI's host arrays (every model placeable).
int make_problem(int32_t G, const int32_t* group_cfg, const int64_t* group_mem_mib, int M, Problem& pr) {
  if (G < 1 || G > AS_MAX_GROUPS) return fail(AS_E_LIMITS, "search: n_groups=%d outside 1..%d", G, AS_MAX_GROUPS);
  if (!group_cfg || !group_mem_mib) return fail(AS_E_INVALID_ARG, "search: NULL group arrays");
  pr.G = G;
  pr.cfg.assign(group_cfg, group_cfg + G);
  pr.mem.assign(group_mem_mib, group_mem_mib + G);
  pr.models = M >= 64 ? ~0ull : ((1ull << M) - 1);
  return AS_OK;
}

int write_trajectory(const Result& r, int M, uint64_t* best_mask, int64_t* best_served, int32_t* step_model,
                     int32_t* step_group, int64_t* step_served, int32_t max_steps, int32_t* n_steps) {
  for (int m = 0; m < M; ++m) best_mask[m] = r.best_mask[m];
  *best_served = r.best_served;
  *n_steps = r.steps;
  for (int i = 0; i < r.steps && i < max_steps; ++i) {
    step_model[i] = r.step_model[i];
    step_group[i] = r.step_group[i];
    step_served[i] = r.step_served[i];
  }
  return ok();
}

int single_search(bool fast, int beam, const as_trace_t* trace, const as_models_t* models,
                  const int64_t* weight_mib, int32_t n_groups, const int32_t* group_cfg,
                  const int64_t* group_mem_mib, double slo_scale, uint64_t* best_mask, int64_t* best_served,
                  int32_t* step_model, int32_t* step_group, int64_t* step_served, int32_t max_steps,
                  int32_t* n_steps, hipStream_t s) {
  if (!models || !best_mask || !best_served || !n_steps) return fail(AS_E_INVALID_ARG, "search: NULL argument");
  if (max_steps < 0 || (max_steps > 0 && (!step_model || !step_group || !step_served)))
    return fail(AS_E_INVALID_ARG, "search: bad trajectory buffers");
  std::vector<Problem> probs(1);
  int rc = make_problem(n_groups, group_cfg, group_mem_mib, models->n_models, probs[0]);
  if (rc != AS_OK) return rc;
  std::vector<Result> res;
  rc = fast ? fast_search(trace, models, weight_mib, slo_scale, probs, res, -1, s)
            : beam_search(trace, models, weight_mib, slo_scale, beam, probs, res, -1, s);
  if (rc != AS_OK) return rc;
  return write_trajectory(res[0], models->n_models, best_mask, best_served, step_model, step_group,
                          step_served, max_steps, n_steps);
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
  return single_search(false, 1, trace, models, weight_mib, n_groups, group_cfg, group_mem_mib, slo_scale,
                       best_mask, best_served, step_model, step_group, step_served, max_steps, n_steps,
                       (hipStream_t)stream);
}

int as_beam_placement(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                      int32_t n_groups, const int32_t* group_cfg, const int64_t* group_mem_mib,
                      double slo_scale, int32_t beam, uint64_t* best_mask, int64_t* best_served,
                      int32_t* step_model, int32_t* step_group, int64_t* step_served, int32_t max_steps,
                      int32_t* n_steps, void* stream) {
  if (beam < 1) return fail(AS_E_INVALID_ARG, "beam=%d < 1", beam);
  return single_search(false, beam, trace, models, weight_mib, n_groups, group_cfg, group_mem_mib, slo_scale,
                       best_mask, best_served, step_model, step_group, step_served, max_steps, n_steps,
                       (hipStream_t)stream);
}

int as_fast_placement(const as_trace_t* trace, const as_models_t* models, const int64_t* weight_mib,
                      int32_t n_groups, const int32_t* group_cfg, const int64_t* group_mem_mib,
                      double slo_scale, uint64_t* best_mask, int64_t* best_served, int32_t* step_model,
                      int32_t* step_group, int64_t* step_served, int32_t max_steps, int32_t* n_steps,
                      void* stream) {
  return single_search(true, 1, trace, models, weight_mib, n_groups, group_cfg, group_mem_mib, slo_scale,
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
  std::vector<Problem> probs(n_partitions);
  int64_t off = 0;
  for (int p = 0; p < n_partitions; ++p) {
    const int rc = make_problem(part_groups[p], part_cfg + off, part_mem_mib + off, M, probs[p]);
    if (rc != AS_OK) return rc;
    off += part_groups[p];
  }
  std::vector<Result> res;
  const int rc = beam_search(trace, models, weight_mib, slo_scale, 1, probs, res, -1, (hipStream_t)stream);
  if (rc != AS_OK) return rc;
  int32_t best_p = -1;
  int64_t best_s = -1;
  for (int p = 0; p < n_partitions; ++p) {
    part_served[p] = res[p].best_served;
    if (res[p].best_served > best_s) {
      best_s = res[p].best_served;
      best_p = p;
    }
  }
  for (int m = 0; m < M; ++m) best_mask[m] = res[best_p].best_mask[m];
  *best_partition = best_p;
  *best_served = best_s;
  return ok();
}

}  // extern "C"
