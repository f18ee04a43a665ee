// Per-job statistics of the serving simulation for the fast placement
// heuristic of Sec. 4.2 (simulate the current selection once, then place the
// model with the most unserved requests on the available group with the
// lowest utilization): besides the served count and digest, every job reports
// the served requests of each model and the busy time of each group.
//
// Layout: one job per wavefront, lane g = group g (up to 64 groups), so a
// group's stage free times and its busy-time sum live in one lane's
// registers; four wavefronts per workgroup share the trace, which is staged
// through LDS in coalesced chunks.  Per request (t, m) of a job:
//   dispatch (Sec. 4.3)  the hosting lane with the smallest stage-0 free time,
//                        the lowest on ties (f64 butterfly min, ballot);
//   projection (3.4)     every lane runs its group's stage chain
//                        f_s = max(f_{s-1}, F[s]) + L[m][c][s];
//   admission (4.3, 3.2) the target accepts iff f_{S-1} <= t + scale*d[m];
//   statistics           on accept the target lane adds the model's slowest
//                        stage latency for its configuration (the stage that
//                        bounds a pipeline's throughput, Sec. 3.4) to its busy
//                        time, in trace order, and bumps the model's served
//                        counter (LDS, one writer per request).
// The operations and their order are the definition's (no FMA, v_max_f64), so
// served counts, digests and busy times are bit-identical to a sequential
// IEEE evaluation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_kernel.hpp"

namespace as_dev {
namespace {

constexpr int kStatChunk = 1024;  // requests per LDS chunk

struct StatsArgs {
  const double* t;
  const int32_t* model;
  int64_t n;
  const double* d_single;
  const double* stage_lat;
  const int32_t* group_cfg;
  const uint64_t* host_mask;
  const double* slo_scale;
  int64_t* out_served;
  uint64_t* out_digest;
  int64_t* out_model_served;
  double* out_group_busy;
  int32_t M, C, smax_in, G, K, J;
  int32_t cfg_stages[AS_MAX_CONFIGS];
};

// LDS: stage-latency table [M][Cp][SMAX] (zero-padded stages), d_single[M],
// the trace chunk and each wavefront's per-model served counters.
__host__ __device__ constexpr size_t stats_lds_bytes(int M, int Cp, int SMAX) {
  return (size_t)M * Cp * SMAX * 8 + (size_t)M * 8 + (size_t)kStatChunk * 12 + (size_t)kWaves * M * 4;
}

template <int SMAX>
__global__ __launch_bounds__(kThreads) void stats_kernel(const StatsArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1;
  while (cp < a.C) cp <<= 1;
  double* sL = reinterpret_cast<double*>(smem);      // [M][cp][SMAX]
  double* sD = sL + (size_t)a.M * cp * SMAX;         // [M]
  double* sT = sD + a.M;                             // chunk times
  int32_t* sM = reinterpret_cast<int32_t*>(sT + kStatChunk);
  uint32_t* sCnt = reinterpret_cast<uint32_t*>(sM + kStatChunk);  // [kWaves][M]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t job = (int64_t)blockIdx.x * kWaves + wave;
  const bool job_ok = job < a.J;
  int p = 0;
  double sigma = 0.0;
  if (job_ok) {
    p = (int)(job / a.K);
    sigma = a.slo_scale[job % a.K];
  }
  int cfg = -1;
  if (job_ok && lane < a.G) cfg = a.group_cfg[(int64_t)p * a.G + lane];
  if (cfg >= a.C || cfg < 0) cfg = -1;
  uint64_t hostbits = 0;  // bit m: this lane's group hosts model m
  if (cfg >= 0) {
    const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
    for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> lane) & 1u) << m;
  }
  const double* lrow = sL + (size_t)(cfg < 0 ? 0 : cfg) * SMAX;  // + m * cp * SMAX
  uint32_t* cnt = sCnt + (size_t)wave * a.M;

  const int nL = a.M * cp * SMAX;
  for (int idx = tid; idx < nL; idx += kThreads) {
    const int s = idx % SMAX;
    const int mc = idx / SMAX;
    const int c = mc % cp;
    const int m = mc / cp;
    sL[idx] = (c < a.C && s < a.cfg_stages[c]) ? a.stage_lat[((int64_t)m * a.C + c) * a.smax_in + s] : 0.0;
  }
  for (int m = tid; m < a.M; m += kThreads) sD[m] = a.d_single[m];
  for (int m = lane; m < a.M; m += 64) cnt[m] = 0;

  double F[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) F[s] = 0.0;
  double busy = 0.0;
  uint64_t fin_sum = 0, h = 0, word = 0;
  int64_t served = 0;
  const double kInf = __builtin_inf();

  for (int64_t base = 0; base < a.n; base += kStatChunk) {
    const int cc = (int)((a.n - base) < kStatChunk ? (a.n - base) : kStatChunk);
    __syncthreads();
    for (int e = tid; e < cc; e += kThreads) {
      sT[e] = a.t[base + e];
      sM[e] = a.model[base + e];
    }
    __syncthreads();
    for (int e = 0; e < cc; ++e) {
      const int64_t i = base + e;
      const double ti = sT[e];
      // a model id outside [0, M) (invalid device data) is a request no group hosts
      const int m0 = sM[e];
      const bool mok = (unsigned)m0 < (unsigned)a.M;
      const int m = mok ? m0 : 0;
      const bool hosted = mok && ((hostbits >> m) & 1u);
      const double key = hosted ? F[0] : kInf;
      const double mn = seg_min<64>(key);
      const uint64_t eqm = __builtin_amdgcn_ballot_w64(hosted && key == mn);
      if (eqm != 0) {
        const int target = __builtin_ctzll(eqm);
        const double* L = lrow + (size_t)m * cp * SMAX;
        double fs[SMAX];
        double f = ti, slowest = 0.0;
#pragma unroll
        for (int s = 0; s < SMAX; ++s) {
          fs[s] = vmax(f, F[s]) + L[s];
          f = fs[s];
          slowest = vmax(slowest, L[s]);
        }
        const double deadline = ti + sigma * sD[m];
        const bool acc = lane == target && !(f > deadline);
        if (acc) {
#pragma unroll
          for (int s = 0; s < SMAX; ++s) F[s] = fs[s];
          busy += slowest;
          fin_sum += (uint64_t)__double_as_longlong(f);
          cnt[m] += 1;
        }
        if (__builtin_amdgcn_ballot_w64(acc) != 0) {
          word |= 1ull << (i & 63);
          ++served;
        }
      }
      if ((i & 63) == 63 || i == a.n - 1) {
        h = (h ^ word) * kHashMul;
        word = 0;
      }
    }
  }
  const uint64_t fsum = seg_sum_u64<64>(fin_sum);
  __syncthreads();
  if (job_ok) {
    if (lane == 0) {
      a.out_served[job] = served;
      if (a.out_digest) {
        a.out_digest[2 * job] = h;
        a.out_digest[2 * job + 1] = fsum;
      }
    }
    if (a.out_group_busy && lane < a.G) a.out_group_busy[job * a.G + lane] = busy;
    if (a.out_model_served)
      for (int m = lane; m < a.M; m += 64) a.out_model_served[job * a.M + m] = (int64_t)cnt[m];
  }
}

}  // namespace
}  // namespace as_dev

using namespace as_host;

extern "C" int as_simulate_stats(const as_trace_t* trace, const as_models_t* models,
                                 const as_placements_t* placements, const double* slo_scale,
                                 int32_t n_scales, int64_t* out_served, uint64_t* out_digest,
                                 int64_t* out_model_served, double* out_group_busy, void* stream) {
  KArgs ka;
  std::memset(&ka, 0, sizeof ka);
  if (!trace) return fail(AS_E_INVALID_ARG, "trace must not be NULL");
  if (trace->n < 0) return fail(AS_E_INVALID_ARG, "trace n=%lld < 0", (long long)trace->n);
  if (trace->n > 0 && (!trace->t || !trace->model))
    return fail(AS_E_INVALID_ARG, "trace arrays must not be NULL");
  int W = 1, smax = 1;
  int rc = check_common(models, placements, ka, W, smax);
  if (rc != AS_OK) return rc;
  if (n_scales < 0) return fail(AS_E_INVALID_ARG, "n_scales=%d < 0", n_scales);
  const int64_t J = (int64_t)placements->n_placements * n_scales;
  if (J > 0x7FFFFFFFLL) return fail(AS_E_LIMITS, "placements x scales = %lld jobs > 2^31-1", (long long)J);
  if (J > 0 && (!slo_scale || !out_served))
    return fail(AS_E_INVALID_ARG, "slo_scale and out_served must not be NULL");
  if (J == 0) return ok();
  hipStream_t s = (hipStream_t)stream;
  if (n_scales == 1) {
    // one scale: the tuned shared-trace kernel with its statistics outputs
    ka.t = trace->t;
    ka.model = trace->model;
    ka.n = trace->n;
    ka.slo_scale = slo_scale;
    ka.K = 1;
    ka.J = (int32_t)J;
    ka.P = placements->n_placements;
    ka.out_served = out_served;
    ka.out_digest = out_digest;
    ka.out_model_served = out_model_served;
    ka.out_group_busy = out_group_busy;
    ka.n_finish = 0;
    const int r = run_shared_stats(ka, smax, s);
    if (r != AS_E_LIMITS) return r;
  }
  as_dev::StatsArgs a;
  std::memset(&a, 0, sizeof a);
  a.t = trace->t;
  a.model = trace->model;
  a.n = trace->n;
  a.d_single = ka.d_single;
  a.stage_lat = ka.stage_lat;
  a.group_cfg = ka.group_cfg;
  a.host_mask = ka.host_mask;
  a.slo_scale = slo_scale;
  a.out_served = out_served;
  a.out_digest = out_digest;
  a.out_model_served = out_model_served;
  a.out_group_busy = out_group_busy;
  a.M = ka.M;
  a.C = ka.C;
  a.smax_in = ka.smax_in;
  a.G = ka.G;
  a.K = n_scales;
  a.J = (int32_t)J;
  for (int c = 0; c < AS_MAX_CONFIGS; ++c) a.cfg_stages[c] = ka.cfg_stages[c];
  const size_t lds = as_dev::stats_lds_bytes(a.M, pow2ceil(a.C), smax);
  if (lds > shared_lds_limit())
    return fail(AS_E_LIMITS, "stage-latency table (%d models x %d configs x %d stages) does not fit in LDS",
                a.M, a.C, smax);
  const int grid = (int)((J + as_dev::kWaves - 1) / as_dev::kWaves);
  switch (smax) {
    case 1: hipLaunchKernelGGL(as_dev::stats_kernel<1>, dim3(grid), dim3(as_dev::kThreads), lds, s, a); break;
    case 2: hipLaunchKernelGGL(as_dev::stats_kernel<2>, dim3(grid), dim3(as_dev::kThreads), lds, s, a); break;
    case 4: hipLaunchKernelGGL(as_dev::stats_kernel<4>, dim3(grid), dim3(as_dev::kThreads), lds, s, a); break;
    default: hipLaunchKernelGGL(as_dev::stats_kernel<8>, dim3(grid), dim3(as_dev::kThreads), lds, s, a); break;
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}
