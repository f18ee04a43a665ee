// Dynamic batching (Sec. 6.5) on the batched simulator: an arriving request
// runs at once on an available group hosting its model, otherwise it waits in
// a per-model queue; a group that becomes idle runs the largest batch of one
// hosted model's queued requests that still meets the SLO; a batch's latency
// grows linearly with its size.  The exact rules are those of
// alpaserve_sim.h's as_simulate_batched.
//
// Layout: one job per wavefront (one wavefront per workgroup), lane g = group
// g: a group's stage free times live in its lane's registers.  The job's
// per-model FIFO queues are ring buffers of trace indices in LDS, with their
// head/tail counters beside them; which models have queued requests is a
// wave-uniform 64-bit mask.  Every decision is wave-uniform: the next idle
// group is a butterfly min over the lanes with queued work, the model with the
// oldest queued head a scalar loop over the group's models, and the batch
// size a loop over b in which every lane runs its own stage chain and the
// chosen lane's finish is read back.  The arithmetic is the definition's
// (no FMA, v_max_f64, the batch factor rounded once), so served counts,
// digests and finish times are bit-identical to a sequential evaluation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_kernel.hpp"

namespace as_dev {
namespace {

struct BatchArgs {
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
  double* out_finish;
  uint32_t* overflow;  // set when a queue would exceed its capacity
  double beta;
  int32_t M, C, smax_in, G, K, J, max_batch, qcap, n_finish;
  int32_t cfg_stages[AS_MAX_CONFIGS];
  int32_t finish_jobs[AS_MAX_FINISH];
};

// SplitMix64 finaliser (the batched digest's per-request term).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

__device__ __forceinline__ double rl_f64(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
  return __hiloint2double(hi, lo);
}

constexpr int kBatchChunk = 512;  // trace requests staged per LDS refill

// LDS of one job: queue entries (trace index and deadline) [M][qcap], heads
// and tails [M], SLOs [M], stage-latency table [M][Cp][SMAX], trace chunk.
__host__ __device__ constexpr size_t batch_lds_bytes(int M, int Cp, int SMAX, int qcap) {
  return (size_t)M * qcap * 12 + (size_t)M * 8 + (size_t)M * 8 + (size_t)M * Cp * SMAX * 8 +
         (size_t)kBatchChunk * 12;
}

// W: lanes reduced per job, the group count rounded up to a power of two (at
// least 16, so the reductions inside a 16-lane row are DPP only).
template <int W, int SMAX>
__global__ __launch_bounds__(64) void batch_kernel(const BatchArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1;
  while (cp < a.C) cp <<= 1;
  double* sL = reinterpret_cast<double*>(smem);                   // [M][cp][SMAX]
  double* sSlo = sL + (size_t)a.M * cp * SMAX;                    // [M]
  double* sQd = sSlo + a.M;                                       // [M][qcap] deadlines
  double* sT = sQd + (size_t)a.M * a.qcap;                        // chunk times
  uint32_t* sHead = reinterpret_cast<uint32_t*>(sT + kBatchChunk);  // [M]
  uint32_t* sTail = sHead + a.M;                                  // [M]
  uint32_t* sQi = sTail + a.M;                                    // [M][qcap] trace indices
  int32_t* sM = reinterpret_cast<int32_t*>(sQi + (size_t)a.M * a.qcap);  // chunk models
  const int lane = threadIdx.x;
  const int64_t job = blockIdx.x;
  const int p = (int)(job / a.K);
  const double sigma = a.slo_scale[job % a.K];
  const uint32_t qmask = (uint32_t)a.qcap - 1u;

  int cfg = lane < a.G ? a.group_cfg[(int64_t)p * a.G + lane] : -1;
  if (cfg >= a.C || cfg < 0) cfg = -1;
  uint64_t hostbits = 0;  // bit m: this lane's group hosts model m
  if (cfg >= 0) {
    const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
    for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> lane) & 1u) << m;
  }
  const int nL = a.M * cp * SMAX;
  for (int idx = lane; idx < nL; idx += 64) {
    const int s = idx % SMAX;
    const int mc = idx / SMAX;
    const int c = mc % cp;
    const int m = mc / cp;
    sL[idx] = (c < a.C && s < a.cfg_stages[c]) ? a.stage_lat[((int64_t)m * a.C + c) * a.smax_in + s] : 0.0;
  }
  for (int m = lane; m < a.M; m += 64) {
    sSlo[m] = sigma * a.d_single[m];
    sHead[m] = 0;
    sTail[m] = 0;
  }
  int frow = -1;
  for (int f = 0; f < a.n_finish; ++f)
    if (a.finish_jobs[f] == job) frow = f;
  double* frowp = frow >= 0 ? a.out_finish + (int64_t)frow * a.n : nullptr;
  __syncthreads();

  const double* lbase = sL + (size_t)(cfg < 0 ? 0 : cfg) * SMAX;  // + m * cp * SMAX
  double F[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) F[s] = 0.0;
  uint64_t nonempty = 0;  // bit m: model m has queued requests (wave-uniform)
  uint64_t h = 0, fin_sum = 0;
  int64_t served = 0;
  const double kInf = __builtin_inf();

  // every lane's chain for a batch of b requests of model m started at x;
  // returns the last stage's finish, fs[] its stage finishes
  auto chain = [&](int m, int b, double x, double (&fs)[SMAX]) {
    const double fac = 1.0 + a.beta * (double)(b - 1);
    const double* L = lbase + (size_t)m * cp * SMAX;
    double f = x;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
      fs[s] = vmax(f, F[s]) + L[s] * fac;
      f = fs[s];
    }
    return f;
  };
  // smallest key over the job's lanes (lane 0's segment), wave-uniform
  auto wave_min = [&](double key) {
    const double v = seg_min<W>(key);
    return rl_f64(v, 0);
  };

  for (int64_t base = 0; base <= a.n; base += kBatchChunk) {
    const int cnt = (int)((a.n - base) < kBatchChunk ? (a.n - base) : kBatchChunk);
    __syncthreads();
    for (int e = lane; e < cnt; e += 64) {
      sT[e] = a.t[base + e];
      sM[e] = a.model[base + e];
    }
    __syncthreads();
    // cnt requests of this chunk, then (after the last one) the final drain
    const int steps = base + kBatchChunk > a.n ? cnt + 1 : cnt;
    for (int e = 0; e < steps; ++e) {
      const bool last = e == cnt;
      const int64_t i = base + e;
      const double horizon = last ? 0.0 : sT[e];
      // idle events up to the arrival (all remaining ones after the last)
      for (;;) {
        const bool work = cfg >= 0 && (hostbits & nonempty) != 0;
        const double key = work ? F[0] : kInf;
        const double mn = wave_min(key);
        const uint64_t wm = __builtin_amdgcn_ballot_w64(work && key == mn);
        if (wm == 0) break;
        if (!last && !(mn <= horizon)) break;
        const int g = __builtin_ctzll(wm);
        const uint64_t ghost = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(hostbits >> 32), g) << 32) |
                               (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)hostbits, g);
        for (;;) {
          uint64_t cand = ghost & nonempty;
          if (cand == 0) break;  // nothing left for this group: it stays idle
          int mc = -1;
          uint32_t hidx = 0;
          while (cand) {
            const int m = __builtin_ctzll(cand);
            cand &= cand - 1;
            const uint32_t r = sQi[(size_t)m * a.qcap + (sHead[m] & qmask)];
            if (mc < 0 || r < hidx) {
              mc = m;
              hidx = r;
            }
          }
          const uint32_t h0 = sHead[mc];
          const double dl = sQd[(size_t)mc * a.qcap + (h0 & qmask)];
          const uint32_t avail = sTail[mc] - h0;
          const int bmax = (int)(avail < (uint32_t)a.max_batch ? avail : (uint32_t)a.max_batch);
          int b = 0;
          double fin = 0.0;
          double fs[SMAX];
          for (int bb = 1; bb <= bmax; ++bb) {
            double fsb[SMAX];
            const double fl = rl_f64(chain(mc, bb, mn, fsb), g);
            if (fl > dl) break;
            b = bb;
            fin = fl;
#pragma unroll
            for (int s = 0; s < SMAX; ++s) fs[s] = fsb[s];
          }
          if (b == 0) {
            // the head cannot meet its deadline: dropped (its output stays -1)
            __syncthreads();
            if (lane == 0) sHead[mc] = h0 + 1;
            __syncthreads();
            if (h0 + 1 == sTail[mc]) nonempty &= ~(1ull << mc);
            continue;
          }
          if (lane == g) {
#pragma unroll
            for (int s = 0; s < SMAX; ++s) F[s] = fs[s];
          }
          for (int k = 0; k < b; ++k) {
            const uint32_t r = sQi[(size_t)mc * a.qcap + ((h0 + k) & qmask)];
            h += mix64(r);
            fin_sum += (uint64_t)__double_as_longlong(fin);
            if (frowp && lane == 0) frowp[r] = fin;
          }
          served += b;
          __syncthreads();
          if (lane == 0) sHead[mc] = h0 + b;
          __syncthreads();
          if (h0 + b == sTail[mc]) nonempty &= ~(1ull << mc);
          break;
        }
      }
      if (last) break;
      // the arrival
      const double ti = horizon;
      const int m0 = sM[e];
      const bool mok = (unsigned)m0 < (unsigned)a.M;
      const int m = mok ? m0 : 0;
      const bool hosted = mok && cfg >= 0 && ((hostbits >> m) & 1u);
      if (__builtin_amdgcn_ballot_w64(hosted) == 0) continue;  // no group hosts it: a miss
      const bool avail = hosted && F[0] <= ti;
      const uint64_t av = __builtin_amdgcn_ballot_w64(avail);
      if (av != 0) {
        const double key = avail ? F[0] : kInf;
        const double mn = wave_min(key);
        const int ga = __builtin_ctzll(__builtin_amdgcn_ballot_w64(avail && key == mn));
        double fs[SMAX];
        const double fl = rl_f64(chain(m, 1, ti, fs), ga);
        if (!(fl > ti + sSlo[m])) {
          if (lane == ga) {
#pragma unroll
            for (int s = 0; s < SMAX; ++s) F[s] = fs[s];
          }
          served += 1;
          h += mix64((uint64_t)i);
          fin_sum += (uint64_t)__double_as_longlong(fl);
          if (frowp && lane == 0) frowp[i] = fl;
        }
      } else {
        // Queue heads of model m that can no longer be served are dropped
        // now rather than when a group reaches them: any batch that could
        // still serve a queued request starts at or after ti, so it finishes
        // no earlier than the chain from ti through a hosting group's stages
        // with single-request latencies, free times ignored (fp64 rounding
        // is monotone); a head whose deadline lies before the smallest such
        // bound is dropped by the definition too, and dropping it earlier
        // changes no other decision.  This keeps each queue to the requests
        // that are still servable.
        double lbv = ti;
        {
          const double* L = lbase + (size_t)m * cp * SMAX;
#pragma unroll
          for (int s = 0; s < SMAX; ++s) lbv = lbv + L[s];
        }
        const double lb = wave_min(hosted ? lbv : kInf);
        uint32_t hd = sHead[m];
        const uint32_t tl = sTail[m];
        while (hd != tl && sQd[(size_t)m * a.qcap + (hd & qmask)] < lb) ++hd;
        if (tl - hd == (uint32_t)a.qcap) {
          if (lane == 0) atomicOr(a.overflow, 1u);  // queue full: the request is lost
        } else {
          __syncthreads();
          if (lane == 0) {
            sHead[m] = hd;
            sQi[(size_t)m * a.qcap + (tl & qmask)] = (uint32_t)i;
            sQd[(size_t)m * a.qcap + (tl & qmask)] = ti + sSlo[m];
            sTail[m] = tl + 1;
          }
          __syncthreads();
          nonempty |= 1ull << m;
        }
      }
    }
  }
  if (lane == 0) {
    a.out_served[job] = served;
    if (a.out_digest) {
      a.out_digest[2 * job] = h;
      a.out_digest[2 * job + 1] = fin_sum;
    }
  }
}

// Per-request output rows before a batched launch: -2 for requests whose model
// the job's placement does not host, -1 for the others (served ones are
// overwritten by the kernel).
__global__ void fill_batch_rows(const BatchArgs a) {
  const int64_t total = (int64_t)a.n_finish * a.n;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
       x += (int64_t)gridDim.x * blockDim.x) {
    const int f = (int)(x / a.n);
    const int64_t i = x % a.n;
    const int p = a.finish_jobs[f] / a.K;
    const int32_t m = a.model[i];
    const bool hosted = (unsigned)m < (unsigned)a.M && a.host_mask[(int64_t)p * a.M + m] != 0;
    a.out_finish[x] = hosted ? -1.0 : -2.0;
  }
}

}  // namespace
}  // namespace as_dev

using namespace as_host;

extern "C" int as_simulate_batched(const as_trace_t* trace, const as_models_t* models,
                                   const as_placements_t* placements, const double* slo_scale,
                                   int32_t n_scales, int32_t max_batch, double beta, int32_t queue_cap,
                                   int64_t* out_served, uint64_t* out_digest, const int32_t* finish_jobs,
                                   int32_t n_finish, double* out_finish, void* stream) {
  KArgs ka;
  std::memset(&ka, 0, sizeof ka);
  if (!trace) return fail(AS_E_INVALID_ARG, "trace must not be NULL");
  if (trace->n < 0) return fail(AS_E_INVALID_ARG, "trace n=%lld < 0", (long long)trace->n);
  if (trace->n > 0 && (!trace->t || !trace->model))
    return fail(AS_E_INVALID_ARG, "trace arrays must not be NULL");
  if (trace->n > 0xFFFFFFFFLL) return fail(AS_E_LIMITS, "batched: trace of %lld requests > 2^32 - 1", (long long)trace->n);
  int W = 1, smax = 1;
  int rc = check_common(models, placements, ka, W, smax);
  if (rc != AS_OK) return rc;
  if (n_scales < 0) return fail(AS_E_INVALID_ARG, "n_scales=%d < 0", n_scales);
  if (max_batch < 1) return fail(AS_E_INVALID_ARG, "max_batch=%d < 1", max_batch);
  if (!(beta >= 0.0) || !(beta <= 1.7976931348623157e308))
    return fail(AS_E_INVALID_ARG, "beta must be finite and >= 0");
  if (queue_cap < 1 || (queue_cap & (queue_cap - 1)) != 0 || queue_cap > (1 << 20))
    return fail(AS_E_INVALID_ARG, "queue_cap=%d must be a power of two in 1..2^20", queue_cap);
  const int64_t J = (int64_t)placements->n_placements * n_scales;
  if (J > 0x7FFFFFFFLL) return fail(AS_E_LIMITS, "placements x scales = %lld jobs > 2^31-1", (long long)J);
  if (J > 0 && (!slo_scale || !out_served))
    return fail(AS_E_INVALID_ARG, "slo_scale and out_served must not be NULL");
  if (n_finish < 0 || n_finish > AS_MAX_FINISH)
    return fail(n_finish < 0 ? AS_E_INVALID_ARG : AS_E_LIMITS, "n_finish=%d outside 0..%d", n_finish, AS_MAX_FINISH);
  if (n_finish > 0 && (!finish_jobs || !out_finish))
    return fail(AS_E_INVALID_ARG, "finish_jobs and out_finish must not be NULL when n_finish > 0");
  as_dev::BatchArgs a;
  std::memset(&a, 0, sizeof a);
  for (int f = 0; f < n_finish; ++f) {
    if (finish_jobs[f] < 0 || finish_jobs[f] >= J)
      return fail(AS_E_INVALID_ARG, "finish_jobs[%d]=%d outside [0, %lld)", f, finish_jobs[f], (long long)J);
    for (int q = 0; q < f; ++q)
      if (finish_jobs[q] == finish_jobs[f]) return fail(AS_E_INVALID_ARG, "finish_jobs[%d] repeats job %d", f, finish_jobs[f]);
    a.finish_jobs[f] = finish_jobs[f];
  }
  const size_t lds = as_dev::batch_lds_bytes(ka.M, pow2ceil(ka.C), smax, queue_cap);
  if (lds > shared_lds_limit())
    return fail(AS_E_LIMITS, "batched: queues and tables need %zu bytes of LDS (> %zu); lower queue_cap", lds,
                shared_lds_limit());
  if (J == 0) return ok();
  hipStream_t s = (hipStream_t)stream;
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
  a.out_finish = out_finish;
  a.beta = beta;
  a.M = ka.M;
  a.C = ka.C;
  a.smax_in = ka.smax_in;
  a.G = ka.G;
  a.K = n_scales;
  a.J = (int32_t)J;
  a.max_batch = max_batch;
  a.qcap = queue_cap;
  a.n_finish = n_finish;
  for (int c = 0; c < AS_MAX_CONFIGS; ++c) a.cfg_stages[c] = ka.cfg_stages[c];
  uint32_t* d_flag = nullptr;
  hipError_t e = hipMallocAsync((void**)&d_flag, sizeof(uint32_t), s);
  if (e != hipSuccess) return fail(AS_E_NOMEM, "hipMallocAsync: %s", hipGetErrorString(e));
  a.overflow = d_flag;
  e = hipMemsetAsync(d_flag, 0, sizeof(uint32_t), s);
  if (e == hipSuccess && n_finish > 0 && a.n > 0) {
    const int64_t cells = (int64_t)n_finish * a.n;
    const int blocks = (int)std::min<int64_t>((cells + 255) / 256, 8192);
    hipLaunchKernelGGL(as_dev::fill_batch_rows, dim3(blocks), dim3(256), 0, s, a);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    const int W = std::max(16, pow2ceil(a.G));
    const dim3 grid((unsigned)J), block(64);
#define AS_BATCH_LAUNCH(WW)                                                                         \
  switch (smax) {                                                                                   \
    case 1: hipLaunchKernelGGL((as_dev::batch_kernel<WW, 1>), grid, block, lds, s, a); break;       \
    case 2: hipLaunchKernelGGL((as_dev::batch_kernel<WW, 2>), grid, block, lds, s, a); break;       \
    case 4: hipLaunchKernelGGL((as_dev::batch_kernel<WW, 4>), grid, block, lds, s, a); break;       \
    default: hipLaunchKernelGGL((as_dev::batch_kernel<WW, 8>), grid, block, lds, s, a); break;      \
  }
    if (W == 16) {
      AS_BATCH_LAUNCH(16)
    } else if (W == 32) {
      AS_BATCH_LAUNCH(32)
    } else {
      AS_BATCH_LAUNCH(64)
    }
#undef AS_BATCH_LAUNCH
    e = hipGetLastError();
  }
  uint32_t flag = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&flag, d_flag, sizeof flag, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  const hipError_t ef = hipFreeAsync(d_flag, s);
  if (e == hipSuccess) e = ef;
  if (e != hipSuccess) return fail(AS_E_HIP, "batched: %s", hipGetErrorString(e));
  if (flag) return fail(AS_E_LIMITS, "batched: a model queue exceeded queue_cap=%d; results are incomplete", queue_cap);
  return ok();
}
