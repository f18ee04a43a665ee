// Batched serving-simulator kernel for gfx950 (CDNA4, wave64).
//
// One job = one (trace, placement, SLO scale).  Its state is the free time
// F[g][s] of every stage s of every group g (Sec. 3.4: each pipeline stage is
// a single server).  Layout: a job owns W consecutive lanes of a wavefront,
// lane r of the job holds group r (W = next power of two >= the group count);
// the stage free times of that group live in the lane's registers.  One
// wavefront therefore carries 64 / W jobs.
//
// Per request (t, m) the lanes of a job:
//   1. dispatch (Sec. 4.3): key = F[g][0] if the lane's group hosts m, else +inf;
//      a butterfly min over the job's W lanes (DPP inside a 16-lane row, lane
//      shuffles across rows), then the lowest lane holding the minimum wins
//      (wavefront ballot restricted to the job's lanes below the caller);
//   2. project (Sec. 3.4): every lane runs its own group's stage chain
//      f_s = max(f_{s-1}, F[s]) + L[m][c][s]; only the chosen lane's result is used;
//   3. admit (Sec. 4.3, Sec. 3.2): the chosen lane accepts iff f_{S-1} <= t + slo_m
//      and then commits F[s] := f_s;
//   4. count: served, accept bits and the finish-time bit sum accumulate per
//      lane and are combined over the job's lanes every 64 requests / at the end.
//
// Arrivals are staged through LDS in chunks loaded with coalesced reads by the
// whole workgroup; a shared trace is read once per workgroup per chunk, every
// wavefront then reads the same LDS words (broadcast).  Segmented traces (one
// per job) are staged per job slot.
//
// Exactness: max and min are emitted as v_max_f64 / v_min_f64 (exact; no NaN
// or -0 ever reaches them), additions are single IEEE v_add_f64, no FMA
// (-ffp-contract=off), and the operation order is the definition's, so every
// finish time is bit-identical to a sequential IEEE evaluation.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alpaserve_sim.h"

namespace as_dev {

constexpr int kWaves = 4;                 // wavefronts per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kChunk = 2048;              // shared-trace requests per LDS chunk
// per-job requests per LDS chunk for segmented traces, sized so that all
// kSlots job slots of a workgroup fit in about 48 KiB
template <int kSlots>
constexpr int seg_chunk() {
  return (4096 / kSlots) > 128 ? 128 : ((4096 / kSlots) < 16 ? 16 : 4096 / kSlots);
}
constexpr uint64_t kHashMul = 0x9E3779B97F4A7C15ULL;

struct KArgs {
  const double* t;
  const int32_t* model;
  int64_t n;                 // shared trace length
  const int64_t* seg_off;    // segmented: [n_segments + 1]
  const as_job_t* jobs;      // segmented: [J]
  const double* d_single;
  const double* stage_lat;
  const int32_t* group_cfg;
  const uint64_t* host_mask;
  const double* slo_scale;   // shared: [K]
  int64_t* out_served;
  double* out_attain;
  uint64_t* out_digest;
  double* out_finish;
  int64_t finish_stride;
  int32_t M, C, smax_in, G, K, J, n_finish;
  int32_t P, n_segments;
  int32_t cfg_stages[AS_MAX_CONFIGS];
  int32_t finish_jobs[AS_MAX_FINISH];
};

__device__ __forceinline__ double vmax(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

__device__ __forceinline__ double vmin(double a, double b) {
  double r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// DPP controls: quad_perm [1,0,3,2] (lane ^ 1), quad_perm [2,3,0,1] (lane ^ 2),
// row_half_mirror (i <-> 7 - i within 8 lanes), row_mirror (i <-> 15 - i
// within 16 lanes).  Applied in this order each doubles the span reduced.
constexpr int kXor1 = 0xB1, kXor2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140;

// Min over each aligned group of W lanes, result in every lane of the group.
template <int W>
__device__ __forceinline__ double seg_min(double v) {
  if constexpr (W >= 2) v = vmin(v, dpp_f64<kXor1>(v));
  if constexpr (W >= 4) v = vmin(v, dpp_f64<kXor2>(v));
  if constexpr (W >= 8) v = vmin(v, dpp_f64<kHalfMirror>(v));
  if constexpr (W >= 16) v = vmin(v, dpp_f64<kMirror>(v));
  if constexpr (W >= 32) v = vmin(v, __shfl_xor(v, 16));
  if constexpr (W >= 64) v = vmin(v, __shfl_xor(v, 32));
  return v;
}

template <int W>
__device__ __forceinline__ uint64_t seg_or(uint64_t v) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  if constexpr (W >= 2) { lo |= dpp_u32<kXor1>(lo); hi |= dpp_u32<kXor1>(hi); }
  if constexpr (W >= 4) { lo |= dpp_u32<kXor2>(lo); hi |= dpp_u32<kXor2>(hi); }
  if constexpr (W >= 8) { lo |= dpp_u32<kHalfMirror>(lo); hi |= dpp_u32<kHalfMirror>(hi); }
  if constexpr (W >= 16) { lo |= dpp_u32<kMirror>(lo); hi |= dpp_u32<kMirror>(hi); }
  if constexpr (W >= 32) { lo |= __shfl_xor(lo, 16); hi |= __shfl_xor(hi, 16); }
  if constexpr (W >= 64) { lo |= __shfl_xor(lo, 32); hi |= __shfl_xor(hi, 32); }
  return ((uint64_t)hi << 32) | lo;
}

template <int W>
__device__ __forceinline__ uint64_t seg_sum_u64(uint64_t v) {
#pragma unroll
  for (int d = 1; d < W; d <<= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, d);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), d);
    v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

// Per-lane simulation state of one group of one job.
template <int SMAX>
struct LaneState {
  double F[SMAX];
  uint64_t served, fin_sum, word, hash;
};

// The request loop over one LDS chunk.  FINISH: some job of this wavefront
// keeps per-request outputs.  Returns nothing; state is updated in place.
template <int W, int SMAX, bool FINISH>
__device__ __forceinline__ void run_chunk(LaneState<SMAX>& st, const double* __restrict__ cT,
                                          const int32_t* __restrict__ cM, int cnt, int64_t base,
                                          int64_t n_job, uint64_t hostbits, uint64_t below,
                                          const double* __restrict__ lrow_base, int lstride,
                                          const double* __restrict__ slo_row, int seg_lane,
                                          int frow, double* __restrict__ out_finish,
                                          int64_t finish_stride) {
  const double kInf = __builtin_inf();
  for (int e = 0; e < cnt; ++e) {
    const double ti = cT[e];
    const int mi = cM[e];
    const int64_t i = base + e;
    // 1. dispatch
    const bool hosted = (hostbits >> mi) & 1u;
    const double key = hosted ? st.F[0] : kInf;
    const double mn = seg_min<W>(key);
    const bool eq = hosted && key == mn;
    const uint64_t ball = __ballot(eq);
    const bool chosen = eq && ((ball & below) == 0);
    // 2. projection through this lane's stage chain
    const double* L = lrow_base + mi * lstride;
    double fs[SMAX];
    double f = ti;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
      fs[s] = vmax(f, st.F[s]) + L[s];
      f = fs[s];
    }
    // 3. admission
    const double deadline = ti + slo_row[mi];
    const bool acc = chosen && !(f > deadline);
    if (acc) {
#pragma unroll
      for (int s = 0; s < SMAX; ++s) st.F[s] = fs[s];
      st.served += 1;
      st.fin_sum += (uint64_t)__double_as_longlong(f);
      st.word |= (uint64_t)1 << (i & 63);
    }
    if constexpr (FINISH) {
      if (frow >= 0 && i < finish_stride) {
        double* dst = out_finish + (int64_t)frow * finish_stride + i;
        if (chosen) *dst = acc ? f : -1.0;
        else if (mn == kInf && seg_lane == 0) *dst = -2.0;
      }
    }
    // 4. fold the accept word of the job every 64 requests and at its end
    if ((i & 63) == 63 || i == n_job - 1) {
      const uint64_t w = seg_or<W>(st.word);
      st.hash = (st.hash ^ w) * kHashMul;
      st.word = 0;
    }
  }
}

template <int W, int SMAX, bool SEG>
__global__ __launch_bounds__(kThreads) void sim_kernel(const KArgs a) {
  constexpr int JW = 64 / W;                 // jobs per wavefront
  constexpr int kSlots = JW * kWaves;        // jobs per workgroup
  extern __shared__ __align__(16) unsigned char smem[];
  double* sL = reinterpret_cast<double*>(smem);                      // [M][C][SMAX]
  double* sSlo = sL + (size_t)a.M * a.C * SMAX;                      // [kSlots][M]
  double* sT = sSlo + (size_t)kSlots * a.M;                          // chunk times
  constexpr int CH = SEG ? seg_chunk<kSlots>() : kChunk;
  int32_t* sM = reinterpret_cast<int32_t*>(sT + (SEG ? kSlots * CH : kChunk));
  __shared__ unsigned long long s_nmax;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int seg_lane = lane & (W - 1);
  const int slot = wave * JW + lane / W;
  const int64_t job = (int64_t)blockIdx.x * kSlots + slot;
  bool job_ok = job < a.J;

  int p = 0;
  double sigma = 0.0;
  int64_t seg_begin = 0, n_job = a.n;
  if (job_ok) {
    if constexpr (SEG) {
      // job records are device data: a record naming a missing placement or
      // segment makes an empty job; segment bounds are clamped to the
      // concatenated trace [0, seg_off[n_segments])
      const as_job_t jb = a.jobs[job];
      p = jb.placement;
      sigma = jb.slo_scale;
      if (p < 0 || p >= a.P || jb.segment < 0 || jb.segment >= a.n_segments) {
        p = 0;
        n_job = 0;
      } else {
        const int64_t total = a.seg_off[a.n_segments];
        int64_t b = a.seg_off[jb.segment], e = a.seg_off[jb.segment + 1];
        b = b < 0 ? 0 : (b > total ? total : b);
        e = e < b ? b : (e > total ? total : e);
        seg_begin = b;
        n_job = e - b;
      }
    } else {
      p = (int)(job / a.K);
      sigma = a.slo_scale[job % a.K];
    }
  } else {
    n_job = SEG ? 0 : a.n;
  }

  // this lane's group
  const int g = seg_lane;
  int cfg = -1;
  if (job_ok && g < a.G) cfg = a.group_cfg[(int64_t)p * a.G + g];
  if (cfg >= a.C) cfg = -1;
  uint64_t hostbits = 0;
  if (cfg >= 0) {
    const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
    for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> g) & 1u) << m;
  }
  const int seg_start = lane & ~(W - 1);
  const uint64_t lt_lane = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const uint64_t lt_start = (seg_start == 0) ? 0ull : (~0ull >> (64 - seg_start));
  const uint64_t below = lt_lane & ~lt_start;

  // finish-output row of this job (first match)
  int frow = -1;
  if (job_ok)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == job) { frow = f; break; }
  const bool wave_finish = __ballot(frow >= 0) != 0;

  // stage-latency table, padded with zero-latency stages up to SMAX; a padded
  // stage adds exactly 0 to a finish time that already dominates its free time
  const int nL = a.M * a.C * SMAX;
  for (int idx = tid; idx < nL; idx += kThreads) {
    const int s = idx % SMAX;
    const int mc = idx / SMAX;
    const int c = mc % a.C;
    const int m = mc / a.C;
    sL[idx] = (s < a.cfg_stages[c]) ? a.stage_lat[((int64_t)m * a.C + c) * a.smax_in + s] : 0.0;
  }
  // SLO of every model for this job: scale * d_single[m], one rounding
  for (int m = seg_lane; m < a.M; m += W) sSlo[slot * a.M + m] = job_ok ? sigma * a.d_single[m] : 0.0;
  if (tid == 0) s_nmax = 0;
  __syncthreads();
  if constexpr (SEG) {
    if (seg_lane == 0) atomicMax(&s_nmax, (unsigned long long)n_job);
  }
  __syncthreads();
  const int64_t n_loop = SEG ? (int64_t)s_nmax : a.n;

  LaneState<SMAX> st;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) st.F[s] = 0.0;
  st.served = st.fin_sum = st.word = st.hash = 0;

  // L row of (m, cfg) is lrow_base + m * lstride
  const double* lrow_base = sL + (cfg < 0 ? 0 : cfg) * SMAX;
  const int lstride = a.C * SMAX;
  const double* slo_row = sSlo + slot * a.M;

  for (int64_t base = 0; base < n_loop; base += CH) {
    const int cnt_all = (int)((n_loop - base) < CH ? (n_loop - base) : CH);
    __syncthreads();
    if constexpr (SEG) {
      const int64_t rem = n_job - base;
      const int cnt_job = rem <= 0 ? 0 : (rem < CH ? (int)rem : CH);
      for (int e = seg_lane; e < cnt_job; e += W) {
        sT[slot * CH + e] = a.t[seg_begin + base + e];
        sM[slot * CH + e] = a.model[seg_begin + base + e];
      }
    } else {
      for (int e = tid; e < cnt_all; e += kThreads) {
        sT[e] = a.t[base + e];
        sM[e] = a.model[base + e];
      }
    }
    __syncthreads();
    const double* cT = SEG ? sT + slot * CH : sT;
    const int32_t* cM = SEG ? sM + slot * CH : sM;
    int cnt = cnt_all;
    if constexpr (SEG) {
      const int64_t rem = n_job - base;
      cnt = rem <= 0 ? 0 : (rem < CH ? (int)rem : CH);
    }
    if (wave_finish)
      run_chunk<W, SMAX, true>(st, cT, cM, cnt, base, n_job, hostbits, below, lrow_base, lstride, slo_row,
                               seg_lane, frow, a.out_finish, a.finish_stride);
    else
      run_chunk<W, SMAX, false>(st, cT, cM, cnt, base, n_job, hostbits, below, lrow_base, lstride, slo_row,
                                seg_lane, frow, a.out_finish, a.finish_stride);
  }

  // combine the job's lanes and write its outputs
  const uint64_t served = seg_sum_u64<W>(st.served);
  const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum);
  if (job_ok && seg_lane == 0) {
    a.out_served[job] = (int64_t)served;
    if (a.out_attain) a.out_attain[job] = n_job > 0 ? (double)served / (double)n_job : 0.0;
    if (a.out_digest) {
      a.out_digest[2 * job] = st.hash;
      a.out_digest[2 * job + 1] = fin_sum;
    }
  }
}

}  // namespace as_dev
