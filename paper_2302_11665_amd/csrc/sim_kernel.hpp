// Batched serving-simulator kernel for gfx950 (CDNA4, wave64).
//
// One job = one (trace, placement, SLO scale).  Its state is the free time
// F[g][s] of every stage s of every group g (Sec. 3.4: each pipeline stage is
// a single server).  Layout: a job owns W consecutive lanes of a wavefront and
// each lane owns GPL consecutive groups (lane r holds groups r*GPL .. r*GPL +
// GPL - 1); a group's stage free times live in the lane's registers.  One
// wavefront carries 64 / W jobs; W * GPL >= the group count.  The host picks
// (W, GPL) so that the jobs fill the GPU's SIMDs with as few instructions per
// job and request as possible.
//
// Per request (t, m) the lanes of a job:
//   1. dispatch (Sec. 4.3): key = F[g][0] for every local group that hosts m,
//      +inf otherwise; the lane keeps its smallest key (lowest local group on
//      ties), a butterfly min over the job's W lanes (DPP inside 16-lane rows,
//      lane shuffles across rows) yields the job minimum, and the lowest lane
//      holding it wins (wavefront ballot restricted to the job's lanes below
//      the caller) -- so ties go to the lowest group index;
//   2. project (Sec. 3.4): each lane runs the stage chain
//      f_s = max(f_{s-1}, F[s]) + L[m][c][s] of each of its local groups;
//   3. admit (Sec. 4.3, Sec. 3.2): the chosen lane accepts iff the chosen
//      group's f_{S-1} <= t + (scale * d_single[m]) and then commits F[s] := f_s;
//   4. count: accept decisions shift into a 32-bit register; every 32
//      requests they become bits of the job's 64-bit accept word, folded into
//      the digest every 64 requests (and at the end); served counts are the
//      population counts of the folded words.
//
// Arrivals are staged through LDS in chunks loaded with coalesced reads by the
// whole workgroup; a shared trace is read once per workgroup per chunk and
// every wavefront then reads the same LDS words (broadcast).  Segmented
// traces (one per job) are staged per job slot.
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

constexpr int kWaves = 4;  // wavefronts per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kChunk = 2048;  // shared-trace requests per LDS chunk (multiple of 64)
// per-job requests per LDS chunk for segmented traces: all job slots of a
// workgroup share about 48 KiB; a multiple of 32
template <int kSlots>
constexpr int seg_chunk() {
  return (4096 / kSlots) > 128 ? 128 : ((4096 / kSlots) < 32 ? 32 : 4096 / kSlots);
}
constexpr uint64_t kHashMul = 0x9E3779B97F4A7C15ULL;

struct KArgs {
  const double* t;
  const int32_t* model;
  int64_t n;               // shared trace length
  const int64_t* seg_off;  // segmented: [n_segments + 1]
  const as_job_t* jobs;    // segmented: [J]
  const int32_t* order;    // segmented, one job per wavefront: slot -> job, a permutation (null: identity)
  int32_t* next_slot;      // segmented: set, the wavefronts take slots in turn from this counter (0 at
                           // launch) until all are taken; null: wavefront w runs slot w
  const double* d_single;
  const double* stage_lat;
  const int32_t* group_cfg;
  const uint64_t* host_mask;
  const double* slo_scale;  // shared: [K]
  int64_t* out_served;
  double* out_attain;
  uint64_t* out_digest;
  double* out_finish;
  int64_t finish_stride;
  int64_t* out_model_served;  // statistics launches: [J][M]
  double* out_group_busy;     // statistics launches: [J][G]
  int32_t M, C, smax_in, G, K, J, n_finish;
  int32_t P, n_segments;
  int32_t cfg_stages[AS_MAX_CONFIGS];
  int32_t finish_jobs[AS_MAX_FINISH];
  // set: the launch does nothing unless *gate != 0 (the speculative kernels'
  // give-up flag, when these kernels stand behind them)
  const int32_t* gate;
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
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(v), CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(v), CTRL, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
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

// Per-lane simulation state: GPL groups of one job.
template <int GPL, int SMAX>
struct LaneState {
  double F[GPL][SMAX];
  uint64_t fin_sum;  // this lane's accepted finish-time bit sum
  uint64_t hash;     // job digest (same in every lane of the job)
  uint64_t served;   // job served count (same in every lane of the job)
  uint32_t wlo;      // accept bits of the first half of the current 64-block
};

// Constant per-lane inputs of the request loop.
template <int GPL>
struct LaneConst {
  uint64_t hostbits[GPL];   // bit m: local group k hosts model m
  const double* lrow[GPL];  // stage-latency row of local group k for model 0
  int lshift;               // log2 of the per-model row stride (bytes) of the LDS table
  const double* dsingle;    // single-device latency of every model (LDS)
  double sigma;             // this job's SLO scale
  uint64_t below;           // lanes of this job below this lane
  int seg_lane;
  int frow;  // per-request output row of this job, -1 if none
};

// One request (t, m) at trace position i: dispatch, projection, admission,
// commit; shifts the accept decision into sr.
template <int W, int GPL, int SMAX, bool FINISH>
__device__ __forceinline__ void step(LaneState<GPL, SMAX>& st, const LaneConst<GPL>& lc, double ti,
                                     int mi, int64_t i, uint32_t& sr,
                                     double* __restrict__ out_finish, int64_t finish_stride) {
  const double kInf = __builtin_inf();
  {
    // 1. dispatch
    double lmin = kInf;
    int kb = 0;
#pragma unroll
    for (int k = 0; k < GPL; ++k) {
      const bool hosted = (lc.hostbits[k] >> mi) & 1u;
      const double key = hosted ? st.F[k][0] : kInf;
      if (k == 0) {
        lmin = key;
      } else if (key < lmin) {
        lmin = key;
        kb = k;
      }
    }
    const double mn = seg_min<W>(lmin);
    const bool eq = (lmin == mn) && (mn != kInf);
    const uint64_t ball = __builtin_amdgcn_ballot_w64(eq);
    const bool chosen = eq && ((ball & lc.below) == 0);
    // 2. projection through the stage chain of every local group
    double fs[GPL][SMAX];
#pragma unroll
    for (int k = 0; k < GPL; ++k) {
      const double* L = (const double*)((const char*)lc.lrow[k] + ((unsigned)mi << lc.lshift));
      double f = ti;
#pragma unroll
      for (int s = 0; s < SMAX; ++s) {
        fs[k][s] = vmax(f, st.F[k][s]) + L[s];
        f = fs[k][s];
      }
    }
    double f = fs[0][SMAX - 1];
#pragma unroll
    for (int k = 1; k < GPL; ++k) f = (kb == k) ? fs[k][SMAX - 1] : f;
    // 3. admission and commit
    const double deadline = ti + lc.sigma * lc.dsingle[mi];
    const bool acc = chosen && !(f > deadline);
#pragma unroll
    for (int k = 0; k < GPL; ++k) {
      const bool ak = acc && (GPL == 1 || kb == k);
#pragma unroll
      for (int s = 0; s < SMAX; ++s) st.F[k][s] = ak ? fs[k][s] : st.F[k][s];
    }
    st.fin_sum += acc ? (uint64_t)__double_as_longlong(f) : 0ull;
    sr = (sr << 1) | (acc ? 1u : 0u);
    if constexpr (FINISH) {
      if (lc.frow >= 0 && i < finish_stride) {
        double* dst = out_finish + (int64_t)lc.frow * finish_stride + i;
        if (chosen) *dst = acc ? f : -1.0;
        else if (mn == kInf && lc.seg_lane == 0) *dst = -2.0;
      }
    }
  }
}

// Requests [i0, i0 + hc) of one LDS chunk, hc <= 32: one 32-request half of a
// 64-request accept word.  Returns the accept bits (bit e = request i0 + e
// accepted by this lane).
template <int W, int GPL, int SMAX, bool FINISH>
__device__ __forceinline__ uint32_t run_half(LaneState<GPL, SMAX>& st, const LaneConst<GPL>& lc,
                                             const double* __restrict__ cT,
                                             const int32_t* __restrict__ cM, int hc, int64_t i0,
                                             double* __restrict__ out_finish,
                                             int64_t finish_stride) {
  uint32_t sr = 0;
  if (hc == 32) {
    // full half: fixed trip count, unrolled so LDS reads use immediate
    // offsets and can be issued ahead of the dependent arithmetic
#pragma unroll 4
    for (int e = 0; e < 32; ++e)
      step<W, GPL, SMAX, FINISH>(st, lc, cT[e], cM[e], i0 + e, sr, out_finish, finish_stride);
    return __builtin_bitreverse32(sr);
  }
  for (int e = 0; e < hc; ++e)
    step<W, GPL, SMAX, FINISH>(st, lc, cT[e], cM[e], i0 + e, sr, out_finish, finish_stride);
  // sr holds request e at bit hc-1-e; return request e at bit e
  return __builtin_bitreverse32(sr) >> (32 - hc);
}

// All requests of one LDS chunk [base, base + cnt); base is a multiple of 64
// and cnt a multiple of 32 unless the job ends inside the chunk.
template <int W, int GPL, int SMAX, bool FINISH>
__device__ __forceinline__ void run_chunk(LaneState<GPL, SMAX>& st, const LaneConst<GPL>& lc,
                                          const double* __restrict__ cT,
                                          const int32_t* __restrict__ cM, int cnt, int64_t base,
                                          int64_t n_job, double* __restrict__ out_finish,
                                          int64_t finish_stride) {
  for (int h = 0; h < cnt; h += 32) {
    const int hc = (cnt - h) < 32 ? (cnt - h) : 32;
    const uint32_t bits = run_half<W, GPL, SMAX, FINISH>(st, lc, cT + h, cM + h, hc, base + h,
                                                         out_finish, finish_stride);
    const int64_t pos = (base + h) & 63;  // 0 or 32
    const bool job_end = base + h + hc == n_job;
    if (pos == 0 && !job_end) {
      st.wlo = bits;
    } else {
      const uint64_t w = pos == 0 ? (uint64_t)bits : (((uint64_t)bits << 32) | st.wlo);
      const uint64_t wj = seg_or<W>(w);
      st.hash = (st.hash ^ wj) * kHashMul;
      st.served += (uint64_t)__popcll(wj);
      st.wlo = 0;
    }
  }
}

template <int W, int GPL, int SMAX, bool SEG>
__global__ __launch_bounds__(kThreads) void sim_kernel(const KArgs a) {
  if (a.gate && *a.gate == 0) return;
  constexpr int JW = 64 / W;           // jobs per wavefront
  constexpr int kSlots = JW * kWaves;  // jobs per workgroup
  constexpr int CH = SEG ? seg_chunk<kSlots>() : kChunk;
  extern __shared__ __align__(16) unsigned char smem[];
  // stage-latency table [M][Cp][SMAX], Cp = C rounded up to a power of two so
  // that a model's rows start at m << lshift bytes
  int cp = 1, lshift = 0;
  while (cp < a.C) cp <<= 1;
  while ((1 << lshift) < cp * SMAX * 8) ++lshift;
  double* sL = reinterpret_cast<double*>(smem);
  double* sD = sL + (size_t)a.M * cp * SMAX;     // [M] d_single
  double* sT = sD + a.M;                         // chunk times
  int32_t* sM = reinterpret_cast<int32_t*>(sT + (SEG ? kSlots * CH : kChunk));
  __shared__ unsigned long long s_nmax;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int seg_lane = lane & (W - 1);
  const int slot = wave * JW + lane / W;
  const int64_t job = (int64_t)blockIdx.x * kSlots + slot;
  const bool job_ok = job < a.J;

  int p = 0;
  double sigma = 0.0;
  int64_t seg_begin = 0, n_job = SEG ? 0 : a.n;
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
  }

  // this lane's groups
  LaneConst<GPL> lc;
#pragma unroll
  for (int k = 0; k < GPL; ++k) {
    const int g = seg_lane * GPL + k;
    int c = -1;
    if (job_ok && g < a.G) c = a.group_cfg[(int64_t)p * a.G + g];
    if (c >= a.C || c < 0) c = -1;
    uint64_t hb = 0;
    if (c >= 0) {
      const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
      for (int m = 0; m < a.M; ++m) hb |= ((hm[m] >> g) & 1u) << m;
    }
    lc.hostbits[k] = hb;
    lc.lrow[k] = sL + (c < 0 ? 0 : c) * SMAX;
  }
  lc.lshift = lshift;
  lc.dsingle = sD;
  lc.sigma = sigma;
  lc.seg_lane = seg_lane;
  {
    const int seg_start = lane & ~(W - 1);
    const uint64_t lt_lane = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t lt_start = (seg_start == 0) ? 0ull : (~0ull >> (64 - seg_start));
    lc.below = lt_lane & ~lt_start;
  }
  // per-request output row of this job (first match)
  lc.frow = -1;
  if (job_ok)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == job) {
        lc.frow = f;
        break;
      }
  const bool wave_finish = __ballot(lc.frow >= 0) != 0;

  // stage-latency table, padded with zero-latency stages up to SMAX; a padded
  // stage adds exactly 0 to a finish time that already dominates its free time
  const int nL = a.M * cp * SMAX;
  for (int idx = tid; idx < nL; idx += kThreads) {
    const int s = idx % SMAX;
    const int mc = idx / SMAX;
    const int c = mc % cp;
    const int m = mc / cp;
    sL[idx] = (c < a.C && s < a.cfg_stages[c])
                  ? a.stage_lat[((int64_t)m * a.C + c) * a.smax_in + s]
                  : 0.0;
  }
  for (int m = tid; m < a.M; m += kThreads) sD[m] = a.d_single[m];
  if (tid == 0) s_nmax = 0;
  __syncthreads();
  if constexpr (SEG) {
    if (seg_lane == 0) atomicMax(&s_nmax, (unsigned long long)n_job);
  }
  __syncthreads();
  const int64_t n_loop = SEG ? (int64_t)s_nmax : a.n;

  LaneState<GPL, SMAX> st;
#pragma unroll
  for (int k = 0; k < GPL; ++k)
#pragma unroll
    for (int s = 0; s < SMAX; ++s) st.F[k][s] = 0.0;
  st.fin_sum = st.hash = st.served = 0;
  st.wlo = 0;

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
      run_chunk<W, GPL, SMAX, true>(st, lc, cT, cM, cnt, base, n_job, a.out_finish, a.finish_stride);
    else
      run_chunk<W, GPL, SMAX, false>(st, lc, cT, cM, cnt, base, n_job, a.out_finish, a.finish_stride);
  }

  // combine the job's lanes and write its outputs
  const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum);
  if (job_ok && seg_lane == 0) {
    a.out_served[job] = (int64_t)st.served;
    if (a.out_attain) a.out_attain[job] = n_job > 0 ? (double)st.served / (double)n_job : 0.0;
    if (a.out_digest) {
      a.out_digest[2 * job] = st.hash;
      a.out_digest[2 * job + 1] = fin_sum;
    }
  }
}

}  // namespace as_dev
