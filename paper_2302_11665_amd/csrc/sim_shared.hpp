// Shared-trace serving-simulator kernel for gfx950: every job of a launch
// simulates the same arrival trace.
//
// Layout as in sim_kernel.hpp with one group per lane: a job owns W lanes of a
// wavefront, lane r of the job holds group r's stage free times in registers;
// 64 / W jobs per wavefront, four wavefronts per workgroup.  The trace is
// staged through LDS in chunks read with coalesced loads by the whole
// workgroup (each request is read from HBM/L2 once per workgroup), together
// with the stage-latency table and the SLO (or single-device latency) table.
//
// Per request, lane sets are kept as 64-bit wavefront masks in scalar
// registers: the hosting lanes come from a vector compare, the dispatch
// target of every job is one mask, and the accepted lanes are that mask ANDed
// with the deadline compare.  Commit and counting run under that mask.
//
// Dispatch (Sec. 4.3): a per-wavefront bit per model, computed once, says
// whether every job of the wavefront has at most one group hosting the model;
// then the hosting lanes are the dispatch targets and no reduction is needed.
// Otherwise the keys (stage-0 free time of hosting groups, +inf elsewhere) go
// through the butterfly min of sim_kernel.hpp, and the lowest lane of each job
// holding the minimum -- the lowest set bit of every W-bit field of the
// equality mask, computed on the scalar unit -- is the target.  Projection,
// admission, commit and counting are sim_kernel.hpp's, so the results are
// bit-identical.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alpaserve_sim.h"
#include "sim_kernel.hpp"

namespace as_dev {

// Lowest set bit of every aligned W-bit field of a 64-bit lane mask (uniform,
// scalar ALU).  Per field, -b is (~b + 1) computed without carries crossing
// field boundaries: fieldwise x + y = ((x & ~H) + (y & ~H)) ^ ((x ^ y) & H),
// H = the top bit of every field, y = L = the bottom bit of every field.
template <int W>
__device__ __forceinline__ uint64_t lowest_per_field(uint64_t b) {
  if constexpr (W == 1) {
    return b;
  } else if constexpr (W == 64) {
    return b & (~b + 1);
  } else {
    uint64_t L = 0, H = 0;
#pragma unroll
    for (int f = 0; f < 64; f += W) {
      L |= 1ull << f;
      H |= 1ull << (f + W - 1);
    }
    const uint64_t x = ~b;
    const uint64_t neg = ((x & ~H) + L) ^ ((x ^ L) & H);
    return b & neg;
  }
}

template <int SMAX>
struct SharedLane {
  double F[SMAX];
  uint64_t fin_sum, hash, served;
  uint32_t wlo;
};

struct SharedConst {
  uint64_t hostbits;      // bit m: this lane's group hosts model m
  uint64_t single;        // bit m: no job of the wavefront has two groups hosting m
  uint64_t segmask;       // lanes of this lane's job
  const double* lrow;     // stage-latency row of this lane's configuration for model 0
  int lshift;             // log2 of the per-model row stride (bytes) of the LDS table
  const double* slo;      // LDS: scale * d_single[m] (one scale) or d_single[m]
  double sigma;           // this job's scale (used when jobs differ in scale)
  int seg_lane;
  int frow;
};

// One request at trace position i.  USIG: every job uses the same scale and
// c.slo holds the SLOs.
template <int W, int SMAX, bool USIG, bool FINISH>
__device__ __forceinline__ void fast_step(SharedLane<SMAX>& st, const SharedConst& c, double ti,
                                          int mi, const double* L, double slo_or_d, int64_t i,
                                          int64_t n, double* __restrict__ out_finish,
                                          uint32_t& sr) {
  const double kInf = __builtin_inf();
  const bool hosted = (c.hostbits >> mi) & 1u;
  const uint64_t hm = __builtin_amdgcn_ballot_w64(hosted);
  const int mu = __builtin_amdgcn_readfirstlane(mi);
  uint64_t cm;  // the dispatch target of every job: one lane per job or none
  if ((c.single >> mu) & 1u) {
    cm = hm;
  } else {
    const double key = hosted ? st.F[0] : kInf;
    const double mn = seg_min<W>(key);
    // mn == +inf: no group of the job hosts the model, so no lane matches
    const bool eq = key == vmin(mn, 1.7976931348623157e308);
    cm = lowest_per_field<W>(__builtin_amdgcn_ballot_w64(eq));
  }
  double fs[SMAX];
  double f = ti;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    fs[s] = vmax(f, st.F[s]) + L[s];
    f = fs[s];
  }
  const double deadline = ti + (USIG ? slo_or_d : c.sigma * slo_or_d);
  const uint64_t am = cm & __builtin_amdgcn_ballot_w64(!(f > deadline));
  const bool acc = __builtin_amdgcn_inverse_ballot_w64(am);
  if (acc) {
#pragma unroll
    for (int s = 0; s < SMAX; ++s) st.F[s] = fs[s];
    st.fin_sum += (uint64_t)__double_as_longlong(f);
  }
  sr = (sr << 1) | (acc ? 1u : 0u);
  if constexpr (FINISH) {
    if (c.frow >= 0) {
      double* dst = out_finish + (int64_t)c.frow * n + i;
      if (__builtin_amdgcn_inverse_ballot_w64(cm)) *dst = acc ? f : -1.0;
      else if ((cm & c.segmask) == 0 && c.seg_lane == 0) *dst = -2.0;
    }
  }
}

// Requests [i0, i0 + B) from the LDS chunk: read all of their inputs first
// (LDS reads in flight together), then run them in order.
template <int W, int SMAX, int B, bool USIG, bool FINISH>
__device__ __forceinline__ void fast_batch(SharedLane<SMAX>& st, const SharedConst& c,
                                           const double* __restrict__ cT,
                                           const int32_t* __restrict__ cM, int64_t i0, int64_t n,
                                           double* __restrict__ out_finish, uint32_t& sr) {
  double t[B], so[B], L[B][SMAX];
  int m[B];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    t[k] = cT[k];
    m[k] = cM[k];
  }
#pragma unroll
  for (int k = 0; k < B; ++k) {
    const double* row = (const double*)((const char*)c.lrow + ((unsigned)m[k] << c.lshift));
#pragma unroll
    for (int s = 0; s < SMAX; ++s) L[k][s] = row[s];
    so[k] = c.slo[m[k]];
  }
#pragma unroll
  for (int k = 0; k < B; ++k)
    fast_step<W, SMAX, USIG, FINISH>(st, c, t[k], m[k], L[k], so[k], i0 + k, n, out_finish, sr);
}

// All requests of one LDS chunk [base, base + cnt): 32-request halves of
// 64-request accept words.
template <int W, int SMAX, bool USIG, bool FINISH>
__device__ __forceinline__ void fast_chunk(SharedLane<SMAX>& st, const SharedConst& c,
                                           const double* __restrict__ cT,
                                           const int32_t* __restrict__ cM, int cnt, int64_t base,
                                           int64_t n, double* __restrict__ out_finish) {
  constexpr int B = SMAX <= 4 ? 4 : 2;
  for (int h = 0; h < cnt; h += 32) {
    const int hc = (cnt - h) < 32 ? (cnt - h) : 32;
    uint32_t sr = 0;
    uint32_t bits;
    if (hc == 32) {
      for (int e = 0; e < 32; e += B)
        fast_batch<W, SMAX, B, USIG, FINISH>(st, c, cT + h + e, cM + h + e, base + h + e, n,
                                             out_finish, sr);
      bits = __builtin_bitreverse32(sr);
    } else {
      for (int e = 0; e < hc; ++e)
        fast_batch<W, SMAX, 1, USIG, FINISH>(st, c, cT + h + e, cM + h + e, base + h + e, n,
                                             out_finish, sr);
      bits = __builtin_bitreverse32(sr) >> (32 - hc);
    }
    const int64_t pos = (base + h) & 63;  // 0 or 32
    const bool end = base + h + hc == n;
    if (pos == 0 && !end) {
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

template <int W, int SMAX, bool USIG>
__global__ __launch_bounds__(kThreads) void shared_kernel(const KArgs a) {
  constexpr int JW = 64 / W;
  constexpr int kSlots = JW * kWaves;
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1, lshift = 0;
  while (cp < a.C) cp <<= 1;
  while ((1 << lshift) < cp * SMAX * 8) ++lshift;
  double* sL = reinterpret_cast<double*>(smem);  // [M][Cp][SMAX]
  double* sS = sL + (size_t)a.M * cp * SMAX;     // [M] SLO (one scale) or d_single
  double* sT = sS + a.M;                         // chunk times
  int32_t* sM = reinterpret_cast<int32_t*>(sT + kChunk);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int seg_lane = lane & (W - 1);
  const int64_t job = (int64_t)blockIdx.x * kSlots + wave * JW + lane / W;
  const bool job_ok = job < a.J;
  int p = 0;
  double sigma = 0.0;
  if (job_ok) {
    p = (int)(job / a.K);
    sigma = a.slo_scale[job % a.K];
  }
  int cfg = -1;
  if (job_ok && seg_lane < a.G) cfg = a.group_cfg[(int64_t)p * a.G + seg_lane];
  if (cfg >= a.C || cfg < 0) cfg = -1;
  uint64_t hb = 0;
  if (cfg >= 0) {
    const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
    for (int m = 0; m < a.M; ++m) hb |= ((hm[m] >> seg_lane) & 1u) << m;
  }
  SharedConst c;
  c.hostbits = hb;
  // single[m]: every job of the wavefront has at most one group hosting m
  {
    uint64_t single = 0;
    for (int m = 0; m < a.M; ++m) {
      const uint64_t hm = __builtin_amdgcn_ballot_w64((hb >> m) & 1u);
      if (lowest_per_field<W>(hm) == hm) single |= 1ull << m;
    }
    c.single = single;
  }
  const int seg_start = lane & ~(W - 1);
  c.segmask = (W == 64 ? ~0ull : ((1ull << W) - 1)) << seg_start;
  c.lrow = sL + (cfg < 0 ? 0 : cfg) * SMAX;
  c.lshift = lshift;
  c.slo = sS;
  c.sigma = sigma;
  c.seg_lane = seg_lane;
  c.frow = -1;
  if (job_ok)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == job) {
        c.frow = f;
        break;
      }
  const bool wave_finish = __builtin_amdgcn_ballot_w64(c.frow >= 0) != 0;

  // stage-latency table padded with zero-latency stages (see sim_kernel.hpp)
  const int nL = a.M * cp * SMAX;
  for (int idx = tid; idx < nL; idx += kThreads) {
    const int s = idx % SMAX;
    const int mc = idx / SMAX;
    const int cc = mc % cp;
    const int m = mc / cp;
    sL[idx] = (cc < a.C && s < a.cfg_stages[cc])
                  ? a.stage_lat[((int64_t)m * a.C + cc) * a.smax_in + s]
                  : 0.0;
  }
  // one scale: the SLO of every model, scale * d_single[m] (one rounding)
  for (int m = tid; m < a.M; m += kThreads)
    sS[m] = USIG ? a.slo_scale[0] * a.d_single[m] : a.d_single[m];

  SharedLane<SMAX> st;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) st.F[s] = 0.0;
  st.fin_sum = st.hash = st.served = 0;
  st.wlo = 0;

  const int64_t n = a.n;
  for (int64_t base = 0; base < n; base += kChunk) {
    const int cnt = (int)((n - base) < kChunk ? (n - base) : kChunk);
    __syncthreads();
    for (int e = tid; e < cnt; e += kThreads) {
      sT[e] = a.t[base + e];
      sM[e] = a.model[base + e];
    }
    __syncthreads();
    if (wave_finish)
      fast_chunk<W, SMAX, USIG, true>(st, c, sT, sM, cnt, base, n, a.out_finish);
    else
      fast_chunk<W, SMAX, USIG, false>(st, c, sT, sM, cnt, base, n, a.out_finish);
  }

  const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum);
  if (job_ok && seg_lane == 0) {
    a.out_served[job] = (int64_t)st.served;
    if (a.out_attain) a.out_attain[job] = n > 0 ? (double)st.served / (double)n : 0.0;
    if (a.out_digest) {
      a.out_digest[2 * job] = st.hash;
      a.out_digest[2 * job + 1] = fin_sum;
    }
  }
}

}  // namespace as_dev
