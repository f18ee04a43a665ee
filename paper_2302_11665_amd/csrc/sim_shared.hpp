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

// Per-lane state: group (lane mod W) of JPL different jobs.
template <int JPL, int SMAX>
struct SharedLane {
  double F[JPL][SMAX];
  uint64_t fin_sum[JPL], hash[JPL], served[JPL];
  uint32_t wlo[JPL];
};

template <int JPL>
struct SharedConst {
  uint64_t hostbits[JPL];  // bit m: this lane's group of job set j hosts model m
  uint64_t single;         // bit m: no job of the wavefront has two groups hosting m
  uint64_t segmask;        // lanes of this lane's jobs
  const double* lrow[JPL]; // stage-latency row of job set j's configuration for model 0
  int lshift;              // log2 of the per-model row stride (bytes) of the LDS table
  const double* slo;       // LDS: scale * d_single[m] (one scale) or d_single[m]
  double sigma[JPL];       // each job's scale (used when jobs differ in scale)
  int seg_lane;
  int frow[JPL];
};

// One request at trace position i for the JPL jobs of every lane.  USIG:
// every job uses the same scale and c.slo holds the SLOs.  The JPL jobs share
// the request inputs and their dependency chains interleave.
template <int W, int JPL, int SMAX, bool USIG, bool FINISH>
__device__ __forceinline__ void fast_step(SharedLane<JPL, SMAX>& st, const SharedConst<JPL>& c,
                                          double ti, int mi, const double (&L)[JPL][SMAX],
                                          double slo_or_d,
                                          int64_t i, int64_t n, double* __restrict__ out_finish,
                                          uint32_t (&sr)[JPL]) {
  const double kInf = __builtin_inf();
  const int mu = __builtin_amdgcn_readfirstlane(mi);
  bool hosted[JPL];
  uint64_t cm[JPL];  // the dispatch target of every job: one lane per job or none
#pragma unroll
  for (int j = 0; j < JPL; ++j) {
    hosted[j] = (c.hostbits[j] >> mi) & 1u;
    cm[j] = __builtin_amdgcn_ballot_w64(hosted[j]);
  }
  if (!((c.single >> mu) & 1u)) {
#pragma unroll
    for (int j = 0; j < JPL; ++j) {
      const double key = hosted[j] ? st.F[j][0] : kInf;
      const double mn = seg_min<W>(key);
      // mn == +inf: no group of the job hosts the model, so no lane matches
      const bool eq = key == vmin(mn, 1.7976931348623157e308);
      cm[j] = lowest_per_field<W>(__builtin_amdgcn_ballot_w64(eq));
    }
  }
  double fs[JPL][SMAX];
  double f[JPL];
#pragma unroll
  for (int j = 0; j < JPL; ++j) f[j] = ti;
#pragma unroll
  for (int s = 0; s < SMAX; ++s)
#pragma unroll
    for (int j = 0; j < JPL; ++j) {
      fs[j][s] = vmax(f[j], st.F[j][s]) + L[j][s];
      f[j] = fs[j][s];
    }
#pragma unroll
  for (int j = 0; j < JPL; ++j) {
    const double deadline = ti + (USIG ? slo_or_d : c.sigma[j] * slo_or_d);
    const uint64_t am = cm[j] & __builtin_amdgcn_ballot_w64(!(f[j] > deadline));
    const bool acc = __builtin_amdgcn_inverse_ballot_w64(am);
    if (acc) {
#pragma unroll
      for (int s = 0; s < SMAX; ++s) st.F[j][s] = fs[j][s];
      st.fin_sum[j] += (uint64_t)__double_as_longlong(f[j]);
    }
    sr[j] = (sr[j] << 1) | (acc ? 1u : 0u);
    if constexpr (FINISH) {
      if (c.frow[j] >= 0) {
        double* dst = out_finish + (int64_t)c.frow[j] * n + i;
        if (__builtin_amdgcn_inverse_ballot_w64(cm[j])) *dst = acc ? f[j] : -1.0;
        else if ((cm[j] & c.segmask) == 0 && c.seg_lane == 0) *dst = -2.0;
      }
    }
  }
}

// Requests [i0, i0 + B) from the LDS chunk: read all of their inputs first
// (LDS reads in flight together), then run them in order.  LSH: the JPL job
// sets of every lane use the same configuration, so one stage-latency row
// serves them all.
template <int W, int JPL, int SMAX, int B, bool USIG, bool FINISH, bool LSH>
__device__ __forceinline__ void fast_batch(SharedLane<JPL, SMAX>& st, const SharedConst<JPL>& c,
                                           const double* __restrict__ cT,
                                           const int32_t* __restrict__ cM, int64_t i0, int64_t n,
                                           double* __restrict__ out_finish, uint32_t (&sr)[JPL]) {
  double t[B], so[B], L[B][JPL][SMAX];
  int m[B];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    t[k] = cT[k];
    m[k] = cM[k];
  }
#pragma unroll
  for (int k = 0; k < B; ++k) {
#pragma unroll
    for (int j = 0; j < JPL; ++j) {
      if (LSH && j > 0) {
#pragma unroll
        for (int s = 0; s < SMAX; ++s) L[k][j][s] = L[k][0][s];
      } else {
        const double* row =
            (const double*)((const char*)c.lrow[j] + ((unsigned)m[k] << c.lshift));
#pragma unroll
        for (int s = 0; s < SMAX; ++s) L[k][j][s] = row[s];
      }
    }
    so[k] = c.slo[m[k]];
  }
#pragma unroll
  for (int k = 0; k < B; ++k)
    fast_step<W, JPL, SMAX, USIG, FINISH>(st, c, t[k], m[k], L[k], so[k], i0 + k, n, out_finish,
                                          sr);
}

// All requests of one LDS chunk [base, base + cnt): 32-request halves of
// 64-request accept words.
template <int W, int JPL, int SMAX, bool USIG, bool FINISH, bool LSH>
__device__ __forceinline__ void fast_chunk(SharedLane<JPL, SMAX>& st, const SharedConst<JPL>& c,
                                           const double* __restrict__ cT,
                                           const int32_t* __restrict__ cM, int cnt, int64_t base,
                                           int64_t n, double* __restrict__ out_finish) {
  constexpr int B = (SMAX <= 4 && JPL == 1) ? 4 : 2;
  for (int h = 0; h < cnt; h += 32) {
    const int hc = (cnt - h) < 32 ? (cnt - h) : 32;
    uint32_t sr[JPL];
#pragma unroll
    for (int j = 0; j < JPL; ++j) sr[j] = 0;
    if (hc == 32) {
      for (int e = 0; e < 32; e += B)
        fast_batch<W, JPL, SMAX, B, USIG, FINISH, LSH>(st, c, cT + h + e, cM + h + e, base + h + e,
                                                       n, out_finish, sr);
    } else {
      for (int e = 0; e < hc; ++e)
        fast_batch<W, JPL, SMAX, 1, USIG, FINISH, LSH>(st, c, cT + h + e, cM + h + e, base + h + e,
                                                       n, out_finish, sr);
    }
    const int64_t pos = (base + h) & 63;  // 0 or 32
    const bool end = base + h + hc == n;
#pragma unroll
    for (int j = 0; j < JPL; ++j) {
      // sr holds request e at bit hc-1-e; bits: request e at bit e
      const uint32_t bits = hc == 32 ? __builtin_bitreverse32(sr[j])
                                     : (__builtin_bitreverse32(sr[j]) >> (32 - hc));
      if (pos == 0 && !end) {
        st.wlo[j] = bits;
      } else {
        const uint64_t w = pos == 0 ? (uint64_t)bits : (((uint64_t)bits << 32) | st.wlo[j]);
        const uint64_t wj = seg_or<W>(w);
        st.hash[j] = (st.hash[j] ^ wj) * kHashMul;
        st.served[j] += (uint64_t)__popcll(wj);
        st.wlo[j] = 0;
      }
    }
  }
}

// Jobs of workgroup b: wavefront v holds jobs b*64*JPL*kWaves/W + v*JW*JPL +
// j*JW + lane/W for job sets j < JPL, JW = 64/W.
template <int W, int JPL, int SMAX, bool USIG>
__global__ __launch_bounds__(kThreads) void shared_kernel(const KArgs a) {
  constexpr int JW = 64 / W;
  constexpr int kSlots = JW * JPL * kWaves;
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
  const int64_t job0 = (int64_t)blockIdx.x * kSlots + wave * JW * JPL + lane / W;

  SharedConst<JPL> c;
  bool job_ok[JPL];
  int cfg_j[JPL];
#pragma unroll
  for (int j = 0; j < JPL; ++j) {
    const int64_t job = job0 + j * JW;
    job_ok[j] = job < a.J;
    int p = 0;
    c.sigma[j] = 0.0;
    if (job_ok[j]) {
      p = (int)(job / a.K);
      c.sigma[j] = a.slo_scale[job % a.K];
    }
    int cfg = -1;
    if (job_ok[j] && seg_lane < a.G) cfg = a.group_cfg[(int64_t)p * a.G + seg_lane];
    if (cfg >= a.C || cfg < 0) cfg = -1;
    cfg_j[j] = cfg;
    uint64_t hb = 0;
    if (cfg >= 0) {
      const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
      for (int m = 0; m < a.M; ++m) hb |= ((hm[m] >> seg_lane) & 1u) << m;
    }
    c.hostbits[j] = hb;
    c.frow[j] = -1;
    if (job_ok[j])
      for (int f = 0; f < a.n_finish; ++f)
        if (a.finish_jobs[f] == job) {
          c.frow[j] = f;
          break;
        }
  }
  // single[m]: every job of the wavefront has at most one group hosting m
  {
    uint64_t single = 0;
    for (int m = 0; m < a.M; ++m) {
      bool ok = true;
#pragma unroll
      for (int j = 0; j < JPL; ++j) {
        const uint64_t hm = __builtin_amdgcn_ballot_w64((c.hostbits[j] >> m) & 1u);
        ok = ok && lowest_per_field<W>(hm) == hm;
      }
      if (ok) single |= 1ull << m;
    }
    c.single = single;
  }
  const int seg_start = lane & ~(W - 1);
  c.segmask = (W == 64 ? ~0ull : ((1ull << W) - 1)) << seg_start;
  // do the job sets of every lane of the wavefront share one configuration?
  bool same = true;
#pragma unroll
  for (int j = 0; j < JPL; ++j) {
    c.lrow[j] = sL + (cfg_j[j] < 0 ? 0 : cfg_j[j]) * SMAX;
    same = same && (cfg_j[j] < 0 || cfg_j[0] < 0 || cfg_j[j] == cfg_j[0]);
  }
  if (cfg_j[0] < 0)
#pragma unroll
    for (int j = 1; j < JPL; ++j)
      if (cfg_j[j] >= 0) c.lrow[0] = c.lrow[j];
  const bool lsh = JPL == 1 || __builtin_amdgcn_ballot_w64(!same) == 0;
  c.lshift = lshift;
  c.slo = sS;
  c.seg_lane = seg_lane;
  bool any_finish = false;
#pragma unroll
  for (int j = 0; j < JPL; ++j) any_finish = any_finish || c.frow[j] >= 0;
  const bool wave_finish = __builtin_amdgcn_ballot_w64(any_finish) != 0;

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

  SharedLane<JPL, SMAX> st;
#pragma unroll
  for (int j = 0; j < JPL; ++j) {
#pragma unroll
    for (int s = 0; s < SMAX; ++s) st.F[j][s] = 0.0;
    st.fin_sum[j] = st.hash[j] = st.served[j] = 0;
    st.wlo[j] = 0;
  }

  const int64_t n = a.n;
  for (int64_t base = 0; base < n; base += kChunk) {
    const int cnt = (int)((n - base) < kChunk ? (n - base) : kChunk);
    __syncthreads();
    for (int e = tid; e < cnt; e += kThreads) {
      sT[e] = a.t[base + e];
      sM[e] = a.model[base + e];
    }
    __syncthreads();
    if (lsh) {
      if (wave_finish)
        fast_chunk<W, JPL, SMAX, USIG, true, true>(st, c, sT, sM, cnt, base, n, a.out_finish);
      else
        fast_chunk<W, JPL, SMAX, USIG, false, true>(st, c, sT, sM, cnt, base, n, a.out_finish);
    } else if constexpr (JPL > 1) {
      if (wave_finish)
        fast_chunk<W, JPL, SMAX, USIG, true, false>(st, c, sT, sM, cnt, base, n, a.out_finish);
      else
        fast_chunk<W, JPL, SMAX, USIG, false, false>(st, c, sT, sM, cnt, base, n, a.out_finish);
    }
  }

#pragma unroll
  for (int j = 0; j < JPL; ++j) {
    const int64_t job = job0 + j * JW;
    const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum[j]);
    if (job_ok[j] && seg_lane == 0) {
      a.out_served[job] = (int64_t)st.served[j];
      if (a.out_attain) a.out_attain[job] = n > 0 ? (double)st.served[j] / (double)n : 0.0;
      if (a.out_digest) {
        a.out_digest[2 * job] = st.hash[j];
        a.out_digest[2 * job + 1] = fin_sum;
      }
    }
  }
}

}  // namespace as_dev
