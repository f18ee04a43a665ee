// Shared-trace serving-simulator kernel for gfx950: every job of a launch
// simulates the same arrival trace.
//
// Layout: a job owns W lanes of a wavefront, lane r of the job holds group r's
// stage free times F[0..SMAX-1] in registers; 64 / W jobs per wavefront, four
// wavefronts per workgroup.  The trace is staged through LDS in chunks read
// with coalesced loads by the whole workgroup (each request is read from
// HBM/L2 once per workgroup); every wavefront then reads the same words.
// Staging also stores each request's model-record offset and, when one SLO
// scale serves every job, its deadline t + SLO (computed once per workgroup
// instead of once per wavefront).
//
// Per-wavefront model records (LDS, one per model m, built when the kernel
// starts): the wavefront's hosting lane mask for m (bit l = lane l's group
// hosts m), the SLO (scale * d_single[m], one scale per launch) or
// d_single[m], a count that is 0 when no job of the wavefront has two groups
// hosting m and otherwise the number of jobs of the wavefront hosting m, and,
// when every group of the wavefront has the same configuration, that
// configuration's stage latencies of m.  A request therefore costs one
// address computation and reads at immediate offsets of one record.
//
// Dispatch (Sec. 4.3): the target of a job is the hosting lane with the
// smallest stage-0 free time, the lowest such lane on ties.  When the record's
// count is 0, the hosting lanes are the targets.  Otherwise the minimum is
// found on the free times' IEEE bit patterns: free times are >= 0, so with the
// sign bit cleared (-0 and +0 become equal) the unsigned order of the 64-bit
// patterns is the numeric order.  The high words are reduced first with
// one-instruction DPP min steps (v_min_u32 with a DPP operand inside 16-lane
// rows, permlane swaps across rows).  If the hosting lanes holding the
// minimal high word are exactly one per hosting job (their population count
// equals the record's count), they are the targets.  Otherwise the low words
// of the tied lanes are reduced as well, and the lowest lane of each job
// holding the minimum -- the lowest set bit of every W-bit field of the
// equality mask, computed on the scalar unit -- is the target.  Projection,
// admission and counting are sim_kernel.hpp's, so the results are
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

__device__ __forceinline__ uint32_t umin32(uint32_t a, uint32_t b) { return a < b ? a : b; }

// Unsigned minimum over each aligned W-lane segment, in every lane of it.
// Inside a 16-lane row each step is one v_min_u32 with a DPP operand; for
// W = 32 the 16-lane step swaps rows with v_permlane16_swap (its two outputs
// are the two halves of the butterfly); for W = 64 row broadcasts gather the
// minimum in lane 63, whose value is returned to every lane.
template <int W>
__device__ __forceinline__ uint32_t seg_min_u32(uint32_t x) {
  if constexpr (W >= 2) x = umin32(x, dpp_u32<kXor1>(x));
  if constexpr (W >= 4) x = umin32(x, dpp_u32<kXor2>(x));
  if constexpr (W >= 8) x = umin32(x, dpp_u32<kHalfMirror>(x));
  if constexpr (W >= 16) x = umin32(x, dpp_u32<kMirror>(x));
  if constexpr (W == 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    x = umin32(r[0], r[1]);
  }
  if constexpr (W == 64) {
    // fold the four row minima into lane 63 (row_bcast:15 into rows 1 and 3,
    // row_bcast:31 into rows 2 and 3; masked-off rows keep their value) and
    // read it back as a wave-uniform scalar
    x = umin32(x, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)x, 0x142, 0xa, 0xf, false));
    x = umin32(x, (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)x, 0x143, 0xc, 0xf, false));
    x = (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
  }
  return x;
}

// Layout of one model record: hosting mask (u64) at 0, count (u32) at 8,
// stage latencies (SMAX doubles) at 16, SLO or d_single (double) after them;
// the record size is a power of two.
constexpr int kRecMask = 0, kRecCount = 8, kRecLat = 16;
__host__ __device__ constexpr int rec_slo(int SMAX) { return kRecLat + 8 * SMAX; }
__host__ __device__ constexpr int rec_shift(int SMAX) { return SMAX == 1 ? 5 : (SMAX <= 4 ? 6 : 7); }

// Per-lane state: group (lane mod W) of one job.
template <int SMAX>
struct SharedLane {
  double F[SMAX];
  uint64_t fin_sum, hash, served;
  uint32_t wlo;
  double busy;  // statistics launches: this lane's group's busy time
};

struct SharedConst {
  const unsigned char* rec;  // this wavefront's model records (LDS)
  const double* lrow;        // stage-latency row of this lane's configuration for model 0 (LDS)
  int lshift;                // log2 of the per-model row stride (bytes) of that table
  double sigma;              // this job's scale (used when jobs differ in scale)
  uint64_t fmask;            // lanes of the wavefront's jobs with per-request output
  double* frowp;             // this job's per-request output row (lanes in fmask),
                             // filled with -2 before the launch; within a chunk:
                             // the element of the chunk's first request
  int64_t flimit;            // requests i < flimit have an output element
  int fcnt;                  // within a chunk: its first fcnt requests have one
  uint32_t* cnt;             // statistics launches: this job's per-model served counters (LDS)
  uint32_t* cntw;            // statistics launches: the wavefront's counters, [job of the wavefront][M]
  int M;                     // statistics launches: models (the counters' row length)
};

// Projection through this lane's stage chain (Sec. 3.4): fs[s] is the
// request's finish time at stage s; returns the last.
template <int SMAX>
__device__ __forceinline__ double chain(const SharedLane<SMAX>& st, double ti,
                                        const double (&L)[SMAX], double (&fs)[SMAX]) {
  double f = ti;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    fs[s] = vmax(f, st.F[s]) + L[s];
    f = fs[s];
  }
  return f;
}

// One request, number ik of its chunk.  hm: the wavefront's hosting lanes; cnt:
// the record's count; L: this lane's stage latencies of the model; dv: the
// deadline t + SLO (USIG, staged with the trace) or d_single of the model.
template <int W, int SMAX, bool USIG, bool FINISH, bool FLIM, bool STATS = false>
__device__ __forceinline__ void fast_step(SharedLane<SMAX>& st, const SharedConst& c, double ti,
                                          uint64_t hm, uint32_t cnt, const double (&L)[SMAX],
                                          double dv, int ik, uint32_t& sr, int mi = 0) {
  uint64_t cm = hm;  // the dispatch target of every job: one lane per job or none
  if (cnt != 0) {
    const bool hosted = __builtin_amdgcn_inverse_ballot_w64(hm);
    const uint64_t kb = (uint64_t)__double_as_longlong(st.F[0]);
    const uint32_t khi = hosted ? ((uint32_t)(kb >> 32) & 0x7fffffffu) : 0xffffffffu;
    const uint32_t mhi = seg_min_u32<W>(khi);
    const uint64_t eqhi = __builtin_amdgcn_ballot_w64(khi == mhi) & hm;
    cm = eqhi;
    if ((uint32_t)__builtin_popcountll(eqhi) != cnt) {
      // some job has two hosting lanes with the same high word: compare the
      // low words of the tied lanes
      const bool tied = __builtin_amdgcn_inverse_ballot_w64(eqhi);
      const uint32_t klo = tied ? (uint32_t)kb : 0xffffffffu;
      const uint32_t mlo = seg_min_u32<W>(klo);
      cm = lowest_per_field<W>(__builtin_amdgcn_ballot_w64(klo == mlo) & eqhi);
    }
  }
  double fs[SMAX];
  const double f = chain<SMAX>(st, ti, L, fs);
  // admission (Sec. 4.3, Sec. 3.2) and commit on the target lane
  const double deadline = USIG ? dv : ti + c.sigma * dv;
  const uint64_t am = cm & __builtin_amdgcn_ballot_w64(!(f > deadline));
  const bool acc = __builtin_amdgcn_inverse_ballot_w64(am);
#pragma unroll
  for (int s = 0; s < SMAX; ++s) st.F[s] = acc ? fs[s] : st.F[s];
  st.fin_sum += acc ? (uint64_t)__double_as_longlong(f) : 0ull;
  sr = (sr << 1) | (acc ? 1u : 0u);
  if constexpr (STATS) {
    // the accepting lane's group was busy for the model's slowest stage
    // (fp64 sum in trace order); the served counts per model are taken per
    // 32 requests from the accept bits (fast_chunk)
    double slowest = 0.0;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) slowest = vmax(slowest, L[s]);
    const double nb = st.busy + slowest;
    st.busy = acc ? nb : st.busy;
  }
  if constexpr (FINISH) {
    // per-request output: the job's target lane writes the finish time, or
    // -1 if rejected; rows start filled with -2 (a request no group hosts)
    if ((!FLIM || ik < c.fcnt) && __builtin_amdgcn_inverse_ballot_w64(cm & c.fmask))
      c.frowp[ik] = acc ? f : -1.0;
  }
}

// Requests [i0, i0 + B) of the LDS chunk (cTD: {t, deadline} pairs, cO:
// record offsets): read all of their inputs first (LDS reads in flight
// together), then run them in order.  UNI: every group of the wavefront has
// the same configuration, whose stage latencies the model records hold;
// otherwise each lane reads its configuration's row.
template <int W, int SMAX, int B, bool USIG, bool FINISH, bool FLIM, bool UNI, bool STATS = false>
__device__ __forceinline__ void fast_batch(SharedLane<SMAX>& st, const SharedConst& c,
                                           const double* __restrict__ cTD,
                                           const uint32_t* __restrict__ cO, int i0, uint32_t& sr) {
  double t[B], dv[B], L[B][SMAX];
  uint64_t hmv[B];
  uint32_t cnv[B], off[B];
#pragma unroll
  for (int k = 0; k < B; ++k) {
    t[k] = cTD[2 * k];
    if (USIG) dv[k] = cTD[2 * k + 1];
    off[k] = cO[k];
  }
#pragma unroll
  for (int k = 0; k < B; ++k) {
    // records are 32-byte aligned: 16-byte loads
    const unsigned char* r = c.rec + off[k];
    const uint4 head = *(const uint4*)(r + kRecMask);  // hosting mask, count
    hmv[k] = ((uint64_t)head.y << 32) | head.x;
    cnv[k] = head.z;
    if (!USIG) dv[k] = *(const double*)(r + rec_slo(SMAX));
    if (UNI) {
#pragma unroll
      for (int s = 0; s + 1 < SMAX; s += 2) {
        const double2 l2 = *(const double2*)(r + kRecLat + 8 * s);
        L[k][s] = l2.x;
        L[k][s + 1] = l2.y;
      }
      if (SMAX & 1) L[k][SMAX - 1] = *(const double*)(r + kRecLat + 8 * (SMAX - 1));
    } else {
      const double* lr =
          (const double*)((const char*)c.lrow + ((off[k] >> rec_shift(SMAX)) << c.lshift));
#pragma unroll
      for (int s = 0; s < SMAX; ++s) L[k][s] = lr[s];
    }
  }
#pragma unroll
  for (int k = 0; k < B; ++k) {
    // record words are the same in every lane: move them to scalar registers
    const uint64_t hm = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(hmv[k] >> 32)) << 32) |
                        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)hmv[k]);
    const uint32_t cnt = (uint32_t)__builtin_amdgcn_readfirstlane((int)cnv[k]);
    fast_step<W, SMAX, USIG, FINISH, FLIM, STATS>(st, c, t[k], hm, cnt, L[k], dv[k], i0 + k, sr,
                                                  (int)(off[k] >> rec_shift(SMAX)));
  }
}

// All requests of one LDS chunk [base, base + cnt): 32-request halves of
// 64-request accept words.
template <int W, int SMAX, bool USIG, bool FINISH, bool FLIM, bool UNI, bool STATS = false>
__device__ __forceinline__ void fast_chunk(SharedLane<SMAX>& st, const SharedConst& c0,
                                           const double* __restrict__ cTD,
                                           const uint32_t* __restrict__ cO, int cnt, int64_t base,
                                           int64_t n) {
  constexpr int B = SMAX <= 4 ? 4 : 2;
  // output row relative to this chunk; FLIM: only the first fcnt requests of
  // the chunk have an output element (the same for the whole wavefront)
  SharedConst c = c0;
  if (FINISH) {
    c.frowp = c0.frowp + base;
    if (FLIM) {
      const int64_t left = c0.flimit - base;
      c.fcnt = __builtin_amdgcn_readfirstlane(left <= 0 ? 0 : (left < cnt ? (int)left : cnt));
    }
  }
  for (int h = 0; h < cnt; h += 32) {
    const int hc = (cnt - h) < 32 ? (cnt - h) : 32;
    uint32_t sr = 0;
    if (hc == 32) {
      for (int e = 0; e < 32; e += B)
        fast_batch<W, SMAX, B, USIG, FINISH, FLIM, UNI, STATS>(st, c, cTD + 2 * (h + e), cO + h + e, h + e, sr);
    } else {
      for (int e = 0; e < hc; ++e)
        fast_batch<W, SMAX, 1, USIG, FINISH, FLIM, UNI, STATS>(st, c, cTD + 2 * (h + e), cO + h + e, h + e, sr);
    }
    const int64_t pos = (base + h) & 63;  // 0 or 32
    const bool end = base + h + hc == n;
    // sr holds request e at bit hc-1-e; bits: request e at bit e
    const uint32_t bits =
        hc == 32 ? __builtin_bitreverse32(sr) : (__builtin_bitreverse32(sr) >> (32 - hc));
    if constexpr (STATS) {
      // served counts per model: lane e counts request h + e for every job
      // of the wavefront that accepted it (integer counts: order-free)
      const uint32_t jb = (uint32_t)seg_or<W>((uint64_t)bits);  // the job's bits, in every lane of it
      const int e = (int)(threadIdx.x & 63);
      const uint32_t me = e < hc ? (cO[h + e] >> rec_shift(SMAX)) : 0u;
#pragma unroll
      for (int j = 0; j < 64 / W; ++j) {
        const uint32_t wj = (uint32_t)__builtin_amdgcn_readlane((int)jb, j * W);
        if (e < hc && ((wj >> e) & 1u)) atomicAdd(c.cntw + j * c.M + me, 1u);
      }
    }
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

// LDS bytes of the shared-trace kernel: model records of the four
// wavefronts, the stage-latency table [M][Cp][SMAX] (Cp = C rounded up to a
// power of two) and the trace chunk ({t, deadline} pairs and record offsets).
__host__ __device__ constexpr size_t shared_lds_bytes(int M, int Cp, int SMAX) {
  return (size_t)kWaves * M * ((size_t)1 << rec_shift(SMAX)) + (size_t)M * Cp * SMAX * 8 +
         (size_t)kChunk * 20;
}

// Statistics launches (STATS, one SLO scale) also count each job's served
// requests per model (LDS counters after the chunk) and sum each group's busy
// time, for the fast placement heuristic.
__host__ __device__ constexpr size_t shared_stats_lds_bytes(int W, int M) {
  return (size_t)kWaves * (64 / W) * M * 4;
}

// Jobs of workgroup b: wavefront v holds jobs b*kWaves*JW + v*JW + lane/W,
// JW = 64/W.  Per-request output rows must hold -2 when the kernel starts.
// The jobs one launch (or one shape segment of a multi-shape launch) runs:
// their count, group-row stride, placement rows and outputs.
struct JobSet {
  int64_t J;
  int32_t G;
  const int32_t* group_cfg;
  const uint64_t* host_mask;
  int64_t* out_served;
  double* out_attain;
  uint64_t* out_digest;
  int64_t* out_model_served;
  double* out_group_busy;
};

__device__ __forceinline__ JobSet job_set(const KArgs& a) {
  return JobSet{a.J, a.G, a.group_cfg, a.host_mask, a.out_served, a.out_attain, a.out_digest,
                a.out_model_served, a.out_group_busy};
}

// One workgroup (block number blk of its job set) of the shared-trace
// simulation.  ROWS: the launch may carry per-request output rows.
template <int W, int SMAX, bool USIG, bool STATS, bool ROWS>
__device__ __forceinline__ void shared_body(const KArgs& a, const JobSet& v, int64_t blk) {
  constexpr int JW = 64 / W;
  constexpr int kSlots = JW * kWaves;
  constexpr int RSH = rec_shift(SMAX);
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1, lshift = 0;
  while (cp < a.C) cp <<= 1;
  while ((1 << lshift) < cp * SMAX * 8) ++lshift;
  unsigned char* sR = smem;                                                        // records
  double* sL = reinterpret_cast<double*>(sR + (size_t)kWaves * a.M * (1 << RSH));  // [M][Cp][SMAX]
  double* sTD = sL + (size_t)a.M * cp * SMAX;                      // chunk {t, deadline}
  uint32_t* sO = reinterpret_cast<uint32_t*>(sTD + 2 * kChunk);    // chunk record offsets

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int seg_lane = lane & (W - 1);
  const int64_t job = blk * kSlots + wave * JW + lane / W;
  const bool job_ok = job < v.J;

  SharedConst c;
  int p = 0;
  c.sigma = 0.0;
  if (job_ok) {
    p = (int)(job / a.K);
    c.sigma = a.slo_scale[job % a.K];
  }
  int cfg = -1;
  if (job_ok && seg_lane < v.G) cfg = v.group_cfg[(int64_t)p * v.G + seg_lane];
  if (cfg >= a.C || cfg < 0) cfg = -1;
  uint64_t hostbits = 0;  // bit m: this lane's group hosts model m
  if (cfg >= 0) {
    const uint64_t* hm = v.host_mask + (int64_t)p * a.M;
    for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> seg_lane) & 1u) << m;
  }
  int frow = -1;  // per-request output row of this job, -1 if none
  if (ROWS && job_ok)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == job) {
        frow = f;
        break;
      }
  c.fmask = __builtin_amdgcn_ballot_w64(frow >= 0);
  c.frowp = ROWS ? a.out_finish + (frow < 0 ? 0 : (int64_t)frow * a.n) : nullptr;
  c.flimit = a.n;
  const bool wave_finish = ROWS && c.fmask != 0;
  // a wavefront with per-request output has more to issue per request than
  // the others and sets the launch time: let it issue first on its SIMD
  if (wave_finish) __builtin_amdgcn_s_setprio(3);
  // one configuration for every group of the wavefront?
  const uint64_t valid = __builtin_amdgcn_ballot_w64(cfg >= 0);
  const int cfg0 = valid ? __builtin_amdgcn_readlane(cfg, __builtin_ctzll(valid)) : 0;
  const bool uni = __builtin_amdgcn_ballot_w64(cfg >= 0 && cfg != cfg0) == 0;
  c.lrow = sL + (cfg < 0 ? 0 : cfg) * SMAX;
  c.lshift = lshift;
  unsigned char* rec = sR + (size_t)wave * a.M * (1 << RSH);
  c.rec = rec;

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
  // this wavefront's model records
  for (int m = 0; m < a.M; ++m) {
    const uint64_t hm = __builtin_amdgcn_ballot_w64((hostbits >> m) & 1u);
    if (lane == 0) {
      const uint64_t one = lowest_per_field<W>(hm);  // lowest hosting lane of each job
      *(uint64_t*)(rec + ((size_t)m << RSH) + kRecMask) = hm;
      *(uint64_t*)(rec + ((size_t)m << RSH) + kRecCount) =
          one == hm ? 0u : (uint32_t)__builtin_popcountll(one);
    }
  }
  for (int m = lane; m < a.M; m += 64) {
    unsigned char* r = rec + ((size_t)m << RSH);
    // one scale: the SLO, scale * d_single[m] (one rounding); else d_single[m]
    *(double*)(r + rec_slo(SMAX)) = USIG ? a.slo_scale[0] * a.d_single[m] : a.d_single[m];
#pragma unroll
    for (int s = 0; s < SMAX; ++s)
      ((double*)(r + kRecLat))[s] = (uni && s < a.cfg_stages[cfg0])
                                        ? a.stage_lat[((int64_t)m * a.C + cfg0) * a.smax_in + s]
                                        : 0.0;
  }

  SharedLane<SMAX> st;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) st.F[s] = 0.0;
  st.fin_sum = st.hash = st.served = 0;
  st.wlo = 0;
  st.busy = 0.0;
  uint32_t* sCnt = sO + kChunk;  // STATS: [kWaves * JW][M]
  if constexpr (STATS) {
    for (int idx = lane; idx < JW * a.M; idx += 64) sCnt[(size_t)wave * JW * a.M + idx] = 0;
    c.cnt = sCnt + ((size_t)wave * JW + lane / W) * a.M;
    c.cntw = sCnt + (size_t)wave * JW * a.M;
    c.M = a.M;
  }

  const int64_t n = a.n;
  for (int64_t base = 0; base < n; base += kChunk) {
    const int cnt = (int)((n - base) < kChunk ? (n - base) : kChunk);
    __syncthreads();
    for (int e = tid; e < cnt; e += kThreads) {
      const double te = a.t[base + e];
      const uint32_t off = (uint32_t)a.model[base + e] << RSH;
      // one scale: the deadline t + SLO (one rounding) is the same for every
      // job; the SLO is read from wave 0's record (all waves hold it)
      const double de = USIG ? te + *(const double*)(sR + off + rec_slo(SMAX)) : te;
      *(double2*)(sTD + 2 * e) = make_double2(te, de);
      sO[e] = off;
    }
    __syncthreads();
    if constexpr (STATS) {
      // statistics launches carry no per-request output rows
      if (uni)
        fast_chunk<W, SMAX, USIG, false, false, true, true>(st, c, sTD, sO, cnt, base, n);
      else
        fast_chunk<W, SMAX, USIG, false, false, false, true>(st, c, sTD, sO, cnt, base, n);
    } else if (uni) {
      if (ROWS && wave_finish)
        fast_chunk<W, SMAX, USIG, ROWS, false, true>(st, c, sTD, sO, cnt, base, n);
      else
        fast_chunk<W, SMAX, USIG, false, false, true>(st, c, sTD, sO, cnt, base, n);
    } else {
      if (ROWS && wave_finish)
        fast_chunk<W, SMAX, USIG, ROWS, false, false>(st, c, sTD, sO, cnt, base, n);
      else
        fast_chunk<W, SMAX, USIG, false, false, false>(st, c, sTD, sO, cnt, base, n);
    }
  }

  const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum);
  if (job_ok && seg_lane == 0) {
    v.out_served[job] = (int64_t)st.served;
    if (v.out_attain) v.out_attain[job] = n > 0 ? (double)st.served / (double)n : 0.0;
    if (v.out_digest) {
      v.out_digest[2 * job] = st.hash;
      v.out_digest[2 * job + 1] = fin_sum;
    }
  }
  if constexpr (STATS) {
    if (job_ok && seg_lane < v.G && v.out_group_busy) v.out_group_busy[job * v.G + seg_lane] = st.busy;
    if (job_ok && v.out_model_served)
      for (int m = seg_lane; m < a.M; m += W) v.out_model_served[job * a.M + m] = (int64_t)c.cnt[m];
  }
}

template <int W, int SMAX, bool USIG, bool STATS = false>
__global__ __launch_bounds__(kThreads) void shared_kernel(const KArgs a) {
  if (a.gate && *a.gate == 0) return;
  shared_body<W, SMAX, USIG, STATS, true>(a, job_set(a), blockIdx.x);
}

// Multi-shape launches: consecutive block ranges run job sets of different
// shapes (lanes per job 2^wl, padded stages 2^sl), so that the jobs of
// several shapes share one dispatch instead of queueing behind each other.
constexpr int kMaxShapeSegs = 16;
struct ShapeSeg {
  int32_t wl, sl;
  int64_t block0;  // first block of the segment
  JobSet v;
};
struct MultiSegs {
  int32_t n;
  ShapeSeg s[kMaxShapeSegs];
};

// ---------------------------------------------------------------------------
// Segmented jobs with up to 64 groups: one job per wavefront (lane g = group
// g), each job simulating its own trace segment at its own SLO scale.  The
// requests of a wavefront are again the same in every lane, so the request
// loop above applies unchanged.  The job's SLOs (scale * d_single[m], one
// rounding) go into its model records, and each wavefront stages its own
// segment through its own LDS region -- deadline t + SLO and record offset
// per request -- with no workgroup barrier in the request loop.

constexpr int kSegChunk = 256;  // requests per staging round of one wavefront

// LDS bytes of seg_kernel: records, the stage-latency table, and each
// wavefront's chunk ({t, deadline} pairs, record offsets).
__host__ __device__ constexpr size_t seg_lds_bytes(int M, int Cp, int SMAX) {
  return (size_t)kWaves * M * ((size_t)1 << rec_shift(SMAX)) + (size_t)M * Cp * SMAX * 8 +
         (size_t)kWaves * kSegChunk * 20;
}

// Length and start of job j's segment: a record naming a missing placement or
// segment makes an empty job; bounds are clamped to [0, seg_off[n_segments]].
__device__ __forceinline__ void seg_job(const KArgs& a, int64_t j, int& p, double& sigma,
                                        int64_t& begin, int64_t& len) {
  const as_job_t jb = a.jobs[j];
  p = jb.placement;
  sigma = jb.slo_scale;
  begin = 0;
  len = 0;
  if (p < 0 || p >= a.P || jb.segment < 0 || jb.segment >= a.n_segments) {
    p = 0;
    return;
  }
  const int64_t total = a.seg_off[a.n_segments];
  int64_t b = a.seg_off[jb.segment], e = a.seg_off[jb.segment + 1];
  b = b < 0 ? 0 : (b > total ? total : b);
  e = e < b ? b : (e > total ? total : e);
  begin = b;
  len = e - b;
}

// Slot blockIdx.x * kWaves + wavefront runs job order[slot] (the slot itself
// without an order); with a slot counter (a.next_slot, 0 at launch) each
// wavefront instead takes slots in turn until none is left, so that a grid
// of fewer wavefronts than jobs works through a longest-first order.
// Per-request output rows must hold -2 over [0, min(segment length,
// finish_stride)) when the kernel starts.
template <int SMAX>
__global__ __launch_bounds__(kThreads) void seg_kernel(const KArgs a) {
  constexpr int W = 64;
  constexpr int RSH = rec_shift(SMAX);
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1, lshift = 0;
  while (cp < a.C) cp <<= 1;
  while ((1 << lshift) < cp * SMAX * 8) ++lshift;
  unsigned char* sR = smem;                                                        // records
  double* sL = reinterpret_cast<double*>(sR + (size_t)kWaves * a.M * (1 << RSH));  // [M][Cp][SMAX]
  double* sTDall = sL + (size_t)a.M * cp * SMAX;
  uint32_t* sOall = reinterpret_cast<uint32_t*>(sTDall + (size_t)kWaves * 2 * kSegChunk);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  double* sTD = sTDall + (size_t)wave * 2 * kSegChunk;
  uint32_t* sO = sOall + (size_t)wave * kSegChunk;
  unsigned char* rec = sR + (size_t)wave * a.M * (1 << RSH);

  // the stage-latency table, once per workgroup (the only barrier: after it
  // every wavefront goes its own way)
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
  __syncthreads();

  auto take_slot = [&]() -> int64_t {
    int v = 0;
    if (lane == 0) v = atomicAdd(a.next_slot, 1);
    return (int64_t)__builtin_amdgcn_readfirstlane(v);
  };
  int64_t slot = a.next_slot ? take_slot() : (int64_t)blockIdx.x * kWaves + wave;
  while (slot < a.J) {
    const int64_t job = a.order ? (int64_t)a.order[slot] : slot;
    int p = 0;
    double sigma = 0.0;
    int64_t begin = 0, n_job = 0;
    seg_job(a, job, p, sigma, begin, n_job);

    SharedConst c;
    c.sigma = sigma;
    int cfg = -1;
    if (lane < a.G) cfg = a.group_cfg[(int64_t)p * a.G + lane];
    if (cfg >= a.C || cfg < 0) cfg = -1;
    uint64_t hostbits = 0;  // bit m: this lane's group hosts model m
    if (cfg >= 0) {
      const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
      for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> lane) & 1u) << m;
    }
    int frow = -1;
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == job) {
        frow = f;
        break;
      }
    c.fmask = __builtin_amdgcn_ballot_w64(frow >= 0);
    c.frowp = a.out_finish + (frow < 0 ? 0 : (int64_t)frow * a.finish_stride);
    c.flimit = n_job < a.finish_stride ? n_job : a.finish_stride;
    const bool wave_finish = c.fmask != 0;
    // whether the row is shorter than the segment (else no per-request limit test)
    const bool row_lim = c.flimit < n_job;
    if (wave_finish)
      __builtin_amdgcn_s_setprio(3);
    else
      __builtin_amdgcn_s_setprio(0);
    const uint64_t valid = __builtin_amdgcn_ballot_w64(cfg >= 0);
    const int cfg0 = valid ? __builtin_amdgcn_readlane(cfg, __builtin_ctzll(valid)) : 0;
    const bool uni = __builtin_amdgcn_ballot_w64(cfg >= 0 && cfg != cfg0) == 0;
    c.lrow = sL + (cfg < 0 ? 0 : cfg) * SMAX;
    c.lshift = lshift;
    c.rec = rec;

    // this job's records: the previous job's reads of them are done (in-order
    // LDS within a wavefront; the fences keep the compiler from moving accesses)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    for (int m = 0; m < a.M; ++m) {
      const uint64_t hm = __builtin_amdgcn_ballot_w64((hostbits >> m) & 1u);
      if (lane == 0) {
        const uint64_t one = lowest_per_field<W>(hm);
        *(uint64_t*)(rec + ((size_t)m << RSH) + kRecMask) = hm;
        *(uint64_t*)(rec + ((size_t)m << RSH) + kRecCount) =
            one == hm ? 0u : (uint32_t)__builtin_popcountll(one);
      }
    }
    for (int m = lane; m < a.M; m += 64) {
      unsigned char* r = rec + ((size_t)m << RSH);
      // this job's SLO of model m: scale * d_single[m] (one rounding)
      *(double*)(r + rec_slo(SMAX)) = sigma * a.d_single[m];
#pragma unroll
      for (int s = 0; s < SMAX; ++s)
        ((double*)(r + kRecLat))[s] = (uni && s < a.cfg_stages[cfg0])
                                          ? a.stage_lat[((int64_t)m * a.C + cfg0) * a.smax_in + s]
                                          : 0.0;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    SharedLane<SMAX> st;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) st.F[s] = 0.0;
    st.fin_sum = st.hash = st.served = 0;
    st.wlo = 0;
    st.busy = 0.0;

    // the segment's arrivals are requested a chunk ahead: each round stages
    // the ones requested during the previous round, then requests the next
    constexpr int kPer = kSegChunk / 64;  // arrivals per lane and round
    double pt[kPer];
    int pm[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int64_t e = (int64_t)q * 64 + lane;
      pt[q] = e < n_job ? a.t[begin + e] : 0.0;
      pm[q] = e < n_job ? a.model[begin + e] : 0;
    }
    for (int64_t base = 0; base < n_job; base += kSegChunk) {
      const int cnt = (int)((n_job - base) < kSegChunk ? (n_job - base) : kSegChunk);
      // this wavefront's chunk: the previous one has been read (in-order LDS
      // within a wavefront; the fences keep the compiler from moving accesses)
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int e = q * 64 + lane;
        if (e < cnt) {
          const double te = pt[q];
          const uint32_t off = (uint32_t)pm[q] << RSH;
          const double de = te + *(const double*)(rec + off + rec_slo(SMAX));
          *(double2*)(sTD + 2 * e) = make_double2(te, de);
          sO[e] = off;
        }
      }
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int64_t e = base + kSegChunk + (int64_t)q * 64 + lane;
        pt[q] = e < n_job ? a.t[begin + e] : 0.0;
        pm[q] = e < n_job ? a.model[begin + e] : 0;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if (uni) {
        if (wave_finish && row_lim)
          fast_chunk<W, SMAX, true, true, true, true>(st, c, sTD, sO, cnt, base, n_job);
        else if (wave_finish)
          fast_chunk<W, SMAX, true, true, false, true>(st, c, sTD, sO, cnt, base, n_job);
        else
          fast_chunk<W, SMAX, true, false, false, true>(st, c, sTD, sO, cnt, base, n_job);
      } else {
        if (wave_finish && row_lim)
          fast_chunk<W, SMAX, true, true, true, false>(st, c, sTD, sO, cnt, base, n_job);
        else if (wave_finish)
          fast_chunk<W, SMAX, true, true, false, false>(st, c, sTD, sO, cnt, base, n_job);
        else
          fast_chunk<W, SMAX, true, false, false, false>(st, c, sTD, sO, cnt, base, n_job);
      }
    }

    const uint64_t fin_sum = seg_sum_u64<W>(st.fin_sum);
    if (lane == 0) {
      a.out_served[job] = (int64_t)st.served;
      if (a.out_attain) a.out_attain[job] = n_job > 0 ? (double)st.served / (double)n_job : 0.0;
      if (a.out_digest) {
        a.out_digest[2 * job] = st.hash;
        a.out_digest[2 * job + 1] = fin_sum;
      }
    }
    if (!a.next_slot) break;
    slot = take_slot();
  }
}

}  // namespace as_dev
