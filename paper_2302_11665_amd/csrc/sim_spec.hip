// Segment-speculative simulation of a shared trace: one lane per job, the
// trace cut into segments that run at the same time.
//
// The definition (Sec. 3.4, Sec. 4.3) is a recurrence over the requests of
// one job: request i is dispatched on the stage free times F left by request
// i-1.  A job's only parallelism is its groups, which the other kernels spread
// over lanes; most of those lanes then idle on every request (a model has one
// or two hosting groups, and only the chosen group runs the stage chain).
// Here one lane carries a whole job -- every lane does useful work on every
// request -- and the missing parallelism comes from the trace instead:
//
//   pass 0   every (job, segment) estimates its start state by simulating
//            the requests just before the segment from the empty state
//            (all F = 0), then runs the segment from that estimate,
//            recording its results and the state at its end;
//   round q  segment k whose recorded start state differs from the end state
//            segment k-1 now has re-runs its requests from that end state and,
//            in lockstep, from its old start state, until the two states are
//            equal bit for bit: from there on both runs take identical
//            decisions (the state is the only thing a request depends on
//            besides its own arrival), so the old results stand and only the
//            re-run prefix is replaced.  A segment whose runs never meet gets
//            a new end state, and its successor is revisited next round.
//   final    per job: served counts and finish-time sums add up over
//            segments; the digest's ordered hash runs over the accept bitmap.
//
// After round q segments 0..q hold exact results (segment 0 starts from the
// true empty state; each round settles at least the next one), so nseg - 1
// rounds always suffice; a round whose predecessor changed nothing returns at
// once.  Bursty arrivals make the speculation cheap: two runs of one job from
// different states become identical within a few thousand requests, so the
// warm-up estimate is usually exact and the rounds re-run little.
//
// State layout: F[g][s] of a lane lives in LDS as [g][s][lane] (conflict-free
// for any per-lane g); each lane's hosting masks live in registers (a uniform
// model index selects one); arrivals are uniform and read with scalar loads.
//
// Exactness: the same IEEE operations in the same order as the definition
// (v_max_f64, single v_add_f64, no FMA), so finish times are bit-identical.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_kernel.hpp"

namespace as_dev {
namespace {

constexpr int kSpecMaxSeg = 64;
constexpr uint64_t kSpecHashMul = 0x9E3779B97F4A7C15ULL;

struct SpecArgs {
  const double* t;
  const int32_t* model;
  int64_t n;
  const double* d_single;
  const double* stage_lat;
  const int32_t* group_cfg;
  const uint64_t* host_mask;
  const double* slo_scale;
  int64_t* out_served;
  double* out_attain;
  uint64_t* out_digest;
  double* out_finish;
  // workspace
  uint64_t* bitmap;     // [nw][J] accept bits, 64 requests per word
  double* st_start;     // [nseg][G*SMAX][J] start state behind each segment's results
  double* st_end;       // [2][nseg][G*SMAX][J] end states, alternating between rounds
  int64_t* seg_served;  // [nseg][J]
  uint64_t* seg_fsum;   // [nseg][J]
  int32_t* changed;     // [nseg] segments whose end state changed, per round
  int32_t* cfg_info;    // [2]: 1 when every used group has one configuration; that configuration
  int64_t nw;
  int64_t warmup;  // requests simulated before a segment to estimate its start state
  int32_t M, C, smax_in, G, K, J, n_finish, nseg, njb;
  int32_t cfg_stages[AS_MAX_CONFIGS];
  int32_t finish_jobs[AS_MAX_FINISH];
};

__device__ __forceinline__ int64_t seg_bound(int64_t n, int nseg, int k) {
  return k >= nseg ? n : ((n * k / nseg) & ~(int64_t)63);
}

__device__ __forceinline__ uint64_t bits_of(double x) { return (uint64_t)__double_as_longlong(x); }

// Hosting masks of one lane's placement for every model, MB bits per model,
// held in vector registers (32-dword vector values: a wavefront-uniform index
// into one lowers to indexed register moves, not memory).  With at most 16
// groups each model also has a host list: its lowest eight hosting groups as
// 4-bit fields in increasing order, unused fields repeating the lowest host.
typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));

// Element m (wavefront-uniform, < 64) of the 64-dword pair (x0, x1): one
// indexed register move per half, then a select of the two dwords (the empty
// asm keeps the compiler from selecting whole vectors first).
__device__ __forceinline__ uint32_t pick2(const u32x32& x0, const u32x32& x1, int m) {
  uint32_t a = x0[m & 31], b = x1[m & 31];
  asm volatile("" : "+v"(a), "+v"(b));
  return m < 32 ? a : b;
}

template <int MB>
struct LaneMasks {
  using MaskT = typename std::conditional<MB <= 32, uint32_t, uint64_t>::type;
  static constexpr int kVecs = 64 * MB / 32 / 32;  // 1, 2 or 4
  static constexpr int kListVecs = MB == 16 ? 2 : 0;
  u32x32 v[kVecs];
  u32x32 hl[kListVecs > 0 ? kListVecs : 1];
  // bits of groups >= G are dropped (they name no state)
  __device__ __forceinline__ void load(const uint64_t* row, int M, int G, bool valid) {
#pragma unroll
    for (int q = 0; q < kVecs; ++q) v[q] = (u32x32)(0u);
#pragma unroll
    for (int q = 0; q < (kListVecs > 0 ? kListVecs : 1); ++q) hl[q] = (u32x32)(0u);
    if (!valid) return;
    const uint64_t keep = G >= 64 ? ~0ull : (1ull << G) - 1;
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      const uint64_t x = m < M ? row[m] & keep : 0;
      if constexpr (MB == 16) {
        v[0][m >> 1] |= (uint32_t)(x & 0xFFFFu) << ((m & 1) * 16);
        uint32_t rest = (uint32_t)x, list = 0;
        const uint32_t low = rest ? (uint32_t)__builtin_ctz(rest) : 0u;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint32_t h = rest ? (uint32_t)__builtin_ctz(rest) : low;
          rest &= rest - 1;
          list |= h << (4 * q);
        }
        hl[m >> 5][m & 31] = list;
      } else if constexpr (MB == 32) {
        v[m >> 5][m & 31] = (uint32_t)x;
      } else {
        v[m >> 4][(2 * m) & 31] = (uint32_t)x;
        v[m >> 4][(2 * m + 1) & 31] = (uint32_t)(x >> 32);
      }
    }
  }
  // m is wavefront-uniform
  __device__ __forceinline__ MaskT get(int m) const {
    if constexpr (MB == 16) {
      return (v[0][m >> 1] >> ((m & 1) * 16)) & 0xFFFFu;
    } else if constexpr (MB == 32) {
      return pick2(v[0], v[1], m);
    } else {
      const int q = m >> 4, e = (2 * m) & 31;
      uint32_t lo = v[0][e], hi = v[0][e + 1];
      if (q == 1) {
        lo = v[1][e];
        hi = v[1][e + 1];
      } else if (q == 2) {
        lo = v[2][e];
        hi = v[2][e + 1];
      } else if (q == 3) {
        lo = v[3][e];
        hi = v[3][e + 1];
      }
      return (uint64_t)lo | ((uint64_t)hi << 32);
    }
  }
  __device__ __forceinline__ uint32_t list(int m) const {
    if constexpr (MB == 16) {
      return pick2(hl[0], hl[1], m);
    } else {
      return 0;
    }
  }
};

template <typename T>
__device__ __forceinline__ int ctz_any(T x) {
  if constexpr (sizeof(T) == 4) {
    return (int)__builtin_ctz(x);
  } else {
    return (int)__builtin_ctzll(x);
  }
}

// Per-wavefront LDS: the stage-latency table and per-lane group
// configurations when groups differ, then one or two state regions.
template <int SMAX, bool UCFG>
struct SpecLds {
  double* L;      // !UCFG: [M][C][SMAX]
  uint16_t* cfg;  // !UCFG: [G][64] = c | S << 8
  double* F0;     // [G][SMAX][64]
  double* F1;     // second state (rounds)
};

__host__ __device__ constexpr size_t spec_lds_bytes(int M, int C, int G, int SMAX, bool ucfg, int states) {
  return (ucfg ? 0 : (size_t)M * C * SMAX * 8 + (size_t)G * 64 * 2) + (size_t)states * G * SMAX * 64 * 8;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), l);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), l);
  return __hiloint2double(hi, lo);
}

template <int SMAX, bool UCFG>
__device__ __forceinline__ SpecLds<SMAX, UCFG> spec_tables(const SpecArgs& a, double* lds, int lane, int p,
                                                           bool valid, int states) {
  SpecLds<SMAX, UCFG> s;
  double* after = lds;
  s.L = nullptr;
  s.cfg = nullptr;
  if constexpr (!UCFG) {
    const int M = a.M, C = a.C;
    s.L = lds;
    s.cfg = reinterpret_cast<uint16_t*>(s.L + (size_t)M * C * SMAX);
    after = reinterpret_cast<double*>(s.cfg + (size_t)a.G * 64);
    // stage latencies (0 beyond S_c: never used)
    for (int e = lane; e < M * C * SMAX; e += 64) {
      const int k = e % SMAX;
      const int c = (e / SMAX) % C;
      const int m = e / (SMAX * C);
      s.L[e] = k < a.cfg_stages[c] ? a.stage_lat[((int64_t)m * C + c) * a.smax_in + k] : 0.0;
    }
    for (int g = 0; g < a.G; ++g) {
      int c = valid ? a.group_cfg[(int64_t)p * a.G + g] : -1;
      if (c < 0 || c >= C) c = 0;  // a group hosting nothing is never chosen
      s.cfg[g * 64 + lane] = (uint16_t)(c | (a.cfg_stages[c] << 8));
    }
  }
  s.F0 = after;
  s.F1 = states > 1 ? s.F0 + (size_t)a.G * SMAX * 64 : nullptr;
  __syncthreads();
  return s;
}

// Uniform data of one request: arrival, model, its SLO base d_single[m] and
// (uniform configuration) its stage latencies, the last two read with scalar
// loads (the tables are read-only for the whole launch).
template <int SMAX, bool UCFG>
struct Req {
  double t;
  int m;
  double L[UCFG ? SMAX : 1];
  double d;
};

typedef const __attribute__((address_space(4))) double* const_f64_ptr;

template <int SMAX, bool UCFG>
__device__ __forceinline__ void req_tables(const SpecArgs& a, int c0, int S0, Req<SMAX, UCFG>& q) {
  const int mi = (unsigned)q.m < (unsigned)a.M ? q.m : 0;
  const const_f64_ptr dc = (const_f64_ptr)a.d_single;
  q.d = dc[mi];
  if constexpr (UCFG) {
    // stages past S0 read stage 0 again (their result is never used)
    const const_f64_ptr Lc = (const_f64_ptr)a.stage_lat;
    const int base = (mi * a.C + c0) * a.smax_in;  // < 64 * 32 * 8
#pragma unroll
    for (int k = 0; k < SMAX; ++k) q.L[k] = Lc[base + (k < S0 ? k : 0)];
  }
}

// One request of one lane on the state F: dispatch (least stage-0 free time
// among the hosting groups, lowest index on ties), stage chain, admission
// (finish <= t + scale * d_single[m]), commit.  Returns the finish time (-1
// dropped, -2 no hosting group) and the chosen group in gs (-1 when nothing
// was committed).  The LDS reads of a request go out together: the rows of
// the two lowest hosting groups and, when some lane of the wavefront has
// more hosts, the stage-0 entries of up to six more; a row is read again only
// when one of those wins.
template <int SMAX, bool UCFG, int MB>
__device__ __forceinline__ double spec_step(const SpecLds<SMAX, UCFG>& s, double* F, int lane,
                                            typename LaneMasks<MB>::MaskT mask, uint32_t hlist,
                                            const Req<SMAX, UCFG>& r, double scale, int C, int S0, int& gs) {
  using MaskT = typename LaneMasks<MB>::MaskT;
  constexpr int kX = 6;
  gs = -1;
  if (mask == 0) return -2.0;
  int g0, g1;
  MaskT rest;  // hosts after the eighth (host lists) or after the second
  bool more;   // this lane has a third host
  int hx[kX];
  if constexpr (MB == 16) {
    g0 = (int)(hlist & 15u);
    g1 = (int)((hlist >> 4) & 15u);
    const int cnt = __builtin_popcount((uint32_t)mask);
    more = cnt > 2;
#pragma unroll
    for (int q = 0; q < kX; ++q) hx[q] = (int)((hlist >> (4 * (q + 2))) & 15u);
    rest = 0;
    if (cnt > 8) {
      rest = mask;
#pragma unroll
      for (int q = 0; q < 8; ++q) rest &= rest - 1;
    }
  } else {
    g0 = ctz_any(mask);
    const MaskT r1 = mask & (mask - 1);
    g1 = r1 ? ctz_any(r1) : g0;
    rest = r1 & (r1 - 1);
    more = rest != 0;
  }
  const bool extra = __builtin_amdgcn_ballot_w64(more) != 0;
  if constexpr (MB != 16) {
    if (extra) {
#pragma unroll
      for (int q = 0; q < kX; ++q) {
        hx[q] = rest ? ctz_any(rest) : g0;
        rest &= rest - 1;
      }
    }
  }
  double A[SMAX], B[SMAX], X[kX];
#pragma unroll
  for (int k = 0; k < SMAX; ++k) {
    A[k] = F[(g0 * SMAX + k) * 64 + lane];
    B[k] = F[(g1 * SMAX + k) * 64 + lane];
  }
  if (extra) {
#pragma unroll
    for (int q = 0; q < kX; ++q) X[q] = F[(hx[q] * SMAX) * 64 + lane];
  }
  // g1 > g0, and further hosts come in increasing order: strict comparisons
  // keep the lowest index among equal free times
  const bool use_b = B[0] < A[0];
  int g = use_b ? g1 : g0;
  double Fv[SMAX];
#pragma unroll
  for (int k = 0; k < SMAX; ++k) Fv[k] = use_b ? B[k] : A[k];
  if (extra) {
    double best = Fv[0];
#pragma unroll
    for (int q = 0; q < kX; ++q) {
      if (X[q] < best) {
        best = X[q];
        g = hx[q];
      }
    }
    while (rest) {  // more than eight hosts
      const int h = ctz_any(rest);
      rest &= rest - 1;
      const double v = F[(h * SMAX) * 64 + lane];
      if (v < best) {
        best = v;
        g = h;
      }
    }
    if (g != g0 && g != g1) {
#pragma unroll
      for (int k = 0; k < SMAX; ++k) Fv[k] = F[(g * SMAX + k) * 64 + lane];
    }
  }
  double Lv[SMAX];
  int S = S0;
  if constexpr (UCFG) {
#pragma unroll
    for (int k = 0; k < SMAX; ++k) Lv[k] = r.L[k];
  } else {
    const uint32_t e = s.cfg[g * 64 + lane];
    const int c = (int)(e & 0xFF);
    S = (int)(e >> 8);
    const double* Lrow = s.L + ((size_t)r.m * C + c) * SMAX;
#pragma unroll
    for (int k = 0; k < SMAX; ++k) Lv[k] = Lrow[k];
  }
  // projection through the stage chain; stages past S keep their state
  double f[SMAX];
  double prev = r.t;
  if (UCFG && S == SMAX) {
#pragma unroll
    for (int k = 0; k < SMAX; ++k) {
      f[k] = vmax(prev, Fv[k]) + Lv[k];
      prev = f[k];
    }
  } else {
#pragma unroll
    for (int k = 0; k < SMAX; ++k) {
      const double x = vmax(prev, Fv[k]) + Lv[k];
      const bool in = k < S;
      f[k] = in ? x : Fv[k];
      prev = in ? x : prev;
    }
  }
  const double slo = scale * r.d;
  const double deadline = r.t + slo;
  if (prev > deadline) return -1.0;
#pragma unroll
  for (int k = 0; k < SMAX; ++k) F[(g * SMAX + k) * 64 + lane] = f[k];
  gs = g;
  return prev;
}

struct SpecLane {
  int job, p, frow;
  bool valid;
  double scale;
};

__device__ __forceinline__ SpecLane spec_lane(const SpecArgs& a, int jb, int lane) {
  SpecLane l;
  l.job = jb * 64 + lane;
  l.valid = l.job < a.J;
  l.p = l.valid ? l.job / a.K : 0;
  l.scale = l.valid ? a.slo_scale[l.job % a.K] : 0.0;
  l.frow = -1;
  if (l.valid)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == l.job) l.frow = f;
  return l;
}

// Arrivals in chunks of 64 (lane r holds request base + r); the next chunk is
// loaded while the current one is simulated.
struct TraceChunks {
  double tv, tn;
  int mv, mn;
  __device__ __forceinline__ void first(const SpecArgs& a, int64_t b, int64_t e, int lane) {
    const int64_t i = b + lane;
    tn = i < e ? a.t[i] : 0.0;
    mn = i < e ? a.model[i] : 0;
  }
  __device__ __forceinline__ void advance(const SpecArgs& a, int64_t next_base, int64_t e, int lane) {
    tv = tn;
    mv = mn;
    const int64_t i = next_base + lane;
    tn = i < e ? a.t[i] : 0.0;
    mn = i < e ? a.model[i] : 0;
  }
  template <int SMAX, bool UCFG>
  __device__ __forceinline__ Req<SMAX, UCFG> get(const SpecArgs& a, int r, int c0, int S0) const {
    Req<SMAX, UCFG> q;
    q.t = readlane_f64(tv, r);
    q.m = __builtin_amdgcn_readlane(mv, r);
    req_tables<SMAX, UCFG>(a, c0, S0, q);
    return q;
  }
};

// Pass 0: every (job, segment) from the empty state.
template <int SMAX, int MB, bool UCFG>
__global__ __launch_bounds__(64) void spec_pass0(const SpecArgs a) {
  // both variants are launched; the one that does not match the placements
  // returns at once
  if ((a.cfg_info[0] != 0) != UCFG) return;
  const int c0 = UCFG ? a.cfg_info[1] : 0;
  extern __shared__ double lds[];
  const int lane = threadIdx.x;
  const int jb = blockIdx.x % a.njb;
  const int k = blockIdx.x / a.njb;
  const SpecLane ln = spec_lane(a, jb, lane);
  LaneMasks<MB> msk;
  msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  const auto s = spec_tables<SMAX, UCFG>(a, lds, lane, ln.p, ln.valid, 1);
  const int GS = a.G * SMAX;
  for (int q = 0; q < GS; ++q) s.F0[q * 64 + lane] = 0.0;
  const int S0 = UCFG ? a.cfg_stages[c0] : 0;
  const bool wave_rows = __builtin_amdgcn_ballot_w64(ln.frow >= 0) != 0;
  if (blockIdx.x == 0 && lane < a.nseg) a.changed[lane] = lane == 0 ? 1 : 0;

  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  const int64_t J = a.J;
  // warm-up: the requests just before the segment, from the empty state, give
  // its start state (usually already the exact one: the rounds then find
  // nothing to redo)
  const int64_t w0 = b > a.warmup ? b - a.warmup : 0;
  if (k > 0 && w0 < b) {
    TraceChunks tw;
    tw.first(a, w0, b, lane);
    for (int64_t cb = w0; cb < b; cb += 64) {
      tw.advance(a, cb + 64, b, lane);
      const int cnt = (int)(b - cb < 64 ? b - cb : 64);
      for (int r = 0; r < cnt; ++r) {
        const Req<SMAX, UCFG> rq = tw.template get<SMAX, UCFG>(a, r, c0, S0);
        const bool known = (unsigned)rq.m < (unsigned)a.M;
        const typename LaneMasks<MB>::MaskT mask = known ? msk.get(rq.m) : 0;
        const uint32_t hl = known ? msk.list(rq.m) : 0u;
        int gs;
        (void)spec_step<SMAX, UCFG, MB>(s, s.F0, lane, mask, hl, rq, ln.scale, a.C, S0, gs);
      }
    }
  }
  const size_t seg_base = ((size_t)k * GS) * J + ln.job;
  if (ln.valid)
    for (int q = 0; q < GS; ++q) a.st_start[seg_base + (size_t)q * J] = s.F0[q * 64 + lane];
  int64_t served = 0;
  uint64_t fsum = 0;
  TraceChunks tc;
  tc.first(a, b, e, lane);
  for (int64_t cb = b; cb < e; cb += 64) {
    tc.advance(a, cb + 64, e, lane);
    const int cnt = (int)(e - cb < 64 ? e - cb : 64);
    uint64_t word = 0;
    for (int r = 0; r < cnt; ++r) {
      const Req<SMAX, UCFG> rq = tc.template get<SMAX, UCFG>(a, r, c0, S0);
      int gs;
      const bool known = (unsigned)rq.m < (unsigned)a.M;
        const typename LaneMasks<MB>::MaskT mask = known ? msk.get(rq.m) : 0;
        const uint32_t hl = known ? msk.list(rq.m) : 0u;
      const double out = spec_step<SMAX, UCFG, MB>(s, s.F0, lane, mask, hl, rq, ln.scale, a.C, S0, gs);
      if (gs >= 0) {
        served += 1;
        fsum += bits_of(out);
        word |= 1ull << r;
      }
      if (wave_rows && ln.frow >= 0) a.out_finish[(int64_t)ln.frow * a.n + cb + r] = out;
    }
    if (ln.valid) a.bitmap[(cb >> 6) * J + ln.job] = word;
  }
  if (!ln.valid) return;
  for (int q = 0; q < GS; ++q) a.st_end[seg_base + (size_t)q * J] = s.F0[q * 64 + lane];  // buffer 0
  a.seg_served[(size_t)k * J + ln.job] = served;
  a.seg_fsum[(size_t)k * J + ln.job] = fsum;
}

// Round q >= 1: segments whose start state is stale re-run in lockstep with
// their old start until the two states meet.
template <int SMAX, int MB, bool UCFG>
__global__ __launch_bounds__(64) void spec_round(const SpecArgs a, int q) {
  if ((a.cfg_info[0] != 0) != UCFG) return;
  if (a.changed[q - 1] == 0) return;  // nothing moved in the previous round: done
  const int c0 = UCFG ? a.cfg_info[1] : 0;
  extern __shared__ double lds[];
  const int lane = threadIdx.x;
  const int jb = blockIdx.x % a.njb;
  const int k = blockIdx.x / a.njb;
  const SpecLane ln = spec_lane(a, jb, lane);
  const int GS = a.G * SMAX;
  const int64_t J = a.J;
  const size_t per_buf = (size_t)a.nseg * GS * J;
  const double* E_in = a.st_end + (size_t)((q - 1) & 1) * per_buf;
  double* E_out = a.st_end + (size_t)(q & 1) * per_buf;
  const size_t own = ((size_t)k * GS) * J + ln.job;
  const size_t prv = k > 0 ? ((size_t)(k - 1) * GS) * J + ln.job : 0;

  // the start state behind this segment's results versus the end state of
  // its predecessor
  bool active = false;
  if (ln.valid && k > 0)
    for (int x = 0; x < GS; ++x)
      active |= bits_of(a.st_start[own + (size_t)x * J]) != bits_of(E_in[prv + (size_t)x * J]);
  const bool ran = active;
  if (__builtin_amdgcn_ballot_w64(active) == 0) {
    if (ln.valid)
      for (int x = 0; x < GS; ++x) E_out[own + (size_t)x * J] = E_in[own + (size_t)x * J];
    return;
  }
  LaneMasks<MB> msk;
  msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  const auto s = spec_tables<SMAX, UCFG>(a, lds, lane, ln.p, ln.valid, 2);
  const int S0 = UCFG ? a.cfg_stages[c0] : 0;
  const bool wave_rows = __builtin_amdgcn_ballot_w64(ln.frow >= 0) != 0;
  // F0: old run (from the stale start), F1: new run (from the predecessor's end)
  uint64_t diff = 0;  // groups whose states differ
  for (int x = 0; x < GS; ++x) {
    const double o = active ? a.st_start[own + (size_t)x * J] : 0.0;
    const double nv = active ? E_in[prv + (size_t)x * J] : 0.0;
    s.F0[x * 64 + lane] = o;
    s.F1[x * 64 + lane] = nv;
    if (bits_of(o) != bits_of(nv)) diff |= 1ull << (x / SMAX);
  }
  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  int64_t d_served = 0;
  uint64_t d_fsum = 0;
  bool coupled = false;
  TraceChunks tc;
  tc.first(a, b, e, lane);
  for (int64_t cb = b; cb < e; cb += 64) {
    if (__builtin_amdgcn_ballot_w64(active) == 0) break;
    tc.advance(a, cb + 64, e, lane);
    const int cnt = (int)(e - cb < 64 ? e - cb : 64);
    uint64_t word = 0;
    const bool part = active;  // this lane re-runs (part of) this chunk
    int stop = cnt;            // its first request left to the old run
    for (int r = 0; r < cnt; ++r) {
      if (__builtin_amdgcn_ballot_w64(active) == 0) break;
      const Req<SMAX, UCFG> rq = tc.template get<SMAX, UCFG>(a, r, c0, S0);
      if (active) {
        const bool known = (unsigned)rq.m < (unsigned)a.M;
        const typename LaneMasks<MB>::MaskT mask = known ? msk.get(rq.m) : 0;
        const uint32_t hl = known ? msk.list(rq.m) : 0u;
        int go, gn;
        const double oo = spec_step<SMAX, UCFG, MB>(s, s.F0, lane, mask, hl, rq, ln.scale, a.C, S0, go);
        const double on = spec_step<SMAX, UCFG, MB>(s, s.F1, lane, mask, hl, rq, ln.scale, a.C, S0, gn);
        d_served += (gn >= 0) - (go >= 0);
        d_fsum += (gn >= 0 ? bits_of(on) : 0) - (go >= 0 ? bits_of(oo) : 0);
        if (gn >= 0) word |= 1ull << r;
        if (wave_rows && ln.frow >= 0) a.out_finish[(int64_t)ln.frow * a.n + cb + r] = on;
        // refresh the difference bits of the groups the two runs touched
#pragma unroll
        for (int w = 0; w < 2; ++w) {
          const int g = w == 0 ? go : gn;
          if (g < 0) continue;
          bool same = true;
#pragma unroll
          for (int st = 0; st < SMAX; ++st)
            same &= bits_of(s.F0[(g * SMAX + st) * 64 + lane]) == bits_of(s.F1[(g * SMAX + st) * 64 + lane]);
          diff = same ? diff & ~(1ull << g) : diff | (1ull << g);
        }
        if (diff == 0) {
          coupled = true;
          active = false;
          stop = r + 1;
        }
      }
    }
    // accept bits of this chunk: the new run's before the lane's stop, the
    // old run's (already stored) from there on
    if (part) {
      uint64_t* wp = a.bitmap + (cb >> 6) * J + ln.job;
      if (stop >= cnt) {
        *wp = word;
      } else {
        const uint64_t low = (1ull << stop) - 1;
        *wp = (*wp & ~low) | word;
      }
    }
  }
  if (!ln.valid) return;
  if (ran) {
    // the predecessor's end state now stands behind this segment's results
    for (int x = 0; x < GS; ++x) a.st_start[own + (size_t)x * J] = E_in[prv + (size_t)x * J];
    a.seg_served[(size_t)k * J + ln.job] += d_served;
    a.seg_fsum[(size_t)k * J + ln.job] += d_fsum;
    if (!coupled) {
      // the runs never met: the segment ends in the new run's state
      for (int x = 0; x < GS; ++x) E_out[own + (size_t)x * J] = s.F1[x * 64 + lane];
      atomicAdd(a.changed + q, 1);
      return;
    }
  }
  for (int x = 0; x < GS; ++x) E_out[own + (size_t)x * J] = E_in[own + (size_t)x * J];
}

// Per job: totals over segments and the ordered digest over the accept words.
__global__ __launch_bounds__(64) void spec_final(const SpecArgs a) {
  const int64_t job = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (job >= a.J) return;
  const int64_t J = a.J;
  int64_t served = 0;
  uint64_t fsum = 0;
  for (int k = 0; k < a.nseg; ++k) {
    served += a.seg_served[(size_t)k * J + job];
    fsum += a.seg_fsum[(size_t)k * J + job];
  }
  uint64_t h = 0;
  const uint64_t* col = a.bitmap + job;
  int64_t w = 0;
  for (; w + 4 <= a.nw; w += 4) {
    const uint64_t x0 = col[(w + 0) * J], x1 = col[(w + 1) * J], x2 = col[(w + 2) * J], x3 = col[(w + 3) * J];
    h = (h ^ x0) * kSpecHashMul;
    h = (h ^ x1) * kSpecHashMul;
    h = (h ^ x2) * kSpecHashMul;
    h = (h ^ x3) * kSpecHashMul;
  }
  for (; w < a.nw; ++w) h = (h ^ col[w * J]) * kSpecHashMul;
  a.out_served[job] = served;
  if (a.out_attain) a.out_attain[job] = a.n > 0 ? (double)served / (double)a.n : 0.0;
  if (a.out_digest) {
    a.out_digest[2 * job] = h;
    a.out_digest[2 * job + 1] = fsum;
  }
}

}  // namespace
}  // namespace as_dev

namespace as_dev {
namespace {

// Whether every group that a placement uses (configuration >= 0) has one and
// the same configuration; cfg_info = {uniform, that configuration}.  One
// workgroup of 1024 threads.
__global__ __launch_bounds__(1024) void spec_cfg_check(const int32_t* group_cfg, int64_t cells, int n_configs,
                                                       int32_t* cfg_info) {
  __shared__ int lo[1024], hi[1024];
  int l = 0x7FFFFFFF, h = -1;
  for (int64_t i = threadIdx.x; i < cells; i += 1024) {
    const int c = group_cfg[i];
    if (c >= 0) {
      l = c < l ? c : l;
      h = c > h ? c : h;
    }
  }
  lo[threadIdx.x] = l;
  hi[threadIdx.x] = h;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      lo[threadIdx.x] = min(lo[threadIdx.x], lo[threadIdx.x + w]);
      hi[threadIdx.x] = max(hi[threadIdx.x], hi[threadIdx.x + w]);
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const bool none = hi[0] < 0;
    // configurations >= n_configs are invalid input: such calls take the
    // per-lane tables, which clamp them
    cfg_info[0] = none || (lo[0] == hi[0] && lo[0] < n_configs) ? 1 : 0;
    cfg_info[1] = none ? 0 : lo[0];
  }
}

template <int SMAX, int MB>
hipError_t spec_launch_all(const SpecArgs& a, size_t lds_u, size_t lds_g, size_t lds2_u, size_t lds2_g,
                           hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)a.njb * a.nseg)), block(64);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, true>), grid, block, lds_u, s, a);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, false>), grid, block, lds_g, s, a);
  for (int q = 1; q < a.nseg; ++q) {
    hipLaunchKernelGGL((spec_round<SMAX, MB, true>), grid, block, lds2_u, s, a, q);
    hipLaunchKernelGGL((spec_round<SMAX, MB, false>), grid, block, lds2_g, s, a, q);
  }
  hipLaunchKernelGGL(spec_final, dim3((unsigned)((a.J + 63) / 64)), block, 0, s, a);
  return hipGetLastError();
}

// Workgroups (one wavefront each) of the pass-0 kernel that one compute unit
// holds at this LDS size.
template <int SMAX, int MB>
int spec_occupancy(size_t lds) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, spec_pass0<SMAX, MB, true>, 64, lds) != hipSuccess)
    return 1;
  return nb > 0 ? nb : 1;
}

template <int SMAX>
int spec_occupancy_mb(int G, size_t lds) {
  if (G <= 16) return spec_occupancy<SMAX, 16>(lds);
  if (G <= 32) return spec_occupancy<SMAX, 32>(lds);
  return spec_occupancy<SMAX, 64>(lds);
}

template <int SMAX>
hipError_t spec_launch_mb(int G, const SpecArgs& a, size_t l1, size_t l2, size_t l3, size_t l4, hipStream_t s) {
  if (G <= 16) return spec_launch_all<SMAX, 16>(a, l1, l2, l3, l4, s);
  if (G <= 32) return spec_launch_all<SMAX, 32>(a, l1, l2, l3, l4, s);
  return spec_launch_all<SMAX, 64>(a, l1, l2, l3, l4, s);
}

}  // namespace
}  // namespace as_dev

namespace as_host {

namespace {

int compute_units() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cache[dev] = v;
  }
  return cache[dev];
}

// Keep freed stream-ordered allocations in the device's pool (the workspace
// of one call is reused by the next instead of going back to the driver).
void keep_pool_memory() {
  static bool done[64] = {false};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64 || done[dev]) return;
  hipMemPool_t pool;
  if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
    uint64_t thr = UINT64_MAX;
    (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &thr);
  }
  done[dev] = true;
}

constexpr int64_t kSpecMinSegment = 32768;  // requests per segment by default
constexpr int64_t kSpecWarmup = 32768;      // warm-up requests before a segment

}  // namespace

// Segments per job for the speculative path: enough (job block, segment)
// wavefronts to fill the device at the occupancy the LDS allows, each segment
// long enough that its lockstep prefix is a small part of it.
// ALPASERVE_SPEC_SEGMENTS forces the count (tests).
int spec_segments(int64_t n, int64_t J, int per_cu) {
  if (const char* e = getenv("ALPASERVE_SPEC_SEGMENTS")) {
    const int v = atoi(e);
    if (v >= 1) return std::min(v, as_dev::kSpecMaxSeg);
  }
  const int64_t slots = (int64_t)compute_units() * std::max(per_cu, 1);
  const int64_t njb = (J + 63) / 64;
  int64_t k = slots / std::max<int64_t>(njb, 1);
  k = std::min<int64_t>(k, n / kSpecMinSegment);
  return (int)std::max<int64_t>(1, std::min<int64_t>(k, as_dev::kSpecMaxSeg));
}

// Shared-trace simulation on the segment-speculative kernels.  Returns
// AS_E_LIMITS without launching when the state of one wavefront (two, in the
// lockstep rounds) does not fit in the LDS.
int run_spec(KArgs& k, int smax, hipStream_t stream) {
  using namespace as_dev;
  if (k.n <= 0 || k.J <= 0) return AS_E_LIMITS;
  const size_t lim = shared_lds_limit();
  const size_t lds_u = spec_lds_bytes(k.M, k.C, k.G, smax, true, 1);
  const size_t lds_g = spec_lds_bytes(k.M, k.C, k.G, smax, false, 1);
  const size_t lds2_u = spec_lds_bytes(k.M, k.C, k.G, smax, true, 2);
  const size_t lds2_g = spec_lds_bytes(k.M, k.C, k.G, smax, false, 2);
  if (lds2_g > lim) return AS_E_LIMITS;

  SpecArgs a;
  std::memset(&a, 0, sizeof a);
  a.t = k.t;
  a.model = k.model;
  a.n = k.n;
  a.d_single = k.d_single;
  a.stage_lat = k.stage_lat;
  a.group_cfg = k.group_cfg;
  a.host_mask = k.host_mask;
  a.slo_scale = k.slo_scale;
  a.out_served = k.out_served;
  a.out_attain = k.out_attain;
  a.out_digest = k.out_digest;
  a.out_finish = k.out_finish;
  a.M = k.M;
  a.C = k.C;
  a.smax_in = k.smax_in;
  a.G = k.G;
  a.K = k.K;
  a.J = k.J;
  a.n_finish = k.n_finish;
  std::memcpy(a.cfg_stages, k.cfg_stages, sizeof a.cfg_stages);
  std::memcpy(a.finish_jobs, k.finish_jobs, sizeof a.finish_jobs);
  a.njb = (int32_t)((k.J + 63) / 64);
  int per_cu = 1;
  switch (smax) {
    case 1: per_cu = spec_occupancy_mb<1>(k.G, lds_u); break;
    case 2: per_cu = spec_occupancy_mb<2>(k.G, lds_u); break;
    case 4: per_cu = spec_occupancy_mb<4>(k.G, lds_u); break;
    default: per_cu = spec_occupancy_mb<8>(k.G, lds_u); break;
  }
  a.nseg = spec_segments(k.n, k.J, per_cu);
  a.warmup = kSpecWarmup;
  if (const char* w = getenv("ALPASERVE_SPEC_WARMUP")) a.warmup = std::max<int64_t>(0, atoll(w));
  while (a.nseg > 1 && (int64_t)a.njb * a.nseg > 0x7FFFFFFFLL) --a.nseg;
  if ((int64_t)a.njb * a.nseg > 0x7FFFFFFFLL) return AS_E_LIMITS;
  a.nw = (k.n + 63) / 64;

  const int64_t J = k.J, GS = (int64_t)k.G * smax;
  const size_t b_bitmap = (size_t)a.nw * J * 8;
  const size_t b_state = (size_t)a.nseg * GS * J * 8;
  const size_t b_seg = (size_t)a.nseg * J * 8;
  const size_t b_small = 256 + (size_t)a.nseg * 4;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t total = up(b_bitmap) + up(b_state) + up(2 * b_state) + 2 * up(b_seg) + up(b_small);
  // a workspace beyond a quarter of the device's memory leaves the call to
  // the kernels that need none
  size_t free_b = 0, total_b = 0;
  if (hipMemGetInfo(&free_b, &total_b) != hipSuccess || total > total_b / 4) return AS_E_LIMITS;
  keep_pool_memory();
  char* ws = nullptr;
  hipError_t e = hipMallocAsync(reinterpret_cast<void**>(&ws), total, stream);
  if (e != hipSuccess || !ws)
    return fail(AS_E_NOMEM, "workspace of %zu bytes: %s", total, hipGetErrorString(e));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = ws + off;
    off += up(bytes);
    return p;
  };
  a.bitmap = reinterpret_cast<uint64_t*>(take(b_bitmap));
  a.st_start = reinterpret_cast<double*>(take(b_state));
  a.st_end = reinterpret_cast<double*>(take(2 * b_state));
  a.seg_served = reinterpret_cast<int64_t*>(take(b_seg));
  a.seg_fsum = reinterpret_cast<uint64_t*>(take(b_seg));
  int32_t* small = reinterpret_cast<int32_t*>(take(b_small));
  a.cfg_info = small;
  a.changed = small + 64;

  hipLaunchKernelGGL(spec_cfg_check, dim3(1), dim3(1024), 0, stream, k.group_cfg, (int64_t)k.P * k.G, k.C,
                     a.cfg_info);
  switch (smax) {
    case 1: e = spec_launch_mb<1>(k.G, a, lds_u, lds_g, lds2_u, lds2_g, stream); break;
    case 2: e = spec_launch_mb<2>(k.G, a, lds_u, lds_g, lds2_u, lds2_g, stream); break;
    case 4: e = spec_launch_mb<4>(k.G, a, lds_u, lds_g, lds2_u, lds2_g, stream); break;
    default: e = spec_launch_mb<8>(k.G, a, lds_u, lds_g, lds2_u, lds2_g, stream); break;
  }
  const hipError_t ef = hipFreeAsync(ws, stream);
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  if (ef != hipSuccess) return fail(AS_E_HIP, "workspace release failed: %s", hipGetErrorString(ef));
  return ok();
}

}  // namespace as_host
