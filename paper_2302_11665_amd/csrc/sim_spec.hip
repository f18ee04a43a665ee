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
//            segment k-1 now has re-runs its requests from that end state
//            until its state equals, bit for bit, the state its current
//            results had at the same request (pass 0 saves the state every
//            few thousand requests): from there on both runs take identical
//            decisions (the state is the only thing a request depends on
//            besides its own arrival), so the old results stand and only the
//            re-run prefix is replaced.  A segment whose runs never meet gets
//            a new end state, and its successor is revisited next round.
//            A round re-runs few jobs and lasts as long as the longest
//            re-run, so for jobs of at most 16 groups it runs in a
//            group-per-lane layout (a job's groups on W lanes, state in
//            registers, DPP min dispatch), whose per-request chain is shorter.
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
// for any per-lane g), with a spare row that unserved requests write and a
// sentinel row that stands for a missing host; each lane's hosting masks live
// in registers (a uniform model index selects one); arrivals come in chunks
// of 64, one per lane, and a request is read from its lane with readlane.
//
// Exactness: the same IEEE operations in the same order as the definition
// (v_max_f64, single v_add_f64, no FMA), so finish times are bit-identical.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <type_traits>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_kernel.hpp"
#include "sim_shared.hpp"

namespace as_dev {
namespace {

constexpr int kSpecMaxSeg = 64;
// A reconciliation re-run that has not met the old results after this many
// requests gives up, and the call falls back to the shared-trace kernels.  On
// bursty traffic runs from different states meet within a few thousand
// requests (on the 8192-placement heavy trace a cap of 32,768 gives up and one
// of 65,536 does not); where groups stay saturated they may never meet, and
// every round would then re-run whole segments (that heavy trace with each
// model kept on two groups: 2.29 s per call without the cap, 0.92 s with it,
// 0.56 s on the shared-trace kernel alone).
constexpr int64_t kSpecGiveUp = 131072;
// Jobs per wavefront: one lane per job.  (32 jobs per wavefront halves the
// state, so a SIMD holds two wavefronts; on the 8192-placement workload that
// took 305 ms against 276: the two did not overlap enough to pay for doubling
// the instructions per job.)
constexpr int kSpecJobsPerWave = 64;
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
  double* ckpt;         // [nseg][ckps][G*SMAX][J] states every ck requests into a segment
  int64_t* ck_served;   // [nseg][ckps][J] served count of the segment before each checkpoint
  uint64_t* ck_fsum;    // [nseg][ckps][J] finish-time sum likewise
  int64_t ck;           // checkpoint interval (a multiple of 64)
  int32_t ckps;         // checkpoints per segment (upper bound)
  int32_t* changed;     // [nseg] segments whose end state changed, per round
  int32_t* cfg_info;    // [3]: 1 when every used group has one configuration; that configuration;
                        // 1 once a re-run gave up (the results are then left to other kernels)
  int64_t cap;          // requests a re-run may take without meeting the old results before giving up
  int64_t nw;
  int64_t warmup;  // requests simulated before a segment to estimate its start state
  int32_t M, C, smax_in, G, K, J, n_finish, nseg, njb;
  int32_t cfg_stages[AS_MAX_CONFIGS];
  int32_t finish_jobs[AS_MAX_FINISH];
};

__host__ __device__ constexpr int pow2ceil_dev(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Rounds in the group-per-lane layout where it applies; ALPASERVE_SPEC_ROUNDS=lane
// keeps the one-lane-per-job round kernel (tests cover both).
inline bool spec_gpl_rounds() {
  const char* e = getenv("ALPASERVE_SPEC_ROUNDS");
  return !(e && std::strcmp(e, "lane") == 0);
}

__device__ __forceinline__ int64_t seg_bound(int64_t n, int nseg, int k) {
  return k >= nseg ? n : ((n * k / nseg) & ~(int64_t)63);
}

__device__ __forceinline__ uint64_t bits_of(double x) { return (uint64_t)__double_as_longlong(x); }

// Accept bits of a chunk: each request's bit enters at the top and moves down
// one place per request, so that after the chunk's cnt requests chunk_word
// has request r's bit at r (bits pushed before them fall out of the word).
__device__ __forceinline__ uint64_t push_bit(uint64_t w, bool bit) {
  const uint32_t lo = (uint32_t)w, hi = (uint32_t)(w >> 32);
  return ((uint64_t)__builtin_amdgcn_alignbit((uint32_t)bit, hi, 1) << 32) | __builtin_amdgcn_alignbit(hi, lo, 1);
}
__device__ __forceinline__ uint64_t chunk_word(uint64_t w, int cnt) { return cnt < 64 ? w >> (64 - cnt) : w; }

// Hosting masks of one lane's placement for every model, MB bits per model,
// held in vector registers (32-dword vector values: a wavefront-uniform index
// into one lowers to indexed register moves, not memory).
typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));

template <int MB>
struct LaneMasks {
  static_assert(MB == 32 || MB == 64, "32- or 64-bit hosting masks");
  using MaskT = typename std::conditional<MB == 32, uint32_t, uint64_t>::type;
  // named vectors, never an array of them: a variable first index would put
  // the registers in memory.  MB 32 uses v0-v1, MB 64 v0-v3.
  u32x32 v0, v1, v2, v3;
  __device__ __forceinline__ void put(int w, uint32_t x) {  // dword w of the masks
    if (w < 32) {
      v0[w & 31] = x;
    } else if (w < 64) {
      v1[w & 31] = x;
    } else if constexpr (MB == 64) {
      if (w < 96) {
        v2[w & 31] = x;
      } else {
        v3[w & 31] = x;
      }
    }
  }
  // bits of groups >= G are dropped (they name no state); returns whether some
  // model has more than two hosting groups
  __device__ __forceinline__ bool load(const uint64_t* row, int M, int G, bool valid) {
    v0 = v1 = (u32x32)(0u);
    if constexpr (MB == 64) v2 = v3 = (u32x32)(0u);
    bool many = false;
    if (!valid) return many;
    const uint64_t keep = G >= 64 ? ~0ull : (1ull << G) - 1;
#pragma unroll
    for (int m = 0; m < 64; ++m) {
      const uint64_t x = m < M ? row[m] & keep : 0;
      many |= __popcll(x) > 2;
      if constexpr (MB == 32) {
        put(m, (uint32_t)x);
      } else {
        put(2 * m, (uint32_t)x);
        put(2 * m + 1, (uint32_t)(x >> 32));
      }
    }
    return many;
  }
  // m is wavefront-uniform; one indexed register move per vector read (the
  // empty asm keeps the compiler from selecting whole vectors first)
  __device__ __forceinline__ MaskT get(int m) const {
    if constexpr (MB == 32) {
      uint32_t lo = v0[m & 31], hi = v1[m & 31];
      asm volatile("" : "+v"(lo), "+v"(hi));
      return m < 32 ? lo : hi;
    } else {
      const int e = (2 * m) & 31;
      uint32_t lo, hi;
      if (m < 16) {
        lo = v0[e];
        hi = v0[e + 1];
      } else if (m < 32) {
        lo = v1[e];
        hi = v1[e + 1];
      } else if (m < 48) {
        lo = v2[e];
        hi = v2[e + 1];
      } else {
        lo = v3[e];
        hi = v3[e + 1];
      }
      asm volatile("" : "+v"(lo), "+v"(hi));
      return (uint64_t)lo | ((uint64_t)hi << 32);
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

// Index of the lowest set bit, -1 when there is none (v_ffbl_b32 returns
// all ones for zero; the asm keeps the compiler from assuming x != 0).
template <typename T>
__device__ __forceinline__ int lowest_or_m1(T x) {
  if constexpr (sizeof(T) == 4) {
    int r;
    asm("v_ffbl_b32 %0, %1" : "=v"(r) : "v"(x));
    return r;
  } else {
    return x ? (int)__builtin_ctzll(x) : -1;
  }
}

// Per-wavefront LDS: the model table, per-lane group configurations when
// groups differ, then the state.
//   uniform configuration c0:  T[m] = {L[m][c0][0..SMAX-1], d_single[m]}
//   otherwise:                 L[m][c][0..SMAX-1], D[m] = d_single[m], cfg[g][lane]
template <int SMAX, bool UCFG>
struct SpecLds {
  double* T;      // UCFG: [M][SMAX + 1]; else L: [M][C][SMAX]
  double* D;      // !UCFG: [M]
  uint16_t* cfg;  // !UCFG: [G][JPW] = c
  double* F;      // rows -1 .. G of [SMAX][JPW]; row -1 is a sentinel, row G is written, never read
};

// jpw: jobs per wavefront (lanes at or above it hold no job).  The state has
// a spare row past the G groups: a request that commits nothing writes
// there, so that the commit is a store without a branch.  Before the groups
// sits a sentinel row -1 whose stage-0 free time is +inf: a lane that has no
// (or no further) hosting group reads it as its host, and it never wins the
// dispatch.
__host__ __device__ constexpr size_t spec_lds_bytes(int M, int C, int G, int SMAX, bool ucfg, int jpw) {
  return (ucfg ? (size_t)M * (SMAX + 1) * 8 : (size_t)M * C * SMAX * 8 + (size_t)M * 8 + (size_t)G * jpw * 2) +
         (size_t)(G + 2) * SMAX * jpw * 8;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  const int lo = __builtin_amdgcn_readlane(__double2loint(v), l);
  const int hi = __builtin_amdgcn_readlane(__double2hiint(v), l);
  return __hiloint2double(hi, lo);
}

template <int SMAX, bool UCFG, int JPW>
__device__ __forceinline__ SpecLds<SMAX, UCFG> spec_tables(const SpecArgs& a, double* lds, int lane, int p,
                                                           bool valid, int c0) {
  SpecLds<SMAX, UCFG> s;
  const int M = a.M, C = a.C;
  s.T = lds;
  if constexpr (UCFG) {
    s.D = nullptr;
    s.cfg = nullptr;
    s.F = s.T + (size_t)M * (SMAX + 1) + SMAX * JPW;
    const int S0 = a.cfg_stages[c0];
    for (int e = lane; e < M * (SMAX + 1); e += 64) {
      const int k = e % (SMAX + 1);
      const int m = e / (SMAX + 1);
      s.T[e] = k == SMAX ? a.d_single[m]
                         : (k < S0 ? a.stage_lat[((int64_t)m * C + c0) * a.smax_in + k] : 0.0);
    }
  } else {
    s.D = s.T + (size_t)M * C * SMAX;
    s.cfg = reinterpret_cast<uint16_t*>(s.D + M);
    s.F = reinterpret_cast<double*>(s.cfg + (size_t)a.G * JPW) + SMAX * JPW;
    // stage latencies (0 beyond S_c: never used)
    for (int e = lane; e < M * C * SMAX; e += 64) {
      const int k = e % SMAX;
      const int c = (e / SMAX) % C;
      const int m = e / (SMAX * C);
      s.T[e] = k < a.cfg_stages[c] ? a.stage_lat[((int64_t)m * C + c) * a.smax_in + k] : 0.0;
    }
    for (int m = lane; m < M; m += 64) s.D[m] = a.d_single[m];
    if (lane < JPW)
      for (int g = 0; g < a.G; ++g) {
        int c = valid ? a.group_cfg[(int64_t)p * a.G + g] : -1;
        if (c < 0 || c >= C) c = 0;  // a group hosting nothing is never chosen
        s.cfg[g * JPW + lane] = (uint16_t)c;
      }
  }
  // the sentinel row: stage 0 never wins, the other stages are never committed
  for (int e = lane; e < SMAX * JPW; e += 64) s.F[e - SMAX * JPW] = e < JPW ? __builtin_inf() : 0.0;
  __syncthreads();
  return s;
}

// The wavefront-uniform part of a request and this lane's hosting groups:
// arrival t, model m, hosting mask and the two lowest hosting groups (-1, the
// sentinel row, where there is none).
template <int MB>
struct Plan {
  using MaskT = typename LaneMasks<MB>::MaskT;
  double t;
  int m;
  MaskT mask;
  int g0, g1;
  // whether some lane of the wavefront hosts the model on more than two
  // groups (a ballot: wavefront-uniform)
  __device__ __forceinline__ bool extra() const {
    const MaskT r1 = mask & (mask - 1);
    return __builtin_amdgcn_ballot_w64((r1 & (r1 - 1)) != 0) != 0;
  }
};

template <int MB>
__device__ __forceinline__ Plan<MB> make_plan(const SpecArgs& a, const LaneMasks<MB>& msk, double t, int m) {
  Plan<MB> pl;
  pl.t = t;
  pl.m = m;
  const bool known = (unsigned)m < (unsigned)a.M;
  const auto x = msk.get(m);  // register moves only: cheaper than a branch around them
  pl.mask = known ? x : 0;
  const auto r1 = pl.mask & (pl.mask - 1);
  pl.g0 = lowest_or_m1(pl.mask);
  pl.g1 = lowest_or_m1(r1);
  return pl;
}

// LDS reads of one request, issued together: the rows of the two lowest
// hosting groups, the stage-0 entries of up to six more hosts when some lane
// of the wavefront has them, and the model's table row.  X: 0 never reads the
// extra hosts, 1 always, 2 when ex (wavefront-uniform) is set.
template <int SMAX, bool UCFG>
struct Reads {
  static constexpr int kX = 6;
  double A[SMAX], B[SMAX], X[kX];
  int hx[kX];
  bool extra;
  double L[UCFG ? SMAX : 1];
  double d;
};

template <int SMAX, bool UCFG, int MB, int JPW, int X>
__device__ __forceinline__ Reads<SMAX, UCFG> issue_reads(const SpecLds<SMAX, UCFG>& s, const Plan<MB>& pl,
                                                         int lane, bool ex) {
  constexpr int kX = Reads<SMAX, UCFG>::kX;
  Reads<SMAX, UCFG> rd;
#pragma unroll
  for (int k = 0; k < SMAX; ++k) {
    rd.A[k] = s.F[(pl.g0 * SMAX + k) * JPW + lane];
    rd.B[k] = s.F[(pl.g1 * SMAX + k) * JPW + lane];
  }
  rd.extra = X == 1 || (X == 2 && ex);
  if (rd.extra) {
    auto rest = pl.mask & (pl.mask - 1);
    rest &= rest - 1;
#pragma unroll
    for (int q = 0; q < kX; ++q) {
      rd.hx[q] = lowest_or_m1(rest);
      rest &= rest - 1;
    }
#pragma unroll
    for (int q = 0; q < kX; ++q) rd.X[q] = s.F[(rd.hx[q] * SMAX) * JPW + lane];
  }
  const int mi = (unsigned)pl.m < 64u ? pl.m : 0;
  if constexpr (UCFG) {
    const double* row = s.T + mi * (SMAX + 1);
#pragma unroll
    for (int k = 0; k < SMAX; ++k) rd.L[k] = row[k];
    rd.d = row[SMAX];
  } else {
    rd.d = s.D[mi];
  }
  return rd;
}

// Dispatch (least stage-0 free time among the hosting groups, lowest index on
// ties), stage chain, admission (finish <= t + scale * d_single[m]) and
// commit of one request on the lane's state.  Returns whether the request is
// served (never on an inactive lane); out is its finish time (-1 dropped, -2
// no hosting group).  Requests that are not served write the spare row G.
// X as for issue_reads (rd.extra: the extra hosts were read).
template <int SMAX, bool UCFG, int MB, int JPW, int X>
__device__ __forceinline__ bool finish_step(const SpecLds<SMAX, UCFG>& s, const Plan<MB>& pl,
                                            const Reads<SMAX, UCFG>& rd, int lane, double scale, int C, int G,
                                            bool active, double& out) {
  constexpr int kX = Reads<SMAX, UCFG>::kX;
  // g1 > g0, and further hosts come in increasing order: strict comparisons
  // keep the lowest index among equal free times (a missing host is the
  // sentinel row, +inf: with no host at all, g is -1 and nothing commits)
  const bool use_b = rd.B[0] < rd.A[0];
  int g = use_b ? pl.g1 : pl.g0;
  double Fv[SMAX];
#pragma unroll
  for (int k = 0; k < SMAX; ++k) Fv[k] = use_b ? rd.B[k] : rd.A[k];
  if (X == 1 || (X == 2 && rd.extra)) {
    double best = Fv[0];
#pragma unroll
    for (int q = 0; q < kX; ++q) {
      if (rd.X[q] < best) {
        best = rd.X[q];
        g = rd.hx[q];
      }
    }
    // hosts after the eighth
    typename LaneMasks<MB>::MaskT rest = pl.mask;
    if (__popcll((uint64_t)pl.mask) > 8) {
#pragma unroll
      for (int q = 0; q < 8; ++q) rest &= rest - 1;
      while (rest) {
        const int h = ctz_any(rest);
        rest &= rest - 1;
        const double v = s.F[(h * SMAX) * JPW + lane];
        if (v < best) {
          best = v;
          g = h;
        }
      }
    }
    if (g != pl.g0 && g != pl.g1) {
#pragma unroll
      for (int k = 0; k < SMAX; ++k) Fv[k] = s.F[(g * SMAX + k) * JPW + lane];
    }
  }
  double Lv[SMAX];
  if constexpr (UCFG) {
#pragma unroll
    for (int k = 0; k < SMAX; ++k) Lv[k] = rd.L[k];
  } else {
    const int c = s.cfg[(g < 0 ? 0 : g) * JPW + lane];
    const int mi = (unsigned)pl.m < 64u ? pl.m : 0;
    const double* Lrow = s.T + ((size_t)mi * C + c) * SMAX;
#pragma unroll
    for (int k = 0; k < SMAX; ++k) Lv[k] = Lrow[k];
  }
  // projection through the stage chain.  A stage past the group's depth has
  // zero latency: its free time is always the last real stage's (so at most
  // the new finish time), and the finish time passes it unchanged.
  double f[SMAX];
  double prev = pl.t;
#pragma unroll
  for (int k = 0; k < SMAX; ++k) {
    f[k] = vmax(prev, Fv[k]) + Lv[k];
    prev = f[k];
  }
  const double slo = scale * rd.d;
  const double deadline = pl.t + slo;
  const bool hosted = pl.mask != 0;
  const bool served = active && hosted && !(prev > deadline);
  out = served ? prev : (hosted ? -1.0 : -2.0);
  const int row = served ? g : G;
#pragma unroll
  for (int k = 0; k < SMAX; ++k) s.F[(row * SMAX + k) * JPW + lane] = f[k];
  return served;
}

struct SpecLane {
  int job, p, frow;
  bool valid;
  double scale;
};

template <int JPW>
__device__ __forceinline__ SpecLane spec_lane(const SpecArgs& a, int jb, int lane) {
  SpecLane l;
  l.job = jb * JPW + lane;
  l.valid = lane < JPW && l.job < a.J;
  l.p = l.valid ? l.job / a.K : 0;
  l.scale = l.valid ? a.slo_scale[l.job % a.K] : 0.0;
  l.frow = -1;
  if (l.valid)
    for (int f = 0; f < a.n_finish; ++f)
      if (a.finish_jobs[f] == l.job) l.frow = f;
  return l;
}

// Arrivals of [from, to) in chunks of 64 (lane r holds request base + r),
// the next chunk loaded while the current one is simulated.
struct TraceChunks {
  double tv, tn;
  int mv, mn;
  int64_t to;
  __device__ __forceinline__ void first(const SpecArgs& a, int64_t from, int64_t to_, int lane) {
    to = to_;
    const int64_t i = from + lane;
    tn = i < to ? a.t[i] : 0.0;
    mn = i < to ? a.model[i] : 0;
  }
  __device__ __forceinline__ void advance(const SpecArgs& a, int64_t next_base, int lane) {
    tv = tn;
    mv = mn;
    const int64_t i = next_base + lane;
    tn = i < to ? a.t[i] : 0.0;
    mn = i < to ? a.model[i] : 0;
  }
};

// Simulate requests [from, to) of one lane (only while the lane is active)
// with the next request's preparation overlapping the current one's LDS
// reads.  EXTRA false: no lane hosts a model on more than two groups.  ROWS
// false: no lane writes finish rows (the code for them is left out).  Per
// chunk of 64 requests: chunk_begin(base) returns 0 to stop the loop (once no
// lane of the wavefront is active), 1 to run the chunk, 2 to run it with
// finish rows; result(i, r, out, served, rows) sees every simulated request
// (on an inactive lane with served false and out meaningless; rows: the chunk
// writes finish rows), after a placeholder call per chunk (i = base - 1,
// served and rows false), chunk_end(base, cnt) closes the chunk.
template <int SMAX, int MB, bool UCFG, int JPW, bool EXTRA, bool ROWS, class Begin, class Result, class End>
__device__ __forceinline__ void spec_range(const SpecArgs& a, const SpecLds<SMAX, UCFG>& s,
                                           const LaneMasks<MB>& msk, const SpecLane& ln, int lane, int64_t from, int64_t to, const bool& active, Begin chunk_begin,
                                           Result result, End chunk_end) {
  if (from >= to) return;
  const int li = lane & (JPW - 1);  // lanes past JPW hold no job: they read a valid lane's slot
  TraceChunks tc;
  tc.first(a, from, to, lane);
  tc.advance(a, from + 64, lane);
  Plan<MB> cur = make_plan<MB>(a, msk, readlane_f64(tc.tv, 0), __builtin_amdgcn_readlane(tc.mv, 0));
  for (int64_t cb = from; cb < to; cb += 64) {
    const int code = chunk_begin(cb);
    if (code == 0) return;
    const int cnt = (int)(to - cb < 64 ? to - cb : 64);
    const bool last_chunk = cb + 64 >= to;
    // lane r: the request after request r (lane 63: the next chunk's first;
    // past the range a placeholder)
    const int from_lane = ((lane + 1) & 63) << 2;
    int t1_lo = __builtin_amdgcn_ds_bpermute(from_lane, __double2loint(tc.tv));
    int t1_hi = __builtin_amdgcn_ds_bpermute(from_lane, __double2hiint(tc.tv));
    int m1 = __builtin_amdgcn_ds_bpermute(from_lane, tc.mv);
    const int n_lo = __builtin_amdgcn_readlane(__double2loint(tc.tn), 0);
    const int n_hi = __builtin_amdgcn_readlane(__double2hiint(tc.tn), 0);
    const int n_m = __builtin_amdgcn_readlane(tc.mn, 0);
    if (lane == 63) {
      t1_lo = n_lo;
      t1_hi = n_hi;
      m1 = n_m;
    }
    const bool rows = ROWS && code == 2;
    // each request's bookkeeping (result) runs one request late, while the
    // next request's reads are in flight; the first call of a chunk is a
    // placeholder (not served: its accept bit is shifted out of the word at
    // the chunk's end, and it writes no row)
    double out_p = 0.0;
    bool served_p = false;
    for (int r = 0; r < cnt; ++r) {
      // the extra-host flag of this request (a ballot) is taken here, at the
      // top, so that its branch is a scalar one
      const bool ex = EXTRA && cur.extra();
      const Reads<SMAX, UCFG> rd = issue_reads<SMAX, UCFG, MB, JPW, EXTRA ? 2 : 0>(s, cur, li, ex);
      result(cb + r - 1, r - 1, out_p, served_p, rows && r > 0);
      // the next request, prepared while this one's reads are in flight
      const double t_nx =
          __hiloint2double(__builtin_amdgcn_readlane(t1_hi, r), __builtin_amdgcn_readlane(t1_lo, r));
      const Plan<MB> nxt = make_plan<MB>(a, msk, t_nx, __builtin_amdgcn_readlane(m1, r));
      served_p = finish_step<SMAX, UCFG, MB, JPW, EXTRA ? 2 : 0>(s, cur, rd, li, ln.scale, a.C, a.G, active, out_p);
      cur = nxt;
    }
    result(cb + cnt - 1, cnt - 1, out_p, served_p, rows);
    chunk_end(cb, cnt);
    if (!last_chunk) tc.advance(a, cb + 128, lane);
  }
}

__device__ __forceinline__ int spec_ckpts(int64_t b, int64_t e, int64_t ck) { return (int)((e - b - 1) / ck); }

// Pass 0 of one wavefront (the per-request output rows are written by
// spec_rows once the rounds have made every saved state exact).
template <int SMAX, int MB, bool UCFG, int JPW, bool EXTRA>
__device__ __forceinline__ void spec_pass0_body(const SpecArgs& a, double* lds, int lane, int k,
                                                const SpecLane& ln, int c0) {
  LaneMasks<MB> msk;
  (void)msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  const auto s = spec_tables<SMAX, UCFG, JPW>(a, lds, lane, ln.p, ln.valid, c0);
  const int GS = a.G * SMAX;
  if (lane < JPW)
    for (int q = 0; q < GS; ++q) s.F[q * JPW + lane] = 0.0;
  if (blockIdx.x == 0 && lane < a.nseg) a.changed[lane] = lane == 0 ? 1 : 0;

  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  const int64_t J = a.J;
  const bool on = true;
  // warm-up: the requests just before the segment, from the empty state, give
  // its start state (usually already the exact one: the rounds then find
  // nothing to redo); one pass over [w0, e) records from b on
  const int64_t wu = (a.warmup + 63) & ~(int64_t)63;
  const int64_t w0 = k == 0 ? b : (b > wu ? b - wu : 0);
  const size_t seg_base = ((size_t)k * GS) * J + ln.job;
  int64_t served = 0;
  uint64_t fsum = 0, word = 0;
  const size_t ck0 = (size_t)k * a.ckps;
  if (w0 == b && ln.valid)
    for (int q = 0; q < GS; ++q) a.st_start[seg_base + (size_t)q * J] = 0.0;
  spec_range<SMAX, MB, UCFG, JPW, EXTRA, false>(
      a, s, msk, ln, lane, w0, e, on,
      [&](int64_t cb) {
        if (cb == b) {
          // the warm-up counts nothing
          served = 0;
          fsum = 0;
        }
        if (cb == b && w0 < b && ln.valid)
          for (int q = 0; q < GS; ++q) a.st_start[seg_base + (size_t)q * J] = s.F[q * JPW + lane];
        if (cb > b && (cb - b) % a.ck == 0 && ln.valid) {
          const size_t j = ck0 + (size_t)((cb - b) / a.ck - 1);
          for (int q = 0; q < GS; ++q) a.ckpt[(j * GS + q) * J + ln.job] = s.F[q * JPW + lane];
          a.ck_served[j * J + ln.job] = served;
          a.ck_fsum[j * J + ln.job] = fsum;
        }
        return 1;
      },
      [&](int64_t i, int r, double out, bool sv, bool rows) {
        (void)i;
        (void)r;
        (void)rows;
        fsum += sv ? bits_of(out) : 0;
        word = push_bit(word, sv);
      },
      [&](int64_t cb, int cnt) {
        word = chunk_word(word, cnt);
        if (cb >= b && ln.valid) a.bitmap[(cb >> 6) * J + ln.job] = word;
        served += __popcll(word);
        word = 0;
      });

  // an empty segment's start state is its warm-up end, and it counts nothing
  if (b == e && w0 < b && ln.valid)
    for (int q = 0; q < GS; ++q) a.st_start[seg_base + (size_t)q * J] = s.F[q * JPW + lane];
  if (b == e) {
    served = 0;
    fsum = 0;
  }
  if (!ln.valid) return;
  for (int q = 0; q < GS; ++q) a.st_end[seg_base + (size_t)q * J] = s.F[q * JPW + lane];  // buffer 0
  a.seg_served[(size_t)k * J + ln.job] = served;
  a.seg_fsum[(size_t)k * J + ln.job] = fsum;
}

// Pass 0: every (job, segment) from a warmed-up estimate of its start state;
// the state is also saved every ck requests (checkpoints for the rounds).
// Every kernel of the speculative pipeline that simulates requests comes in
// four variants, all launched: UCFG (all groups of all placements share one
// configuration) and EXTRA (some lane of the wavefront hosts a model on more
// than two groups) select the code; a workgroup whose data do not match its
// variant returns at once, before any side effect.
template <int SMAX, int MB, bool UCFG, int JPW, bool EXTRA>
__global__ __launch_bounds__(64) void spec_pass0(const SpecArgs a) {
  if ((a.cfg_info[0] != 0) != UCFG) return;
  const int c0 = UCFG ? a.cfg_info[1] : 0;
  extern __shared__ double lds[];
  const int lane = threadIdx.x;
  const int jb = blockIdx.x % a.njb;
  const int k = blockIdx.x / a.njb;
  const SpecLane ln = spec_lane<JPW>(a, jb, lane);
  {
    LaneMasks<MB> m0;
    const bool many = m0.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
    if ((__builtin_amdgcn_ballot_w64(many) != 0) != EXTRA) return;
  }
  spec_pass0_body<SMAX, MB, UCFG, JPW, EXTRA>(a, lds, lane, k, ln, c0);
}

// Per job: served counts and finish-time sums over the segments, and the
// ordered hash over the accept words (the final step of the pipeline).
__device__ __forceinline__ void final_body(const SpecArgs& a, int64_t job) {
  if (job >= a.J) return;
  const int64_t J = a.J;
  int64_t served = 0;
  uint64_t fsum = 0;
  for (int k = 0; k < a.nseg; ++k) {
    served += a.seg_served[(size_t)k * J + job];
    fsum += a.seg_fsum[(size_t)k * J + job];
  }
  // the hash is sequential over words: the next 16 words are loaded while
  // the current 16 are folded in
  constexpr int kB = 16;
  uint64_t h = 0;
  const uint64_t* col = a.bitmap + job;
  const int64_t nb = a.nw / kB;
  uint64_t cur[kB], nxt[kB];
  if (nb > 0) {
#pragma unroll
    for (int q = 0; q < kB; ++q) cur[q] = col[(int64_t)q * J];
  }
  for (int64_t bi = 0; bi < nb; ++bi) {
    const int64_t nbase = (bi + 1 < nb ? bi + 1 : bi) * kB;
#pragma unroll
    for (int q = 0; q < kB; ++q) nxt[q] = col[(nbase + q) * J];
#pragma unroll
    for (int q = 0; q < kB; ++q) h = (h ^ cur[q]) * kSpecHashMul;
#pragma unroll
    for (int q = 0; q < kB; ++q) cur[q] = nxt[q];
  }
  for (int64_t w = nb * kB; w < a.nw; ++w) h = (h ^ col[w * J]) * kSpecHashMul;
  a.out_served[job] = served;
  if (a.out_attain) a.out_attain[job] = a.n > 0 ? (double)served / (double)a.n : 0.0;
  if (a.out_digest) {
    a.out_digest[2 * job] = h;
    a.out_digest[2 * job + 1] = fsum;
  }
}

// Per-request output rows of the jobs that have one.  Pass 0 and the rounds
// write none: once the rounds are done, every saved state is the exact state
// at its point of the trace (a segment's start, and every ck requests into
// it), so each piece of ck requests is simulated again from the state before
// it, all pieces at once, and only the rows are written.  Lanes are jobs with
// a row (JPW per wavefront); blocks are row blocks x segments x pieces, and a
// piece past its segment's end returns at once.
// The extra-host code (some lane hosts a model on more than two groups) is
// chosen per wavefront at run time, so that every row piece, and the final
// step in the dispatch's first nfb workgroups, run in one dispatch.
template <int SMAX, int MB, bool UCFG, int JPW, bool EXTRA>
__device__ __forceinline__ void rows_body(const SpecArgs& a, double* lds, int lane, const SpecLane& ln, int c0,
                                          int k, int pc, int64_t pb, int64_t pe) {
  LaneMasks<MB> msk;  // loaded again here: one copy per body keeps it in registers
  (void)msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  const auto s = spec_tables<SMAX, UCFG, JPW>(a, lds, lane, ln.p, ln.valid, c0);
  const int GS = a.G * SMAX;
  const int64_t J = a.J;
  if (lane < JPW)
    for (int q = 0; q < GS; ++q)
      s.F[q * JPW + lane] = !ln.valid ? 0.0
                            : pc == 0 ? a.st_start[((size_t)k * GS + q) * J + ln.job]
                                      : a.ckpt[(((size_t)k * a.ckps + pc - 1) * GS + q) * J + ln.job];
  const bool on = true;
  spec_range<SMAX, MB, UCFG, JPW, EXTRA, true>(
      a, s, msk, ln, lane, pb, pe, on, [](int64_t) { return 2; },
      [&](int64_t i, int r, double out, bool sv, bool rows) {
        (void)r;
        (void)sv;
        if (rows && ln.valid) a.out_finish[(int64_t)ln.frow * a.n + i] = out;
      },
      [](int64_t, int) {});
}

template <int SMAX, int MB, bool UCFG, int JPW>
__global__ __launch_bounds__(64) void spec_rows(const SpecArgs a, int nfb) {
  if (a.cfg_info[2] != 0) return;  // a re-run gave up: other kernels write the rows
  if ((a.cfg_info[0] != 0) != UCFG) return;
  if ((int)blockIdx.x < nfb) {
    final_body(a, (int64_t)blockIdx.x * 64 + threadIdx.x);
    return;
  }
  const int bx = (int)blockIdx.x - nfb;
  const int c0 = UCFG ? a.cfg_info[1] : 0;
  extern __shared__ double lds[];
  const int lane = threadIdx.x;
  const int nrb = (a.n_finish + JPW - 1) / JPW;
  const int np = a.ckps + 1;
  const int rb = bx % nrb;
  const int pc = (bx / nrb) % np;
  const int k = bx / (nrb * np);
  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  const int64_t pb = b + (int64_t)pc * a.ck;
  if (pb >= e) return;
  const int64_t pe = e - pb < a.ck ? e : pb + a.ck;
  SpecLane ln;
  const int f = rb * JPW + lane;
  ln.valid = lane < JPW && f < a.n_finish;
  ln.job = ln.valid ? a.finish_jobs[f] : 0;
  ln.p = ln.valid ? ln.job / a.K : 0;
  ln.scale = ln.valid ? a.slo_scale[ln.job % a.K] : 0.0;
  ln.frow = ln.valid ? f : -1;
  bool many;
  {
    LaneMasks<MB> msk;
    many = msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  }
  if (__builtin_amdgcn_ballot_w64(many) != 0)
    rows_body<SMAX, MB, UCFG, JPW, true>(a, lds, lane, ln, c0, k, pc, pb, pe);
  else
    rows_body<SMAX, MB, UCFG, JPW, false>(a, lds, lane, ln, c0, k, pc, pb, pe);
}

// Round q >= 1: a segment whose start state differs from its predecessor's
// end state re-runs from that end state, comparing its state with the saved
// checkpoints of its current results: where they are equal the two runs
// coincide from there on, so the re-run stops and only its prefix replaces
// the old results.  Checkpoints passed before that point are replaced with
// the new run's.
template <int SMAX, int MB, bool UCFG, int JPW, bool EXTRA>
__global__ __launch_bounds__(64) void spec_round(const SpecArgs a, int q) {
  if ((a.cfg_info[0] != 0) != UCFG) return;
  if (a.cfg_info[2] != 0) return;     // a re-run gave up: other kernels take over
  if (a.changed[q - 1] == 0) return;  // nothing moved in the previous round: done
  const int c0 = UCFG ? a.cfg_info[1] : 0;
  extern __shared__ double lds[];
  const int lane = threadIdx.x;
  const int jb = blockIdx.x % a.njb;
  const int k = blockIdx.x / a.njb;
  const SpecLane ln = spec_lane<JPW>(a, jb, lane);
  const int GS = a.G * SMAX;
  const int64_t J = a.J;
  const size_t per_buf = (size_t)a.nseg * GS * J;
  const double* E_in = a.st_end + (size_t)((q - 1) & 1) * per_buf;
  double* E_out = a.st_end + (size_t)(q & 1) * per_buf;
  const size_t own = ((size_t)k * GS) * J + ln.job;
  const size_t prv = k > 0 ? ((size_t)(k - 1) * GS) * J + ln.job : 0;
  LaneMasks<MB> msk;
  const bool many = msk.load(a.host_mask + (int64_t)ln.p * a.M, a.M, a.G, ln.valid);
  if ((__builtin_amdgcn_ballot_w64(many) != 0) != EXTRA) return;

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
  const auto s = spec_tables<SMAX, UCFG, JPW>(a, lds, lane, ln.p, ln.valid, c0);
  if (lane < JPW)
    for (int x = 0; x < GS; ++x) s.F[x * JPW + lane] = active ? E_in[prv + (size_t)x * J] : 0.0;

  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  const size_t ck0 = (size_t)k * a.ckps;
  const int nck = b < e ? spec_ckpts(b, e, a.ck) : 0;
  int64_t served = 0;
  uint64_t fsum = 0, word = 0;
  bool coupled = false, gave_up = false;
  spec_range<SMAX, MB, UCFG, JPW, EXTRA, false>(
      a, s, msk, ln, lane, b, e, active,
      [&](int64_t cb) {
        if (cb > b && (cb - b) % a.ck == 0 && active) {
          const int jl = (int)((cb - b) / a.ck) - 1;
          const size_t j = ck0 + (size_t)jl;
          bool same = true;
          for (int x = 0; x < GS; ++x)
            same &= bits_of(a.ckpt[(j * GS + x) * J + ln.job]) == bits_of(s.F[x * JPW + lane]);
          const int64_t old_s = a.ck_served[j * J + ln.job];
          const uint64_t old_f = a.ck_fsum[j * J + ln.job];
          if (same) {
            // the old results stand from here on; later checkpoints' running
            // totals shift by the prefix's change
            coupled = true;
            active = false;
            const int64_t ds = served - old_s;
            const uint64_t df = fsum - old_f;
            a.seg_served[(size_t)k * J + ln.job] += ds;
            a.seg_fsum[(size_t)k * J + ln.job] += df;
            a.ck_served[j * J + ln.job] = served;
            a.ck_fsum[j * J + ln.job] = fsum;
            for (int j2 = jl + 1; j2 < nck; ++j2) {
              a.ck_served[(ck0 + j2) * J + ln.job] += ds;
              a.ck_fsum[(ck0 + j2) * J + ln.job] += df;
            }
          } else {
            for (int x = 0; x < GS; ++x) a.ckpt[(j * GS + x) * J + ln.job] = s.F[x * JPW + lane];
            a.ck_served[j * J + ln.job] = served;
            a.ck_fsum[j * J + ln.job] = fsum;
          }
        }
        const bool any = __builtin_amdgcn_ballot_w64(active) != 0;
        if (any && cb - b >= a.cap) {
          // runs from the two states do not meet: the pipeline gives up
          if (lane == 0) a.cfg_info[2] = 1;
          gave_up = true;
          return 0;
        }
        return any ? 1 : 0;
      },
      [&](int64_t i, int r, double out, bool sv, bool rows) {
        (void)i;
        (void)r;
        (void)rows;
        fsum += sv ? bits_of(out) : 0;
        word = push_bit(word, sv);
      },
      [&](int64_t cb, int cnt) {
        word = chunk_word(word, cnt);
        if (active) a.bitmap[(cb >> 6) * J + ln.job] = word;
        served += __popcll(word);
        word = 0;
      });

  if (gave_up || !ln.valid) return;
  if (ran) {
    // the predecessor's end state now stands behind this segment's results
    for (int x = 0; x < GS; ++x) a.st_start[own + (size_t)x * J] = E_in[prv + (size_t)x * J];
    if (!coupled) {
      // re-run to the end: its totals replace the old ones, and unless it
      // ends in the old end state its successor must be revisited
      a.seg_served[(size_t)k * J + ln.job] = served;
      a.seg_fsum[(size_t)k * J + ln.job] = fsum;
      bool same = true;
      for (int x = 0; x < GS; ++x) same &= bits_of(E_in[own + (size_t)x * J]) == bits_of(s.F[x * JPW + lane]);
      if (!same) {
        for (int x = 0; x < GS; ++x) E_out[own + (size_t)x * J] = s.F[x * JPW + lane];
        atomicAdd(a.changed + q, 1);
        return;
      }
    }
  }
  for (int x = 0; x < GS; ++x) E_out[own + (size_t)x * J] = E_in[own + (size_t)x * J];
}

// One 64-request chunk (cnt <= 64 of them, staged in LDS) of a round in the
// group-per-lane layout, run by the shared-trace kernel's request step;
// returns the job's accept word (request r at bit r, in every lane of the
// job) and adds its population count to the job's served count.
template <int W, int SMAX, bool UNI>
__device__ __forceinline__ uint64_t round_chunk(SharedLane<SMAX>& st, const SharedConst& c, const double* sT,
                                                const uint32_t* sO, int cnt) {
  uint64_t word = 0;
  for (int h = 0; h < cnt; h += 32) {
    const int hc = (cnt - h) < 32 ? (cnt - h) : 32;
    uint32_t sr = 0;  // request e of the half at bit hc - 1 - e
    if (hc == 32) {
      for (int e = 0; e < 32; e += 4)
        fast_batch<W, SMAX, 4, false, false, false, UNI>(st, c, sT + 2 * (h + e), sO + h + e, h + e, sr);
    } else {
      for (int e = 0; e < hc; ++e)
        fast_batch<W, SMAX, 1, false, false, false, UNI>(st, c, sT + 2 * (h + e), sO + h + e, h + e, sr);
    }
    const uint32_t bits = hc == 32 ? __builtin_bitreverse32(sr) : (__builtin_bitreverse32(sr) >> (32 - hc));
    word |= (uint64_t)bits << h;
  }
  const uint64_t wj = seg_or<W>(word);
  st.served += (uint64_t)__popcll(wj);
  return wj;
}

// LDS bytes of spec_round_fast: M + 1 model records (the last hosts nothing
// and stands for an out-of-range model id), the stage-latency table
// [M][Cp][SMAX] and one staged chunk (arrivals at stride 2, record offsets).
__host__ __device__ constexpr size_t round_fast_lds_bytes(int M, int Cp, int SMAX) {
  return (size_t)(M + 1) * ((size_t)1 << rec_shift(SMAX)) + (size_t)M * Cp * SMAX * 8 + 128 * 8 + 64 * 4;
}

// Round q >= 1 in the group-per-lane layout (jobs of at most 16 groups): the
// protocol of spec_round with a job's groups on W lanes, their stage free
// times in registers, and the shared-trace kernel's request step --
// per-wavefront model records in LDS (hosting lanes, the count that says
// whether a dispatch minimum is needed, stage latencies, d_single), the
// two-level integer minimum, four requests' inputs read together.  A round
// re-runs few jobs and lasts as long as its longest re-run, and per request
// this layout is a shorter chain than one lane per job.  Stages past a
// group's depth have zero latency, as in the other speculative kernels, so
// saved states compare bit for bit.  Only the jobs that re-run host models in
// the records; a job that has met the old results keeps simulating with the
// others but writes nothing more.  Each 64-request chunk is staged in LDS
// from registers loaded a chunk ahead.
template <int W, int SMAX>
__global__ __launch_bounds__(64) void spec_round_fast(const SpecArgs a, int q) {
  constexpr int JW = 64 / W;  // jobs per wavefront
  constexpr int RSH = rec_shift(SMAX);
  if (a.cfg_info[2] != 0) return;  // a re-run gave up: other kernels take over
  if (a.changed[q - 1] == 0) return;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x;
  const int g = lane % W, slot = lane / W;
  const int njbw = (a.J + JW - 1) / JW;
  const int k = blockIdx.x / njbw, jb = blockIdx.x % njbw;
  const int job = jb * JW + slot;
  const bool valid = job < a.J;
  const bool mine = valid && g < a.G;  // this lane holds a group of a job
  const int GS = a.G * SMAX;
  const int64_t J = a.J;
  const size_t per_buf = (size_t)a.nseg * GS * J;
  const double* E_in = a.st_end + (size_t)((q - 1) & 1) * per_buf;
  double* E_out = a.st_end + (size_t)(q & 1) * per_buf;
  const size_t own = ((size_t)k * GS + (size_t)g * SMAX) * J + job;  // my group's first entry
  const size_t prv = k > 0 ? ((size_t)(k - 1) * GS + (size_t)g * SMAX) * J + job : 0;
  const uint64_t field = (W == 64 ? ~0ull : ((1ull << W) - 1)) << ((uint64_t)slot * W);

  // stale start state?  (every lane of a job agrees through the ballot)
  bool differ = false;
  if (mine && k > 0)
#pragma unroll
    for (int st = 0; st < SMAX; ++st)
      differ |= bits_of(a.st_start[own + (size_t)st * J]) != bits_of(E_in[prv + (size_t)st * J]);
  bool active = (__builtin_amdgcn_ballot_w64(differ) & field) != 0 && valid;
  const bool ran = active;
  if (__builtin_amdgcn_ballot_w64(active) == 0) {
    if (mine)
#pragma unroll
      for (int st = 0; st < SMAX; ++st) E_out[own + (size_t)st * J] = E_in[own + (size_t)st * J];
    return;
  }

  // the models this lane's group hosts (re-running jobs only) and its configuration
  const int p = valid ? job / a.K : 0;
  int cfg = -1;
  uint64_t hostbits = 0;  // bit m: this lane's group hosts model m
  if (mine && ran) {
    cfg = a.group_cfg[(int64_t)p * a.G + g];
    if (cfg < 0 || cfg >= a.C) cfg = -1;  // an unused group hosts nothing
    if (cfg >= 0) {
      const uint64_t* hm = a.host_mask + (int64_t)p * a.M;
      for (int m = 0; m < a.M; ++m) hostbits |= ((hm[m] >> g) & 1ull) << m;
    }
  }
  int cp = 1, lshift = 0;
  while (cp < a.C) cp <<= 1;
  while ((1 << lshift) < cp * SMAX * 8) ++lshift;
  unsigned char* rec = smem;
  double* sL = reinterpret_cast<double*>(rec + (size_t)(a.M + 1) * (1 << RSH));  // [M][Cp][SMAX]
  double* sT = sL + (size_t)a.M * cp * SMAX;                                    // arrivals, stride 2
  uint32_t* sO = reinterpret_cast<uint32_t*>(sT + 128);                          // record offsets
  const uint64_t vmask = __builtin_amdgcn_ballot_w64(cfg >= 0);
  const int cfg0 = vmask ? __builtin_amdgcn_readlane(cfg, __builtin_ctzll(vmask)) : 0;
  const bool uni = __builtin_amdgcn_ballot_w64(cfg >= 0 && cfg != cfg0) == 0;
  for (int idx = lane; idx < a.M * cp * SMAX; idx += 64) {
    const int st = idx % SMAX, mc = idx / SMAX, cc = mc % cp, m = mc / cp;
    sL[idx] = (cc < a.C && st < a.cfg_stages[cc]) ? a.stage_lat[((int64_t)m * a.C + cc) * a.smax_in + st] : 0.0;
  }
  for (int m = 0; m <= a.M; ++m) {
    const uint64_t hm = m < a.M ? __builtin_amdgcn_ballot_w64((hostbits >> (m & 63)) & 1u) : 0;
    if (lane == 0) {
      const uint64_t one = lowest_per_field<W>(hm);  // lowest hosting lane of each job
      *(uint64_t*)(rec + ((size_t)m << RSH) + kRecMask) = hm;
      *(uint64_t*)(rec + ((size_t)m << RSH) + kRecCount) = one == hm ? 0u : (uint32_t)__builtin_popcountll(one);
    }
  }
  for (int m = lane; m <= a.M; m += 64) {
    unsigned char* r = rec + ((size_t)m << RSH);
    *(double*)(r + rec_slo(SMAX)) = m < a.M ? a.d_single[m] : 0.0;
#pragma unroll
    for (int st = 0; st < SMAX; ++st)
      ((double*)(r + kRecLat))[st] =
          (m < a.M && uni && st < a.cfg_stages[cfg0]) ? a.stage_lat[((int64_t)m * a.C + cfg0) * a.smax_in + st]
                                                      : 0.0;
  }
  SharedConst c;
  c.rec = rec;
  c.lrow = sL + (cfg < 0 ? 0 : cfg) * SMAX;
  c.lshift = lshift;
  c.sigma = valid ? a.slo_scale[job % a.K] : 0.0;
  c.fmask = 0;
  c.frowp = nullptr;
  c.flimit = 0;
  c.fcnt = 0;
  c.cnt = nullptr;
  SharedLane<SMAX> st;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) st.F[s] = (mine && ran) ? E_in[prv + (size_t)s * J] : 0.0;
  st.fin_sum = st.hash = st.served = 0;  // served: the job's count, in every lane of it
  st.wlo = 0;
  st.busy = 0.0;
  __syncthreads();

  const int64_t b = seg_bound(a.n, a.nseg, k), e = seg_bound(a.n, a.nseg, k + 1);
  const size_t ck0 = (size_t)k * a.ckps;
  const int nck = b < e ? spec_ckpts(b, e, a.ck) : 0;
  bool coupled = false;
  TraceChunks tc;
  tc.first(a, b, e, lane);
  for (int64_t cb = b; cb < e; cb += 64) {
    tc.advance(a, cb + 64, lane);
    if (cb > b && (cb - b) % a.ck == 0) {
      // saved state of the current results at cb: compare, then keep or stop
      const int jl = (int)((cb - b) / a.ck) - 1;
      const size_t j = ck0 + (size_t)jl;
      bool same = true;
      if (mine && active)
#pragma unroll
        for (int s = 0; s < SMAX; ++s)
          same &= bits_of(a.ckpt[(j * GS + (size_t)g * SMAX + s) * J + job]) == bits_of(st.F[s]);
      const bool job_same = (__builtin_amdgcn_ballot_w64(!same) & field) == 0;
      const uint64_t js = st.served, jf = seg_sum_u64<W>(st.fin_sum);  // uniform flow
      if (active) {
        const size_t cj = j * J + job;
        if (job_same) {
          if (g == 0) {
            const int64_t ds = (int64_t)js - a.ck_served[cj];
            const uint64_t df = jf - a.ck_fsum[cj];
            a.seg_served[(size_t)k * J + job] += ds;
            a.seg_fsum[(size_t)k * J + job] += df;
            a.ck_served[cj] = (int64_t)js;
            a.ck_fsum[cj] = jf;
            for (int j2 = jl + 1; j2 < nck; ++j2) {
              a.ck_served[(ck0 + j2) * J + job] += ds;
              a.ck_fsum[(ck0 + j2) * J + job] += df;
            }
          }
          coupled = true;
          active = false;
        } else {
          if (mine)
#pragma unroll
            for (int s = 0; s < SMAX; ++s) a.ckpt[(j * GS + (size_t)g * SMAX + s) * J + job] = st.F[s];
          if (g == 0) {
            a.ck_served[cj] = (int64_t)js;
            a.ck_fsum[cj] = jf;
          }
        }
      }
      if (__builtin_amdgcn_ballot_w64(active) == 0) break;
    }
    if (cb - b >= a.cap && __builtin_amdgcn_ballot_w64(active) != 0) {
      // runs from the two states do not meet: the pipeline gives up
      if (lane == 0) a.cfg_info[2] = 1;
      return;
    }
    const int cnt = __builtin_amdgcn_readfirstlane((int)(e - cb < 64 ? e - cb : 64));
    // stage the chunk: lane r holds request cb + r
    sT[2 * lane] = tc.tv;
    sO[lane] = (uint32_t)((unsigned)tc.mv < (unsigned)a.M ? tc.mv : a.M) << RSH;
    __syncthreads();
    const uint64_t word = uni ? round_chunk<W, SMAX, true>(st, c, sT, sO, cnt)
                              : round_chunk<W, SMAX, false>(st, c, sT, sO, cnt);
    __syncthreads();
    if (active && g == 0) a.bitmap[(cb >> 6) * J + job] = word;
  }
  const uint64_t js = st.served, jf = seg_sum_u64<W>(st.fin_sum);  // uniform flow
  bool end_same = true;
  if (mine && ran && !coupled)
#pragma unroll
    for (int s = 0; s < SMAX; ++s) end_same &= bits_of(E_in[own + (size_t)s * J]) == bits_of(st.F[s]);
  const bool job_end_same = (__builtin_amdgcn_ballot_w64(!end_same) & field) == 0;
  if (!valid) return;
  if (ran) {
    if (mine)
#pragma unroll
      for (int s = 0; s < SMAX; ++s) a.st_start[own + (size_t)s * J] = E_in[prv + (size_t)s * J];
    if (!coupled) {
      if (g == 0) {
        a.seg_served[(size_t)k * J + job] = (int64_t)js;
        a.seg_fsum[(size_t)k * J + job] = jf;
      }
      if (!job_end_same) {
        if (mine)
#pragma unroll
          for (int s = 0; s < SMAX; ++s) E_out[own + (size_t)s * J] = st.F[s];
        if (g == 0) atomicAdd(a.changed + q, 1);
        return;
      }
    }
  }
  if (mine)
#pragma unroll
    for (int s = 0; s < SMAX; ++s) E_out[own + (size_t)s * J] = E_in[own + (size_t)s * J];
}

// Per job: totals over segments and the ordered digest over the accept words.
__global__ __launch_bounds__(64) void spec_final(const SpecArgs a) {
  if (a.cfg_info[2] != 0) return;  // a re-run gave up: other kernels write the results
  final_body(a, (int64_t)blockIdx.x * 64 + threadIdx.x);
}

}  // namespace
}  // namespace as_dev

namespace as_dev {
namespace {

// Whether every group that a placement uses (configuration >= 0) has one and
// the same configuration; cfg_info = {uniform, that configuration, 0 (no
// re-run has given up)}.  One workgroup of 1024 threads.
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
    cfg_info[2] = 0;
  }
}

// Rounds in the group-per-lane layout (jobs of at most 16 groups).
template <int W, int SMAX>
void spec_rounds_gpl(const SpecArgs& a, hipStream_t s) {
  const int njbw = (a.J + 64 / W - 1) / (64 / W);
  const dim3 grid((unsigned)((int64_t)njbw * a.nseg)), block(64);
  int cp = 1;
  while (cp < a.C) cp <<= 1;
  const size_t lds = round_fast_lds_bytes(a.M, cp, SMAX);
  for (int q = 1; q < a.nseg; ++q) hipLaunchKernelGGL((spec_round_fast<W, SMAX>), grid, block, lds, s, a, q);
}

template <int SMAX>
void spec_rounds_gpl_w(const SpecArgs& a, hipStream_t s) {
  switch (pow2ceil_dev(a.G)) {
    case 1: spec_rounds_gpl<1, SMAX>(a, s); break;
    case 2: spec_rounds_gpl<2, SMAX>(a, s); break;
    case 4: spec_rounds_gpl<4, SMAX>(a, s); break;
    case 8: spec_rounds_gpl<8, SMAX>(a, s); break;
    default: spec_rounds_gpl<16, SMAX>(a, s); break;
  }
}


template <int SMAX, int MB, int JPW>
hipError_t spec_launch_all(const SpecArgs& a, size_t lds_u, size_t lds_g, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)a.njb * a.nseg)), block(64);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, true, JPW, false>), grid, block, lds_u, s, a);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, true, JPW, true>), grid, block, lds_u, s, a);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, false, JPW, false>), grid, block, lds_g, s, a);
  hipLaunchKernelGGL((spec_pass0<SMAX, MB, false, JPW, true>), grid, block, lds_g, s, a);
  if (a.G <= 16 && spec_gpl_rounds()) {
    spec_rounds_gpl_w<SMAX>(a, s);
  } else {
    for (int q = 1; q < a.nseg; ++q) {
      hipLaunchKernelGGL((spec_round<SMAX, MB, true, JPW, false>), grid, block, lds_u, s, a, q);
      hipLaunchKernelGGL((spec_round<SMAX, MB, true, JPW, true>), grid, block, lds_u, s, a, q);
      hipLaunchKernelGGL((spec_round<SMAX, MB, false, JPW, false>), grid, block, lds_g, s, a, q);
      hipLaunchKernelGGL((spec_round<SMAX, MB, false, JPW, true>), grid, block, lds_g, s, a, q);
    }
  }
  const int nfb = (int)((a.J + 63) / 64);
  if (a.n_finish > 0) {
    // the output rows, from the exact saved states, all pieces at once, and
    // in the same dispatch (its first nfb workgroups) the final step
    const dim3 rgrid((unsigned)(nfb + (int64_t)((a.n_finish + JPW - 1) / JPW) * a.nseg * (a.ckps + 1)));
    hipLaunchKernelGGL((spec_rows<SMAX, MB, true, JPW>), rgrid, block, lds_u, s, a, nfb);
    hipLaunchKernelGGL((spec_rows<SMAX, MB, false, JPW>), rgrid, block, lds_g, s, a, nfb);
  } else {
    hipLaunchKernelGGL(spec_final, dim3((unsigned)nfb), block, 0, s, a);
  }
  return hipGetLastError();
}

// Workgroups (one wavefront each) of the pass-0 kernel that one compute unit
// holds at this LDS size.
template <int SMAX, int MB, int JPW>
int spec_occupancy(size_t lds) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, spec_pass0<SMAX, MB, true, JPW, false>, 64, lds) != hipSuccess)
    return 1;
  return nb > 0 ? nb : 1;
}

template <int SMAX>
int spec_occupancy_mb(int G, size_t lds) {
  return G <= 32 ? spec_occupancy<SMAX, 32, kSpecJobsPerWave>(lds) : spec_occupancy<SMAX, 64, kSpecJobsPerWave>(lds);
}

template <int SMAX>
hipError_t spec_launch_mb(int G, const SpecArgs& a, size_t l1, size_t l2, hipStream_t s) {
  return G <= 32 ? spec_launch_all<SMAX, 32, kSpecJobsPerWave>(a, l1, l2, s)
                 : spec_launch_all<SMAX, 64, kSpecJobsPerWave>(a, l1, l2, s);
}

}  // namespace
}  // namespace as_dev

namespace as_host {

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

namespace {



// warm-up requests before a segment (measured on the 8192-placement workload:
// 32768 -> 255.7 ms per step, 16384 -> 249.5, 8192 -> 242-244, 2048 -> 251,
// none -> 261: a shorter warm-up leaves more to the rounds)
constexpr int64_t kSpecWarmup = 8192;
// requests per segment at least: the warm-up and the rounds' re-runs stay a
// small part of a segment's work (shorter traces, like the searches' 151k
// requests, ran slower on these kernels)
constexpr int64_t kSpecMinSegment = 131072;
constexpr int64_t kSpecCheckpoint = 8192;   // requests between saved states

}  // namespace

// Stream-ordered workspace allocation from a memory pool private to this
// library, one per device, whose release threshold is at its maximum: the
// workspace freed by one call is reused by the next instead of going back to
// the driver, and the process's default pool keeps its own settings.  Where a
// private pool cannot be created, the default pool serves as it is.
hipError_t pool_alloc(void** p, size_t bytes, hipStream_t s) {
  static std::mutex mu;
  static hipMemPool_t pools[64];
  static int state[64] = {0};  // 0 not tried, 1 private pool, 2 default pool
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipMallocAsync(p, bytes, s);
  int st = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    if (state[dev] == 0) {
      hipMemPoolProps props;
      std::memset(&props, 0, sizeof props);
      props.allocType = hipMemAllocationTypePinned;
      props.handleTypes = hipMemHandleTypeNone;
      props.location.type = hipMemLocationTypeDevice;
      props.location.id = dev;
      state[dev] = 2;
      if (hipMemPoolCreate(&pools[dev], &props) == hipSuccess) {
        uint64_t thr = UINT64_MAX;
        (void)hipMemPoolSetAttribute(pools[dev], hipMemPoolAttrReleaseThreshold, &thr);
        state[dev] = 1;
      } else {
        (void)hipGetLastError();
      }
    }
    st = state[dev];
  }
  return st == 1 ? hipMallocFromPoolAsync(p, bytes, pools[dev], s) : hipMallocAsync(p, bytes, s);
}

// Segments per job for the speculative path: enough (job block, segment)
// wavefronts to fill the device at the occupancy the LDS allows, each segment
// long enough that the warm-up and the rounds' re-runs are a small part of it.
// ALPASERVE_SPEC_SEGMENTS forces the count (tests).
int spec_segments(int64_t n, int64_t J, int jpw, int per_cu) {
  if (const char* e = getenv("ALPASERVE_SPEC_SEGMENTS")) {
    const int v = atoi(e);
    if (v >= 1) return std::min(v, as_dev::kSpecMaxSeg);
  }
  const int64_t slots = (int64_t)compute_units() * std::max(per_cu, 1);
  const int64_t njb = (J + jpw - 1) / jpw;
  int64_t k = slots / std::max<int64_t>(njb, 1);
  k = std::min<int64_t>(k, n / kSpecMinSegment);
  return (int)std::max<int64_t>(1, std::min<int64_t>(k, as_dev::kSpecMaxSeg));
}

// Whether the speculative kernels beat the shared-trace kernel on this call,
// by a cost model in cycles per request of one wavefront, measured on gfx950
// with the 8192-placement, 3.6 M-request workload: the shared-trace kernel
// about 300 cycles with one wavefront per SIMD and 195 per wavefront beyond
// that (it is issue-bound there); the speculative kernels about 1150 (one
// wavefront per SIMD: the LDS holds no more) over a segment plus its warm-up,
// and a fifth more for the rounds.  A single segment never pays.
bool spec_pays(const KArgs& k, int nseg, int jpw, int per_cu) {
  if (nseg < 2) return false;
  const double simds = 4.0 * compute_units();
  const int Wp = pow2ceil(k.G);
  const double waves_shared = std::ceil((double)k.J / (64 / Wp));
  const double t_shared = (double)k.n * std::max(300.0, 195.0 * waves_shared / simds);
  const double slots = (double)compute_units() * std::max(per_cu, 1);
  const double waves_spec = std::ceil((double)k.J / jpw) * nseg;
  const double seg = (double)k.n / nseg + (double)std::min<int64_t>(kSpecWarmup, k.n);
  const double t_spec = seg * 1150.0 * 1.2 * std::ceil(waves_spec / slots);
  return t_spec < t_shared;
}

// Shared-trace simulation on the segment-speculative kernels.  Returns
// AS_E_LIMITS without launching when the state of one wavefront does not fit
// in the LDS, when the trace does not split into segments that pay (unless
// ALPASERVE_PATH=spec forces the kernels), or when the workspace would be too
// large.  With can_give_up the workspace outlives the call: the caller's
// gated fallback kernels read the give-up flag in it, then release it.
namespace {

// Whether the speculative kernels take the call (sizes, LDS, segments that
// pay or are forced), with their LDS sizes, occupancy and segment count.
bool spec_plan(const KArgs& k, int smax, size_t& lds_u, size_t& lds_g, int& per_cu, int& nseg) {
  using namespace as_dev;
  if (k.n <= 0 || k.J <= 0) return false;
  const size_t lim = shared_lds_limit();
  const int jpw = kSpecJobsPerWave;
  lds_u = spec_lds_bytes(k.M, k.C, k.G, smax, true, jpw);
  lds_g = spec_lds_bytes(k.M, k.C, k.G, smax, false, jpw);
  if (lds_g > lim || lds_u > lim) return false;
  per_cu = 1;
  switch (smax) {
    case 1: per_cu = spec_occupancy_mb<1>(k.G, lds_u); break;
    case 2: per_cu = spec_occupancy_mb<2>(k.G, lds_u); break;
    case 4: per_cu = spec_occupancy_mb<4>(k.G, lds_u); break;
    default: per_cu = spec_occupancy_mb<8>(k.G, lds_u); break;
  }
  nseg = spec_segments(k.n, k.J, jpw, per_cu);
  return spec_forced() || spec_pays(k, nseg, jpw, per_cu);
}

}  // namespace

bool spec_takes(const KArgs& k, int smax) {
  size_t lds_u = 0, lds_g = 0;
  int per_cu = 1, nseg = 1;
  return spec_plan(k, smax, lds_u, lds_g, per_cu, nseg);
}

int run_spec(KArgs& k, int smax, hipStream_t stream, bool can_give_up, void* caller_ws,
             size_t caller_ws_bytes, void** workspace, const int32_t** gave_up) {
  using namespace as_dev;
  *workspace = nullptr;
  *gave_up = nullptr;
  const int jpw = kSpecJobsPerWave;
  size_t lds_u = 0, lds_g = 0;
  int per_cu = 1, nseg = 1;
  if (!spec_plan(k, smax, lds_u, lds_g, per_cu, nseg)) return AS_E_LIMITS;

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
  a.njb = (int32_t)((k.J + jpw - 1) / jpw);
  a.nseg = nseg;
  a.warmup = kSpecWarmup;
  if (const char* w = getenv("ALPASERVE_SPEC_WARMUP")) a.warmup = std::max<int64_t>(0, atoll(w));
  a.ck = kSpecCheckpoint;
  if (const char* c = getenv("ALPASERVE_SPEC_CKPT")) a.ck = std::max<int64_t>(64, atoll(c) & ~(int64_t)63);
  a.ckps = (int32_t)((k.n / a.nseg + 64) / a.ck + 1);
  a.cap = can_give_up ? kSpecGiveUp : INT64_MAX;
  if (const char* c = getenv("ALPASERVE_SPEC_CAP"); c && can_give_up) a.cap = std::max<int64_t>(64, atoll(c));
  while (a.nseg > 1 && (int64_t)a.njb * a.nseg > 0x7FFFFFFFLL) --a.nseg;
  if ((int64_t)a.njb * a.nseg > 0x7FFFFFFFLL) return AS_E_LIMITS;
  a.nw = (k.n + 63) / 64;

  const int64_t J = k.J, GS = (int64_t)k.G * smax;
  const size_t b_bitmap = (size_t)a.nw * J * 8;
  const size_t b_state = (size_t)a.nseg * GS * J * 8;
  const size_t b_seg = (size_t)a.nseg * J * 8;
  const size_t b_ckpt = (size_t)a.nseg * a.ckps * GS * J * 8;
  const size_t b_cks = (size_t)a.nseg * a.ckps * J * 8;
  const size_t b_small = 256 + (size_t)a.nseg * 4;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t total = up(b_bitmap) + up(b_state) + up(2 * b_state) + 2 * up(b_seg) + up(b_ckpt) +
                       2 * up(b_cks) + up(b_small);
  char* ws = nullptr;
  hipError_t e = hipSuccess;
  if (caller_ws) {
    if (total > caller_ws_bytes) {
      fail(AS_E_LIMITS,
           "this call needs %zu bytes of speculative-kernel workspace, more than the %zu-byte "
           "no-allocation scratch; as_simulate_placements takes it",
           total, caller_ws_bytes);
      return kSpecScratchTooSmall;
    }
    ws = static_cast<char*>(caller_ws);
  } else {
    // a workspace beyond a quarter of the device's memory leaves the call to
    // the kernels that need none
    size_t free_b = 0, total_b = 0;
    if (hipMemGetInfo(&free_b, &total_b) != hipSuccess || total > total_b / 4) return AS_E_LIMITS;
    // ALPASERVE_SPEC_MAX_WORKSPACE (bytes) makes a larger workspace fail as a
    // failed allocation does (tests of the fallback to the other kernels)
    if (const char* cap = getenv("ALPASERVE_SPEC_MAX_WORKSPACE"))
      if ((long long)total > atoll(cap))
        return fail(AS_E_NOMEM, "workspace of %zu bytes above ALPASERVE_SPEC_MAX_WORKSPACE", total);
    e = pool_alloc(reinterpret_cast<void**>(&ws), total, stream);
    if (e != hipSuccess || !ws)
      return fail(AS_E_NOMEM, "workspace of %zu bytes: %s", total, hipGetErrorString(e));
  }
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
  a.ckpt = reinterpret_cast<double*>(take(b_ckpt));
  a.ck_served = reinterpret_cast<int64_t*>(take(b_cks));
  a.ck_fsum = reinterpret_cast<uint64_t*>(take(b_cks));
  int32_t* small = reinterpret_cast<int32_t*>(take(b_small));
  a.cfg_info = small;
  a.changed = small + 64;

  hipLaunchKernelGGL(spec_cfg_check, dim3(1), dim3(1024), 0, stream, k.group_cfg, (int64_t)k.P * k.G, k.C,
                     a.cfg_info);
  switch (smax) {
    case 1: e = spec_launch_mb<1>(k.G, a, lds_u, lds_g, stream); break;
    case 2: e = spec_launch_mb<2>(k.G, a, lds_u, lds_g, stream); break;
    case 4: e = spec_launch_mb<4>(k.G, a, lds_u, lds_g, stream); break;
    default: e = spec_launch_mb<8>(k.G, a, lds_u, lds_g, stream); break;
  }
  if (e != hipSuccess || !can_give_up) {
    const hipError_t ef = caller_ws ? hipSuccess : hipFreeAsync(ws, stream);
    if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    if (ef != hipSuccess) return fail(AS_E_HIP, "workspace release failed: %s", hipGetErrorString(ef));
    return ok();
  }
  *workspace = caller_ws ? nullptr : ws;
  *gave_up = a.cfg_info + 2;
  return ok();
}

}  // namespace as_host
