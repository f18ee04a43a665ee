// Dynamic batching (Sec. 6.5) on the batched simulator: an arriving request
// runs at once on an available group hosting its model, otherwise it waits in
// a per-model queue; a group that becomes idle runs the largest batch of one
// hosted model's queued requests that still meets the SLO; a batch's latency
// grows linearly with its size.  The exact rules are those of
// alpaserve_sim.h's as_simulate_batched.
//
// A queue needs no storage of its own.  A request joins its model's queue
// only when no hosting group is available at its arrival, and a group that
// is available then has already drained every queue of the models it hosts
// (the idle events up to the arrival are handled first, and a group with
// queued work stays busy or takes that work).  So an arrival served or
// dropped at once finds its model's queue empty, and a non-empty queue holds
// every arrival of its model since its head.  Requests leave a queue only at
// its head.  A queue is therefore a run [head, tail) of its model's arrivals
// in trace order: the launch first lists each model's arrivals (time, trace
// index, digest term) once for all jobs, and a job keeps per model only two
// positions in that list and its head's time and index.
//
// Layout: one job per wavefront (one wavefront per workgroup).  Lane g holds
// group g's stage free times; lane m holds model m's queue (positions, head
// time and index, SLO); the trace is read 64 requests at a time into
// registers.  Every decision is wave-uniform: the next idle group is a
// butterfly min over the lanes with queued work, the model with the oldest
// queued head a scalar pass over lane reads, and the batch size one pass in
// which lane l runs the chain of a batch of l + 1 requests.  Only the
// stage-latency table sits in LDS, so every job of a launch is resident at
// once.  The arithmetic is the definition's (no FMA, v_max_f64, the batch
// factor rounded once), so served counts, digests and finish times are
// bit-identical to a sequential evaluation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "alpaserve_sim.h"
#include "sim_internal.hpp"
#include "sim_kernel.hpp"

namespace as_dev {
namespace {

// Per-model arrival lists of a trace: the requests of model m in trace order
// occupy positions [off[m], off[m + 1]) of lt (arrival time), li (trace
// index) and lmix (the digest term of the index); ord[i] is request i's rank
// among its model's requests (0 for requests of no model).
struct ListArgs {
  const double* t;
  const int32_t* model;
  int64_t n;
  int32_t M;
  uint32_t* blk;  // [nblk][M] requests of each model per block, then the exclusive prefix over blocks
  int64_t nblk;
  uint32_t* off;  // [M + 1]
  uint32_t* ord;  // [n]
  double* lt;     // [n]
  uint32_t* li;   // [n]
  uint64_t* lmix; // [n]
  uint32_t* flags;  // the batch kernel's flags word (cleared here)
};

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
  uint32_t* flags;  // bit 0: a queue would exceed its capacity; bit 1: a queue broke the run invariant
  const uint32_t* off;
  const uint32_t* ord;
  const double* lt;
  const uint32_t* li;
  const uint64_t* lmix;
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

__device__ __forceinline__ uint64_t rl_u64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

constexpr int kListBlock = 4096;  // trace requests per wavefront of the list kernels

// Walks one block's requests 64 at a time; for every chunk, body(i, ok, x,
// rank_base, mask) is called once per distinct model x of the chunk, where
// mask holds the chunk's lanes with model x and rank_base the number of
// earlier requests of x in the block (held in lane x of cnt).
template <class Body>
__device__ __forceinline__ void list_walk(const ListArgs& a, int64_t blk, uint32_t& cnt, Body body) {
  const int lane = threadIdx.x;
  const uint64_t below = (1ull << lane) - 1;
  const int64_t b = blk * kListBlock, e = std::min<int64_t>(a.n, b + kListBlock);
  for (int64_t c = b; c < e; c += 64) {
    const int64_t i = c + lane;
    const int x = i < e ? a.model[i] : -1;
    const bool ok = (unsigned)x < (unsigned)a.M;
    uint64_t rem = __builtin_amdgcn_ballot_w64(ok);
    uint32_t rank = 0;
    while (rem) {
      const int xm = __builtin_amdgcn_readlane(x, __builtin_ctzll(rem));
      const uint64_t mask = __builtin_amdgcn_ballot_w64(ok && x == xm);
      const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)cnt, xm);
      if (ok && x == xm) rank = base + (uint32_t)__builtin_popcountll(mask & below);
      if (lane == xm) cnt += (uint32_t)__builtin_popcountll(mask);
      rem &= ~mask;
    }
    body(i, i < e, ok, x, rank);
  }
}

// Requests of each model per block.
__global__ __launch_bounds__(64) void list_count(const ListArgs a) {
  uint32_t cnt = 0;
  list_walk(a, blockIdx.x, cnt, [](int64_t, bool, bool, int, uint32_t) {});
  if ((int)threadIdx.x < a.M) a.blk[(int64_t)blockIdx.x * a.M + threadIdx.x] = cnt;
}

// Exclusive prefixes: per model over the blocks, then over the models.
__global__ __launch_bounds__(64) void list_scan(const ListArgs a) {
  const int lane = threadIdx.x;
  uint32_t run = 0;
  if (lane < a.M) {
    for (int64_t b = 0; b < a.nblk; b += 8) {  // 8 loads in flight at a time
      uint32_t v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = b + k < a.nblk ? a.blk[(b + k) * a.M + lane] : 0u;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (b + k < a.nblk) a.blk[(b + k) * a.M + lane] = run;
        run += v[k];
      }
    }
  }
  uint32_t acc = 0, mine = 0;
  for (int m = 0; m < a.M; ++m) {
    if (lane == m) mine = acc;
    acc += (uint32_t)__builtin_amdgcn_readlane((int)run, m);
  }
  if (lane < a.M) a.off[lane] = mine;
  if (lane == 0) {
    a.off[a.M] = acc;
    *a.flags = 0u;
  }
}

// Ranks and list entries.
__global__ __launch_bounds__(64) void list_fill(const ListArgs a) {
  const int lane = threadIdx.x;
  uint32_t cnt = lane < a.M ? a.blk[(int64_t)blockIdx.x * a.M + lane] : 0;
  const uint32_t offl = lane < a.M ? a.off[lane] : 0;
  list_walk(a, blockIdx.x, cnt, [&](int64_t i, bool in, bool ok, int x, uint32_t rank) {
    const uint32_t o = (uint32_t)__builtin_amdgcn_ds_bpermute((ok ? x : 0) << 2, (int)offl);
    if (!in) return;
    a.ord[i] = ok ? rank : 0u;
    if (ok) {
      const uint32_t pos = o + rank;
      a.lt[pos] = a.t[i];
      a.li[pos] = (uint32_t)i;
      a.lmix[pos] = mix64((uint64_t)i);
    }
  });
}

// LDS of one job: the stage-latency table [M][Cp][SMAX].
__host__ __device__ constexpr size_t batch_lds_bytes(int M, int Cp, int SMAX) {
  return (size_t)M * Cp * SMAX * 8;
}

// W: lanes reduced per job, the group count rounded up to a power of two (at
// least 16, so the reductions inside a 16-lane row are DPP only).
template <int W, int SMAX>
__global__ __launch_bounds__(64) void batch_kernel(const BatchArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  int cp = 1;
  while (cp < a.C) cp <<= 1;
  double* sL = reinterpret_cast<double*>(smem);  // [M][cp][SMAX]
  const int lane = threadIdx.x;
  const int64_t job = blockIdx.x;
  const int p = (int)(job / a.K);
  const double sigma = a.slo_scale[job % a.K];

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
  int frow = -1;
  for (int f = 0; f < a.n_finish; ++f)
    if (a.finish_jobs[f] == job) frow = f;
  double* frowp = frow >= 0 ? a.out_finish + (int64_t)frow * a.n : nullptr;
  __syncthreads();

  // lane m: model m's SLO and queue, the run [qh, qt) of its list starting
  // at loff, with the head's arrival time and trace index
  const bool mlane = lane < a.M;
  const double slo = mlane ? sigma * a.d_single[lane] : 0.0;
  const uint32_t loff = mlane ? a.off[lane] : 0u;
  uint32_t qh = 0, qt = 0, qidx = 0;
  double qht = 0.0;
  uint64_t nonempty = 0;  // bit m: model m has queued requests (wave-uniform)

  const double* lbase = sL + (size_t)(cfg < 0 ? 0 : cfg) * SMAX;  // + m * cp * SMAX
  double F[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) F[s] = 0.0;
  uint64_t h = 0, fin_sum = 0;  // wave-uniform parts of the digest
  uint64_t hl = 0, pend = 0;    // per-lane digest terms of batched requests (pend: the last batch's, in flight)
  int64_t served = 0;
  uint32_t flags = 0;
  const double kInf = __builtin_inf();

  // every lane's chain, through its own group, for one request of model m
  // started at x; returns the last stage's finish, fs[] its stage finishes
  auto chain1 = [&](int m, double x, double (&fs)[SMAX]) {
    const double fac = 1.0 + a.beta * 0.0;
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
  // model mc's queue head moves to list position hn (< tail: its entry is
  // loaded by lane mc; the value is first needed at the next decision)
  auto set_head = [&](int mc, uint32_t hn, uint32_t tl) {
    if (lane == mc) qh = hn;
    if (hn == tl) {
      nonempty &= ~(1ull << mc);
    } else if (lane == mc) {
      qht = a.lt[loff + hn];
      qidx = a.li[loff + hn];
    }
  };

  // the trace, 64 requests per register chunk, the next chunk in flight
  auto load_chunk = [&](int64_t base, double& tv, int& mv, uint32_t& ov) {
    const int64_t i = base + lane;
    tv = i < a.n ? a.t[i] : 0.0;
    mv = i < a.n ? a.model[i] : -1;
    ov = i < a.n ? a.ord[i] : 0u;
  };
  double tv, tvn = 0.0;
  int mv, mvn = -1;
  uint32_t ov, ovn = 0;
  load_chunk(0, tv, mv, ov);

  for (int64_t base = 0; base <= a.n; base += 64) {
    const int cnt = (int)((a.n - base) < 64 ? (a.n - base) : 64);
    if (base + 64 < a.n) load_chunk(base + 64, tvn, mvn, ovn);
    // cnt requests of this chunk, then (after the last one) the final drain
    const int steps = base + 64 > a.n ? cnt + 1 : cnt;
    for (int e = 0; e < steps; ++e) {
      const bool last = e == cnt;
      const int64_t i = base + e;
      const double horizon = last ? 0.0 : rl_f64(tv, e);
      // idle events up to the arrival (all remaining ones after the last)
      for (;;) {
        const bool work = cfg >= 0 && (hostbits & nonempty) != 0;
        const double key = work ? F[0] : kInf;
        const double mn = wave_min(key);
        const uint64_t wm = __builtin_amdgcn_ballot_w64(work && key == mn);
        if (wm == 0) break;
        if (!last && !(mn <= horizon)) break;
        const int g = __builtin_ctzll(wm);
        const uint64_t ghost = rl_u64(hostbits, g);
        const int gcfg = __builtin_amdgcn_readlane(cfg, g);
        double Fg[SMAX];
#pragma unroll
        for (int s = 0; s < SMAX; ++s) Fg[s] = rl_f64(F[s], g);
        for (;;) {
          uint64_t cand = ghost & nonempty;
          if (cand == 0) break;  // nothing left for this group: it stays idle
          // the queued model whose head has the lowest trace index
          int mc = __builtin_ctzll(cand);
          uint32_t hidx = (uint32_t)__builtin_amdgcn_readlane((int)qidx, mc);
          cand &= cand - 1;
          while (cand) {
            const int m = __builtin_ctzll(cand);
            cand &= cand - 1;
            const uint32_t r = (uint32_t)__builtin_amdgcn_readlane((int)qidx, m);
            if (r < hidx) {
              mc = m;
              hidx = r;
            }
          }
          const uint32_t h0 = (uint32_t)__builtin_amdgcn_readlane((int)qh, mc);
          const uint32_t tl = (uint32_t)__builtin_amdgcn_readlane((int)qt, mc);
          const double dl = rl_f64(qht + slo, mc);  // the head's deadline
          const uint32_t avail = tl - h0;
          const int bmax = (int)(avail < (uint32_t)a.max_batch ? avail : (uint32_t)a.max_batch);
          // the largest batch meeting the deadline: the sizes are tried 64 at
          // a time, lane l the size p0 + l + 1, and the first size that
          // misses ends the search (as trying them one by one would)
          const double* L = sL + ((size_t)mc * cp + gcfg) * SMAX;
          int b = 0;
          double fin = 0.0;
          double fsel[SMAX];
#pragma unroll
          for (int s = 0; s < SMAX; ++s) fsel[s] = 0.0;
          for (int p0 = 0; p0 < bmax; p0 += 64) {
            const int bb = p0 + lane + 1;
            const double fac = 1.0 + a.beta * (double)(bb - 1);
            double f = mn;
            double fs[SMAX];
#pragma unroll
            for (int s = 0; s < SMAX; ++s) {
              fs[s] = vmax(f, Fg[s]) + L[s] * fac;
              f = fs[s];
            }
            const uint64_t miss = __builtin_amdgcn_ballot_w64(bb <= bmax && f > dl);
            const int lim = bmax - p0 < 64 ? bmax - p0 : 64;
            const int nok = miss ? __builtin_ctzll(miss) : lim;  // sizes p0+1 .. p0+nok meet it
            if (nok > 0) {
              b = p0 + nok;
              fin = rl_f64(f, nok - 1);
#pragma unroll
              for (int s = 0; s < SMAX; ++s) fsel[s] = rl_f64(fs[s], nok - 1);
            }
            if (nok < 64) break;
          }
          if (b == 0) {
            // the head cannot meet its deadline: dropped (its output stays -1)
            set_head(mc, h0 + 1, tl);
            continue;
          }
          if (lane == g) {
#pragma unroll
            for (int s = 0; s < SMAX; ++s) F[s] = fsel[s];
          }
          // the batch's digest terms: the first 64 arrive while the
          // simulation goes on and are added at the next batch
          const uint32_t lb0 = (uint32_t)__builtin_amdgcn_readlane((int)loff, mc) + h0;
          hl += pend;
          pend = 0;
          if (lane < b) pend = a.lmix[lb0 + lane];
          for (int k0 = 64; k0 < b; k0 += 64)
            if (k0 + lane < b) hl += a.lmix[lb0 + k0 + lane];
          fin_sum += (uint64_t)b * (uint64_t)__double_as_longlong(fin);
          served += b;
          if (frowp) {
            for (int k0 = 0; k0 < b; k0 += 64)
              if (k0 + lane < b) frowp[a.li[lb0 + k0 + lane]] = fin;
          }
          set_head(mc, h0 + (uint32_t)b, tl);
          break;
        }
      }
      if (last) break;
      // the arrival
      const double ti = horizon;
      const int m0 = __builtin_amdgcn_readlane(mv, e);
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
        const double fl = rl_f64(chain1(m, ti, fs), ga);
        if (!(fl > ti + rl_f64(slo, m))) {
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
        const uint32_t rank = (uint32_t)__builtin_amdgcn_readlane((int)ov, e);
        uint32_t hd = (uint32_t)__builtin_amdgcn_readlane((int)qh, m);
        const uint32_t tl = (uint32_t)__builtin_amdgcn_readlane((int)qt, m);
        while (hd != tl && rl_f64(qht + slo, m) < lb) {
          ++hd;
          set_head(m, hd, tl);
        }
        if (hd == tl) {
          // an empty queue: request i becomes its head
          if (lane == m) {
            qh = rank;
            qht = ti;
            qidx = (uint32_t)i;
          }
        } else {
          if (rank != tl) flags |= 2u;  // not the run's next arrival (cannot happen by the rules)
          if (tl - hd >= (uint32_t)a.qcap) flags |= 1u;  // past the capacity: the results are incomplete
        }
        if (lane == m) qt = rank + 1;
        nonempty |= 1ull << m;
      }
    }
    tv = tvn;
    mv = mvn;
    ov = ovn;
  }
  hl += pend;
  const uint64_t hsum = seg_sum_u64<64>(hl);
  if (lane == 0) {
    if (flags) atomicOr(a.flags, flags);
    a.out_served[job] = served;
    if (a.out_digest) {
      a.out_digest[2 * job] = h + hsum;
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
  const size_t lds = as_dev::batch_lds_bytes(ka.M, pow2ceil(ka.C), smax);
  if (lds > shared_lds_limit())
    return fail(AS_E_LIMITS, "batched: the stage-latency table needs %zu bytes of LDS (> %zu)", lds,
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
  // one workspace: the flags word, then the per-model arrival lists
  as_dev::ListArgs la;
  std::memset(&la, 0, sizeof la);
  la.t = trace->t;
  la.model = trace->model;
  la.n = trace->n;
  la.M = ka.M;
  la.nblk = (trace->n + as_dev::kListBlock - 1) / as_dev::kListBlock;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t n = (size_t)trace->n;
  const size_t o_blk = 256, o_off = o_blk + up((size_t)la.nblk * ka.M * 4), o_ord = o_off + up((size_t)(ka.M + 1) * 4),
               o_lt = o_ord + up(n * 4), o_li = o_lt + up(n * 8), o_mix = o_li + up(n * 4), total = o_mix + up(n * 8);
  unsigned char* ws = nullptr;
  hipError_t e = pool_alloc(reinterpret_cast<void**>(&ws), total, s);
  if (e != hipSuccess) return fail(AS_E_NOMEM, "device allocation of %zu bytes: %s", total, hipGetErrorString(e));
  a.flags = reinterpret_cast<uint32_t*>(ws);
  la.flags = a.flags;
  la.blk = reinterpret_cast<uint32_t*>(ws + o_blk);
  la.off = reinterpret_cast<uint32_t*>(ws + o_off);
  la.ord = reinterpret_cast<uint32_t*>(ws + o_ord);
  la.lt = reinterpret_cast<double*>(ws + o_lt);
  la.li = reinterpret_cast<uint32_t*>(ws + o_li);
  la.lmix = reinterpret_cast<uint64_t*>(ws + o_mix);
  a.off = la.off;
  a.ord = la.ord;
  a.lt = la.lt;
  a.li = la.li;
  a.lmix = la.lmix;
  if (la.nblk > 0) hipLaunchKernelGGL(as_dev::list_count, dim3((unsigned)la.nblk), dim3(64), 0, s, la);
  hipLaunchKernelGGL(as_dev::list_scan, dim3(1), dim3(64), 0, s, la);  // also clears the flags
  if (la.nblk > 0) hipLaunchKernelGGL(as_dev::list_fill, dim3((unsigned)la.nblk), dim3(64), 0, s, la);
  e = hipGetLastError();
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
  if (e == hipSuccess) e = hipMemcpyAsync(&flag, a.flags, sizeof flag, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  const hipError_t ef = hipFreeAsync(ws, s);
  if (e == hipSuccess) e = ef;
  if (e != hipSuccess) return fail(AS_E_HIP, "batched: %s", hipGetErrorString(e));
  if (flag & 2u)
    return fail(AS_E_INVALID_DATA, "batched: a queue was not a run of its model's arrivals; results are invalid");
  if (flag & 1u) return fail(AS_E_LIMITS, "batched: a model queue exceeded queue_cap=%d; results are incomplete", queue_cap);
  return ok();
}
