// C-ABI of the batched serving simulator: argument checks, kernel selection,
// launches on the caller's stream, error reporting.  See alpaserve_sim.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "alpaserve_sim.h"
#include "sim_kernel.hpp"
#include "sim_shared.hpp"
#include "sim_launch.hpp"
#include "sim_internal.hpp"

namespace as_host {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return AS_OK;
}

int pow2ceil(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

using as_dev::KArgs;

// LDS bytes of one workgroup for lanes-per-job W and padded stage count SMAX.
size_t lds_bytes(int W, int SMAX, bool seg, int M, int C) {
  const int slots = (64 / W) * as_dev::kWaves;
  int ch = as_dev::kChunk;
  if (seg) {
    ch = 4096 / slots;
    if (ch > 128) ch = 128;
    if (ch < 32) ch = 32;
    ch *= slots;
  }
  return (size_t)M * pow2ceil(C) * SMAX * 8 + (size_t)M * 8 + (size_t)ch * 12;
}

constexpr size_t kMaxLds = 64 * 1024;

// LDS a workgroup of the shared-trace kernel may use: the device's per-block
// limit (160 KiB on gfx950), cached per device.
size_t shared_lds_limit() {
  static size_t cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return kMaxLds;
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
      v = (int)kMaxLds;
    cache[dev] = (size_t)(v > 160 * 1024 ? 160 * 1024 : v);
  }
  return cache[dev];
}


hipError_t launch_lds_any(int W, int gpl, int smax, bool seg, const KArgs& a, size_t lds, hipStream_t s) {
  switch (W) {
    case 1: return as_host::launch_lds<1>(gpl, smax, seg, a, lds, s);
    case 2: return as_host::launch_lds<2>(gpl, smax, seg, a, lds, s);
    case 4: return as_host::launch_lds<4>(gpl, smax, seg, a, lds, s);
    case 8: return as_host::launch_lds<8>(gpl, smax, seg, a, lds, s);
    case 16: return as_host::launch_lds<16>(gpl, smax, seg, a, lds, s);
    case 32: return as_host::launch_lds<32>(gpl, smax, seg, a, lds, s);
    default: return as_host::launch_lds<64>(gpl, smax, seg, a, lds, s);
  }
}

hipError_t launch_shared_any(int W, int smax, bool usig, const KArgs& a, size_t lds, hipStream_t s,
                             bool stats) {
  switch (W) {
    case 1: return as_host::launch_shared<1>(smax, usig, stats, a, lds, s);
    case 2: return as_host::launch_shared<2>(smax, usig, stats, a, lds, s);
    case 4: return as_host::launch_shared<4>(smax, usig, stats, a, lds, s);
    case 8: return as_host::launch_shared<8>(smax, usig, stats, a, lds, s);
    case 16: return as_host::launch_shared<16>(smax, usig, stats, a, lds, s);
    case 32: return as_host::launch_shared<32>(smax, usig, stats, a, lds, s);
    default: return as_host::launch_shared<64>(smax, usig, stats, a, lds, s);
  }
}

// SIMDs of the current device (4 per compute unit), cached per device.
int simd_count() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (cache[dev] == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return 1024;
    cache[dev] = prop.multiProcessorCount * 4;
  }
  return cache[dev];
}

// Lanes per job W and groups per lane GPL (W * GPL >= G, powers of two).
// Cost model: a wavefront issues in order, so the time of a launch is about
// (wavefronts per SIMD, at least 1) x (instructions per request of one
// wavefront); a lane that carries more groups needs more instructions per
// request but fewer wavefronts.  Relative instruction counts per request for
// GPL = 1, 2, 4 are measured values.  Shapes whose LDS tables do not fit are
// skipped (a wider W means fewer job slots per workgroup).  ALPASERVE_GPL=1|2|4
// forces GPL.  Returns false when no shape fits.
bool choose_shape(int G, int64_t J, bool seg, int M, int C, int smax, int& W, int& GPL,
                  bool allow_force = true) {
  const int Gp = pow2ceil(G);
  const double instr[3] = {1.0, 1.45, 2.3};
  const int n_simd = simd_count();
  int force = 0;
  if (const char* e = getenv("ALPASERVE_GPL"); e && allow_force) force = atoi(e);
  double best = 1e300;
  bool found = false;
  for (int i = 0; i < 3; ++i) {
    const int gpl = 1 << i;
    if (gpl > Gp || (force && force != gpl)) continue;
    for (int w = Gp / gpl; w <= 64 && w * gpl <= 64; w *= 2) {
      if (lds_bytes(w, smax, seg, M, C) > kMaxLds) continue;
      const int64_t waves = (J + (64 / w) - 1) / (64 / w);
      const double occ = (double)waves / n_simd;
      const double cost = (occ > 1.0 ? occ : 1.0) * instr[i];
      if (cost < best) {
        best = cost;
        W = w;
        GPL = gpl;
        found = true;
      }
      break;  // the narrowest W that fits is the cheapest for this GPL
    }
  }
  // a forced GPL that does not apply to this problem yields to the cost model
  if (!found && force) return choose_shape(G, J, seg, M, C, smax, W, GPL, false);
  return found;
}

// Which kernel family runs a shared-trace call: by default the
// segment-speculative kernels when the trace splits into segments, else the
// shared-trace kernel; ALPASERVE_PATH=lds selects the LDS-staged kernel,
// =spec the segment-speculative one, =shared the shared-trace one (tests
// cover each).
bool use_shared_path() {
  const char* e = getenv("ALPASERVE_PATH");
  return !(e && std::strcmp(e, "lds") == 0);
}

// The segment-speculative kernels take a call unless another family is
// forced; they decline (AS_E_LIMITS) calls they cannot cut into segments.
bool want_spec(const KArgs& a, int smax) {
  (void)a;
  (void)smax;
  const char* e = getenv("ALPASERVE_PATH");
  return !(e && *e) || std::strcmp(e, "spec") == 0;
}

bool spec_forced() {
  const char* e = getenv("ALPASERVE_PATH");
  return e && std::strcmp(e, "spec") == 0;
}

// Checks shared by both simulate entry points; fills the model/placement part
// of KArgs and the kernel shape.
int check_common(const as_models_t* models, const as_placements_t* plc, KArgs& a, int& W,
                 int& smax) {
  if (!models || !plc) return fail(AS_E_INVALID_ARG, "models and placements must not be NULL");
  const as_models_t& md = *models;
  const as_placements_t& pl = *plc;
  if (md.n_models < 1 || md.n_models > AS_MAX_MODELS)
    return fail(md.n_models < 1 ? AS_E_INVALID_ARG : AS_E_LIMITS, "n_models=%d outside 1..%d",
                md.n_models, AS_MAX_MODELS);
  if (md.n_configs < 1 || md.n_configs > AS_MAX_CONFIGS)
    return fail(md.n_configs < 1 ? AS_E_INVALID_ARG : AS_E_LIMITS, "n_configs=%d outside 1..%d",
                md.n_configs, AS_MAX_CONFIGS);
  if (md.max_stages < 1) return fail(AS_E_INVALID_ARG, "max_stages=%d < 1", md.max_stages);
  if (!md.d_single || !md.stage_lat || !md.cfg_stages)
    return fail(AS_E_INVALID_ARG, "d_single, cfg_stages and stage_lat must not be NULL");
  int smax_used = 1;
  for (int c = 0; c < md.n_configs; ++c) {
    const int S = md.cfg_stages[c];
    if (S < 1 || S > md.max_stages)
      return fail(AS_E_INVALID_ARG, "cfg_stages[%d]=%d outside 1..max_stages=%d", c, S, md.max_stages);
    if (S > AS_MAX_STAGES)
      return fail(AS_E_LIMITS, "cfg_stages[%d]=%d > %d", c, S, AS_MAX_STAGES);
    if (S > smax_used) smax_used = S;
  }
  if (pl.n_placements < 0) return fail(AS_E_INVALID_ARG, "n_placements=%d < 0", pl.n_placements);
  if (pl.max_groups < 1 || pl.max_groups > AS_MAX_GROUPS)
    return fail(pl.max_groups < 1 ? AS_E_INVALID_ARG : AS_E_LIMITS, "max_groups=%d outside 1..%d",
                pl.max_groups, AS_MAX_GROUPS);
  if (pl.n_placements > 0 && (!pl.group_cfg || !pl.host_mask))
    return fail(AS_E_INVALID_ARG, "group_cfg and host_mask must not be NULL");
  a.d_single = md.d_single;
  a.stage_lat = md.stage_lat;
  a.group_cfg = pl.group_cfg;
  a.host_mask = pl.host_mask;
  a.M = md.n_models;
  a.C = md.n_configs;
  a.smax_in = md.max_stages;
  a.G = pl.max_groups;
  a.P = pl.n_placements;
  for (int c = 0; c < AS_MAX_CONFIGS; ++c) a.cfg_stages[c] = c < md.n_configs ? md.cfg_stages[c] : 1;
  W = pl.max_groups;  // group count; the shape is chosen per call
  smax = pow2ceil(smax_used);
  return AS_OK;
}

int check_finish(const int32_t* finish_jobs, int32_t n_finish, double* out_finish, int64_t J,
                 KArgs& a) {
  if (n_finish < 0) return fail(AS_E_INVALID_ARG, "n_finish=%d < 0", n_finish);
  if (n_finish > AS_MAX_FINISH) return fail(AS_E_LIMITS, "n_finish=%d > %d", n_finish, AS_MAX_FINISH);
  if (n_finish > 0 && (!finish_jobs || !out_finish))
    return fail(AS_E_INVALID_ARG, "finish_jobs and out_finish must not be NULL when n_finish > 0");
  for (int f = 0; f < n_finish; ++f) {
    if (finish_jobs[f] < 0 || finish_jobs[f] >= J)
      return fail(AS_E_INVALID_ARG, "finish_jobs[%d]=%d outside [0, %lld)", f, finish_jobs[f],
                  (long long)J);
    for (int q = 0; q < f; ++q)
      if (finish_jobs[q] == finish_jobs[f])
        return fail(AS_E_INVALID_ARG, "finish_jobs[%d] repeats job %d", f, finish_jobs[f]);
    a.finish_jobs[f] = finish_jobs[f];
  }
  a.n_finish = n_finish;
  a.out_finish = out_finish;
  return AS_OK;
}


// ---------------------------------------------------------------- validation
enum : uint32_t {
  V_T_ORDER = 1u << 0,   // t not finite, negative or decreasing
  V_MODEL = 1u << 1,     // model id out of range
  V_CFG = 1u << 2,       // group configuration outside [-1, C)
  V_MASK = 1u << 3,      // hosting bit on a missing group
  V_LAT = 1u << 4,       // stage latency not finite or negative
  V_DSINGLE = 1u << 5,   // d_single not finite or not positive
  V_SCALE = 1u << 6,     // SLO scale negative or NaN
};
const char* kValidateMsg[] = {
    "trace times must be finite, >= 0 and nondecreasing",
    "model ids must lie in [0, n_models)",
    "group_cfg entries must lie in [-1, n_configs)",
    "host_mask may only set bits of groups with group_cfg >= 0",
    "stage latencies (s < S_c) must be finite and >= 0",
    "d_single must be finite and > 0",
    "slo_scale must be >= 0 and not NaN",
};

__global__ void validate_kernel(const double* t, const int32_t* model, int64_t n, int M, int C,
                                const int32_t* group_cfg, const uint64_t* host_mask, int64_t P, int G,
                                const double* stage_lat, int smax_in, const double* d_single,
                                const double* scales, int K, KArgs cfgs, uint32_t* flags) {
  uint32_t bad = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t tid0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = tid0; i < n; i += stride) {
    const double ti = t[i];
    if (!(ti >= 0.0) || !(ti <= 1.7976931348623157e308)) bad |= V_T_ORDER;
    if (i > 0 && !(t[i - 1] <= ti)) bad |= V_T_ORDER;
    const int32_t m = model[i];
    if (m < 0 || m >= M) bad |= V_MODEL;
  }
  for (int64_t j = tid0; j < P * G; j += stride) {
    const int32_t c = group_cfg[j];
    if (c < -1 || c >= C) bad |= V_CFG;
  }
  for (int64_t j = tid0; j < P * M; j += stride) {
    const int64_t p = j / M;
    const uint64_t mask = host_mask[j];
    for (int g = 0; g < 64; ++g)
      if ((mask >> g) & 1u)
        if (g >= G || group_cfg[p * G + g] < 0) bad |= V_MASK;
  }
  for (int64_t j = tid0; j < (int64_t)M * C * smax_in; j += stride) {
    const int s = (int)(j % smax_in);
    const int c = (int)((j / smax_in) % C);
    const double v = stage_lat[j];
    if (s < cfgs.cfg_stages[c] && (!(v >= 0.0) || !(v <= 1.7976931348623157e308))) bad |= V_LAT;
  }
  for (int64_t j = tid0; j < M; j += stride) {
    const double d = d_single[j];
    if (!(d > 0.0) || !(d <= 1.7976931348623157e308)) bad |= V_DSINGLE;
  }
  for (int64_t j = tid0; j < K; j += stride)
    if (!(scales[j] >= 0.0)) bad |= V_SCALE;
  if (bad) atomicOr(flags, bad);
}

// Fill p[0, n) with v (per-request output rows before a shared-trace launch);
// nothing when gate is set and *gate == 0.
__global__ void fill_f64(double* __restrict__ p, int64_t n, double v, const int32_t* gate) {
  if (gate && *gate == 0) return;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Fill the per-request output rows of segmented jobs with -2 over
// [0, min(segment length, finish_stride)) (the rest stays untouched).
__global__ void fill_seg_rows(const KArgs a) {
  const int64_t total = (int64_t)a.n_finish * a.finish_stride;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int f = (int)(i / a.finish_stride);
    const int64_t k = i % a.finish_stride;
    int p = 0;
    double sigma = 0.0;
    int64_t begin = 0, len = 0;
    as_dev::seg_job(a, a.finish_jobs[f], p, sigma, begin, len);
    if (k < len) a.out_finish[i] = -2.0;
  }
}

// Statistics launch of the shared-trace kernel (one SLO scale, no per-request
// rows): AS_E_LIMITS when its tables do not fit in a workgroup's LDS.
int run_shared_stats(KArgs& a, int smax, hipStream_t stream) {
  const int Ws = pow2ceil(a.G);
  const size_t lds = as_dev::shared_lds_bytes(a.M, pow2ceil(a.C), smax) + as_dev::shared_stats_lds_bytes(Ws, a.M);
  if (!use_shared_path() || a.K != 1 || a.n_finish != 0 || lds > shared_lds_limit())
    return AS_E_LIMITS;
  const hipError_t e = launch_shared_any(Ws, smax, true, a, lds, stream, true);
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// Multi-shape dispatches pay where the jobs are few: a step whose shapes run
// on separate streams costs a trace pass of latency per shape that shares a
// hardware queue.  Where the blocks fill the device many times over, launches
// of their own shapes run faster (the multi-shape kernel holds the registers
// and LDS of its largest shape), and they overlap anyway.
constexpr int64_t kMultiMaxBlocks = 2048;

int run_shared_multi(const KArgs& a, void* dev_args, const ShapeJobs* sh, int n, bool stats, hipStream_t stream) {
  if (!use_shared_path() || a.K != 1 || a.n_finish != 0 || n < 1 || n > as_dev::kMaxShapeSegs || !dev_args)
    return AS_E_LIMITS;
  size_t lds = 0;
  as_dev::MultiSegs ms;
  std::memset(&ms, 0, sizeof ms);
  int64_t blocks = 0;
  for (int i = 0; i < n; ++i) {
    const int W = sh[i].W, sm = sh[i].smax;
    if (W < 1 || W > 64 || (W & (W - 1)) != 0 || sh[i].v.G > W || (sm != 1 && sm != 2 && sm != 4 && sm != 8))
      return AS_E_LIMITS;
    if (sh[i].v.J <= 0) continue;
    if (!stats) {
      KArgs ak = a;
      ak.J = sh[i].v.J;
      ak.G = sh[i].v.G;
      if (want_spec(ak, sm) && spec_takes(ak, sm)) return AS_E_LIMITS;
    }
    const size_t l = as_dev::shared_lds_bytes(a.M, pow2ceil(a.C), sm) +
                     (stats ? as_dev::shared_stats_lds_bytes(W, a.M) : 0);
    lds = std::max(lds, l);
    as_dev::ShapeSeg& g = ms.s[ms.n++];
    int wl = 0, sl = 0;
    while ((1 << wl) < W) ++wl;
    while ((1 << sl) < sm) ++sl;
    g.wl = wl;
    g.sl = sl;
    g.block0 = blocks;
    g.v = sh[i].v;
    const int64_t slots = (int64_t)(64 / W) * as_dev::kWaves;
    blocks += (sh[i].v.J + slots - 1) / slots;
  }
  if (lds > shared_lds_limit() || blocks > kMultiMaxBlocks) return AS_E_LIMITS;
  if (ms.n == 0) return ok();
  hipError_t e = hipMemcpyAsync(dev_args, &a, sizeof(KArgs), hipMemcpyHostToDevice, stream);
  if (e == hipSuccess) e = launch_shared_multi(stats, static_cast<const KArgs*>(dev_args), ms, blocks, lds, stream);
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// The shared-trace kernel (one group per lane, W = G rounded up to a power of
// two) unless its tables exceed the LDS of a workgroup; then the general
// kernel, whose tables are smaller.  With only_check, whether one of them
// takes the call (AS_OK) or not (AS_E_LIMITS), without launching.
int run_trace_kernels(KArgs& a, int W, int smax, hipStream_t stream, bool only_check) {
  const int64_t J = a.J;
  const size_t lds_shared = as_dev::shared_lds_bytes(a.M, pow2ceil(a.C), smax);
  if (use_shared_path() && lds_shared <= shared_lds_limit()) {
    if (only_check) return AS_OK;
    const int Ws = pow2ceil(a.G);
    hipError_t e = hipSuccess;
    if (a.n_finish > 0 && a.n > 0) {
      // rows start at -2 (no hosting group); the kernel writes the others
      const int64_t cells = (int64_t)a.n_finish * a.n;
      const int64_t blocks = std::min<int64_t>((cells + 255) / 256, 8192);
      hipLaunchKernelGGL(fill_f64, dim3((unsigned)blocks), dim3(256), 0, stream, a.out_finish,
                         cells, -2.0, a.gate);
      if ((e = hipGetLastError()) != hipSuccess)
        return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    }
    e = launch_shared_any(Ws, smax, a.K == 1, a, lds_shared, stream, false);
    if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return ok();
  }
  int GPL = 1;
  if (!choose_shape(a.G, J, false, a.M, a.C, smax, W, GPL))
    return only_check ? AS_E_LIMITS
                      : fail(AS_E_LIMITS, "stage-latency tables (%d models x %d configs x %d stages) do not fit in LDS",
                             a.M, a.C, smax);
  if (only_check) return AS_OK;
  const size_t lds = lds_bytes(W, smax, false, a.M, a.C);
  hipError_t e = launch_lds_any(W, GPL, smax, false, a, lds, stream);
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

// Launch the batched simulation of a shared trace (a fully filled except the
// kernel shape).  W is the group count on entry.  The segment-speculative
// kernels go first where they take the call; when one of their re-runs gives
// up (traffic under which runs from different states do not meet), the
// kernels above, launched behind them and gated on that flag, produce the
// results instead.  All of it stays stream-ordered: no host synchronisation.
// A workspace allocation that fails leaves the call to those kernels where
// they can take it (they need no workspace).  With scratch, the speculative
// workspace comes from it (nothing is allocated), and a call that needs more
// than scratch_bytes returns AS_E_LIMITS.
int run_shared_trace(KArgs& a, int W, int smax, hipStream_t stream, void* scratch, size_t scratch_bytes) {
  if (want_spec(a, smax)) {
    const bool fallback = run_trace_kernels(a, W, smax, stream, true) == AS_OK;
    void* ws = nullptr;
    const int32_t* gave_up = nullptr;
    int rc = run_spec(a, smax, stream, fallback, scratch, scratch_bytes, &ws, &gave_up);
    if (rc == kSpecScratchTooSmall) return AS_E_LIMITS;
    if (rc == AS_E_NOMEM && fallback) rc = AS_E_LIMITS;
    if (rc != AS_E_LIMITS) {
      if (rc != AS_OK || !fallback) return rc;
      a.gate = gave_up;
      const int rc2 = run_trace_kernels(a, W, smax, stream, false);
      a.gate = nullptr;
      const hipError_t ef = ws ? hipFreeAsync(ws, stream) : hipSuccess;
      if (rc2 != AS_OK) return rc2;
      if (ef != hipSuccess) return fail(AS_E_HIP, "workspace release failed: %s", hipGetErrorString(ef));
      return ok();
    }
  }
  return run_trace_kernels(a, W, smax, stream, false);
}

}  // namespace as_host

using namespace as_host;

extern "C" {

const char* as_last_error(void) { return g_err.c_str(); }

const char* as_version(void) { return "alpaserve_sim 0.1 gfx950"; }

}  // extern "C"

namespace as_host {
namespace {

// Workspace of as_simulate_placements_noalloc: one array per device, held
// until the process ends, shared by every call on that device.
static __device__ __align__(256) unsigned char scratch[AS_NOALLOC_SCRATCH_BYTES];

// Device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept; null with a message set when
// the lookup fails.  In host code the array's name is only a stand-in for
// the symbol, never a device address.
void* scratch_ptr() {
  static std::mutex mu;
  static void* ptrs[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    fail(AS_E_HIP, "no current HIP device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!ptrs[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      fail(AS_E_HIP, "scratch address on device %d: %s", dev, hipGetErrorString(e));
      return nullptr;
    }
    ptrs[dev] = p;
  }
  return ptrs[dev];
}

// Body of as_simulate_placements; with no_alloc, the speculative kernels'
// workspace comes from `scratch` and nothing is allocated.
int simulate_placements(const as_trace_t* trace, const as_models_t* models,
                        const as_placements_t* placements, const double* slo_scale, int32_t n_scales,
                        int64_t* out_served, double* out_attain, uint64_t* out_digest,
                        const int32_t* finish_jobs, int32_t n_finish, double* out_finish, void* stream,
                        bool no_alloc) {
  KArgs a;
  std::memset(&a, 0, sizeof a);
  if (!trace) return fail(AS_E_INVALID_ARG, "trace must not be NULL");
  if (trace->n < 0) return fail(AS_E_INVALID_ARG, "trace n=%lld < 0", (long long)trace->n);
  if (trace->n > 0 && (!trace->t || !trace->model))
    return fail(AS_E_INVALID_ARG, "trace arrays must not be NULL");
  int W = 1, smax = 1;
  int rc = check_common(models, placements, a, W, smax);
  if (rc != AS_OK) return rc;
  if (n_scales < 0) return fail(AS_E_INVALID_ARG, "n_scales=%d < 0", n_scales);
  const int64_t J = (int64_t)placements->n_placements * n_scales;
  if (J > 0x7FFFFFFFLL) return fail(AS_E_LIMITS, "placements x scales = %lld jobs > 2^31-1", (long long)J);
  if (J > 0 && (!slo_scale || !out_served))
    return fail(AS_E_INVALID_ARG, "slo_scale and out_served must not be NULL");
  rc = check_finish(finish_jobs, n_finish, out_finish, J, a);
  if (rc != AS_OK) return rc;
  if (J == 0) return ok();
  a.t = trace->t;
  a.model = trace->model;
  a.n = trace->n;
  a.slo_scale = slo_scale;
  a.K = n_scales;
  a.J = (int32_t)J;
  a.out_served = out_served;
  a.out_attain = out_attain;
  a.out_digest = out_digest;
  a.finish_stride = trace->n;
  if (!no_alloc) return run_shared_trace(a, W, smax, (hipStream_t)stream);
  void* ws = scratch_ptr();
  if (!ws) return AS_E_HIP;
  return run_shared_trace(a, W, smax, (hipStream_t)stream, ws, AS_NOALLOC_SCRATCH_BYTES);
}

}  // namespace
}  // namespace as_host

extern "C" {

int as_simulate_placements(const as_trace_t* trace, const as_models_t* models,
                           const as_placements_t* placements, const double* slo_scale,
                           int32_t n_scales, int64_t* out_served, double* out_attain,
                           uint64_t* out_digest, const int32_t* finish_jobs, int32_t n_finish,
                           double* out_finish, void* stream) {
  return simulate_placements(trace, models, placements, slo_scale, n_scales, out_served, out_attain,
                             out_digest, finish_jobs, n_finish, out_finish, stream, false);
}

int as_simulate_placements_noalloc(const as_trace_t* trace, const as_models_t* models,
                                   const as_placements_t* placements, const double* slo_scale,
                                   int32_t n_scales, int64_t* out_served, double* out_attain,
                                   uint64_t* out_digest, const int32_t* finish_jobs, int32_t n_finish,
                                   double* out_finish, void* stream) {
  return simulate_placements(trace, models, placements, slo_scale, n_scales, out_served, out_attain,
                             out_digest, finish_jobs, n_finish, out_finish, stream, true);
}

namespace as_dev {
namespace {

constexpr int kOrderMaxJobs = 4096;  // jobs the one-workgroup sort below takes

// Launch order of the one-job-per-wavefront kernel: the jobs sorted by
// segment length (longest first, lower index first on ties).  queue 0: one
// job per wavefront, the longest and the shortest alternating -- order[2i]
// the i-th longest, order[2i + 1] the i-th shortest -- so that the longest
// chains share their SIMDs with short ones.  queue 1: fewer wavefronts than
// jobs take the jobs in turn, longest first, from the slot counter
// order[J], which is set to 0 here.  One workgroup of 1024 threads,
// J <= 4096.
__global__ __launch_bounds__(1024) void seg_order(const KArgs a, int32_t* __restrict__ order, int queue) {
  __shared__ int64_t key[kOrderMaxJobs];
  __shared__ int32_t val[kOrderMaxJobs];
  const int J = (int)a.J;
  int P = 1;
  while (P < J) P <<= 1;
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    int64_t len = -1;  // padding sorts after every job
    if (i < J) {
      const as_job_t jb = a.jobs[i];
      len = 0;
      if (jb.placement >= 0 && jb.placement < a.P && jb.segment >= 0 && jb.segment < a.n_segments) {
        const int64_t total = a.seg_off[a.n_segments];
        int64_t b = a.seg_off[jb.segment], e = a.seg_off[jb.segment + 1];
        b = b < 0 ? 0 : (b > total ? total : b);
        e = e < b ? b : (e > total ? total : e);
        len = e - b;
      }
    }
    key[i] = len;
    val[i] = i;
  }
  __syncthreads();
  // bitonic sort: descending length, ascending index on ties
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += blockDim.x) {
        const int l = i ^ j;
        if (l > i) {
          const bool before = key[i] > key[l] || (key[i] == key[l] && val[i] < val[l]);  // i precedes l
          const bool desc = (i & k) == 0;
          if (desc != before) {
            const int64_t tk = key[i];
            key[i] = key[l];
            key[l] = tk;
            const int32_t tv = val[i];
            val[i] = val[l];
            val[l] = tv;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < J; i += blockDim.x) {
    const int h = i >> 1;
    order[i] = queue ? val[i] : (i & 1) == 0 ? val[h] : val[J - 1 - h];
  }
  if (queue && threadIdx.x == 0) order[J] = 0;
}

// Wavefronts per SIMD that take the sweep's jobs in turn.  Two: the longest
// job shares its SIMD with one other wavefront, which works through shorter
// jobs meanwhile (ALPASERVE_SEG_WAVES sets 1-4, for measurements).
int seg_waves_per_simd() {
  const char* e = getenv("ALPASERVE_SEG_WAVES");
  const int v = e ? atoi(e) : 2;
  return v < 1 ? 1 : (v > 4 ? 4 : v);
}

// Workgroups that take the jobs in turn: seg_waves_per_simd() per compute
// unit (ALPASERVE_SEG_BLOCKS sets the count, 1-4096, for the tests: a few
// workgroups then each work through many jobs).
int64_t seg_queue_blocks(int wps) {
  const char* e = getenv("ALPASERVE_SEG_BLOCKS");
  const int v = e ? atoi(e) : 0;
  if (v >= 1 && v <= 4096) return v;
  return (int64_t)wps * as_host::compute_units();
}

}  // namespace
}  // namespace as_dev

int as_simulate_jobs(const double* t, const int32_t* model, const int64_t* seg_offsets,
                     int32_t n_segments, const as_models_t* models,
                     const as_placements_t* placements, const as_job_t* jobs, int32_t n_jobs,
                     int64_t* out_served, double* out_attain, uint64_t* out_digest,
                     const int32_t* finish_jobs, int32_t n_finish, double* out_finish,
                     int64_t finish_stride, void* stream) {
  KArgs a;
  std::memset(&a, 0, sizeof a);
  if (n_segments < 0 || n_jobs < 0) return fail(AS_E_INVALID_ARG, "negative n_segments or n_jobs");
  int W = 1, smax = 1;
  int rc = check_common(models, placements, a, W, smax);
  if (rc != AS_OK) return rc;
  if (n_jobs > 0 && n_segments < 1)
    return fail(AS_E_INVALID_ARG, "n_segments must be >= 1 when there are jobs");
  if (n_jobs > 0 && (!t || !model || !seg_offsets || !jobs || !out_served))
    return fail(AS_E_INVALID_ARG, "t, model, seg_offsets, jobs and out_served must not be NULL");
  if (finish_stride < 0) return fail(AS_E_INVALID_ARG, "finish_stride < 0");
  rc = check_finish(finish_jobs, n_finish, out_finish, n_jobs, a);
  if (rc != AS_OK) return rc;
  if (n_jobs == 0) return ok();
  a.t = t;
  a.model = model;
  a.seg_off = seg_offsets;
  a.n_segments = n_segments;
  a.jobs = jobs;
  a.J = n_jobs;
  a.out_served = out_served;
  a.out_attain = out_attain;
  a.out_digest = out_digest;
  a.finish_stride = finish_stride;
  hipStream_t s = (hipStream_t)stream;
  // more than 32 groups: one job per wavefront with the shared-trace request
  // loop (the requests of a wavefront are one job's)
  const size_t lds_seg = as_dev::seg_lds_bytes(a.M, pow2ceil(a.C), smax);
  if (use_shared_path() && pow2ceil(a.G) == 64 && lds_seg <= shared_lds_limit()) {
    hipError_t e = hipSuccess;
    if (a.n_finish > 0 && finish_stride > 0) {
      const int64_t cells = (int64_t)a.n_finish * finish_stride;
      const int64_t blocks = std::min<int64_t>((cells + 255) / 256, 8192);
      hipLaunchKernelGGL(fill_seg_rows, dim3((unsigned)blocks), dim3(256), 0, s, a);
      if ((e = hipGetLastError()) != hipSuccess)
        return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    }
    // Jobs longest first.  With more jobs than seg_waves_per_simd()
    // wavefronts per SIMD, that many wavefronts take them in turn (each
    // compute unit holds that many workgroups of one wavefront per SIMD: the
    // LDS request leaves room for no more); otherwise one job per wavefront,
    // long and short chains interleaved.  Skipped, never an error, where the
    // jobs are too many for the sort or its array cannot be allocated.
    const int wps = as_dev::seg_waves_per_simd();
    const int64_t queue_blocks = as_dev::seg_queue_blocks(wps);
    int64_t blocks = (n_jobs + as_dev::kWaves - 1) / as_dev::kWaves;
    size_t lds = lds_seg;
    int32_t* order = nullptr;
    if (n_jobs >= 2 && n_jobs <= as_dev::kOrderMaxJobs &&
        pool_alloc(reinterpret_cast<void**>(&order), ((size_t)n_jobs + 1) * 4, s) == hipSuccess) {
      const bool queue = blocks > queue_blocks;
      hipLaunchKernelGGL(as_dev::seg_order, dim3(1), dim3(1024), 0, s, a, order, queue ? 1 : 0);
      if ((e = hipGetLastError()) != hipSuccess) {
        (void)hipFreeAsync(order, s);
        return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
      }
      a.order = order;
      if (queue) {
        a.next_slot = order + n_jobs;
        blocks = queue_blocks;
        const size_t per_cu = 160 * 1024;  // LDS of a compute unit
        const size_t cap = per_cu / (size_t)(wps + 1) + 1024;
        if (cap > lds && cap <= shared_lds_limit()) lds = cap;
      }
    } else {
      (void)hipGetLastError();
    }
    e = as_host::launch_seg64(smax, a, blocks, lds, s);
    const hipError_t ef = order ? hipFreeAsync(order, s) : hipSuccess;
    if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    if (ef != hipSuccess) return fail(AS_E_HIP, "order release failed: %s", hipGetErrorString(ef));
    return ok();
  }
  int GPL = 1;
  if (!choose_shape(a.G, n_jobs, true, a.M, a.C, smax, W, GPL))
    return fail(AS_E_LIMITS, "stage-latency tables (%d models x %d configs x %d stages) do not fit in LDS",
                a.M, a.C, smax);
  const size_t lds = lds_bytes(W, smax, true, a.M, a.C);
  hipError_t e = launch_lds_any(W, GPL, smax, true, a, lds, s);
  if (e != hipSuccess) return fail(AS_E_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return ok();
}

int as_validate(const as_trace_t* trace, const as_models_t* models,
                const as_placements_t* placements, const double* slo_scale, int32_t n_scales,
                void* stream) {
  KArgs a;
  std::memset(&a, 0, sizeof a);
  if (!trace) return fail(AS_E_INVALID_ARG, "trace must not be NULL");
  if (trace->n < 0) return fail(AS_E_INVALID_ARG, "trace n=%lld < 0", (long long)trace->n);
  if (trace->n > 0 && (!trace->t || !trace->model))
    return fail(AS_E_INVALID_ARG, "trace arrays must not be NULL");
  int W = 1, smax = 1;
  int rc = check_common(models, placements, a, W, smax);
  if (rc != AS_OK) return rc;
  if (n_scales < 0) return fail(AS_E_INVALID_ARG, "n_scales=%d < 0", n_scales);
  if (n_scales > 0 && !slo_scale) return fail(AS_E_INVALID_ARG, "slo_scale must not be NULL");
  hipStream_t s = (hipStream_t)stream;
  uint32_t* d_flags = nullptr;
  hipError_t e = hipMallocAsync((void**)&d_flags, sizeof(uint32_t), s);
  if (e != hipSuccess) return fail(AS_E_NOMEM, "hipMallocAsync: %s", hipGetErrorString(e));
  uint32_t flags = 0;
  e = hipMemsetAsync(d_flags, 0, sizeof(uint32_t), s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(validate_kernel, dim3(1024), dim3(256), 0, s, trace->t, trace->model,
                       trace->n, a.M, a.C, a.group_cfg, a.host_mask,
                       (int64_t)placements->n_placements, a.G, a.stage_lat, a.smax_in, a.d_single,
                       slo_scale, n_scales, a, d_flags);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpyAsync(&flags, d_flags, sizeof flags, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  hipError_t ef = hipFreeAsync(d_flags, s);
  if (e == hipSuccess) e = ef;
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(AS_E_HIP, "as_validate: %s", hipGetErrorString(e));
  for (int b = 0; b < 7; ++b)
    if (flags & (1u << b)) return fail(AS_E_INVALID_DATA, "%s", kValidateMsg[b]);
  return ok();
}

}  // extern "C"
