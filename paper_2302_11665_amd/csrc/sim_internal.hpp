// Host-side helpers of the C-ABI shared by its translation units (checks,
// error reporting, the shared-trace launch).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alpaserve_sim.h"
#include "sim_kernel.hpp"
#include "sim_shared.hpp"

namespace as_host {

using as_dev::KArgs;

// Record a message for as_last_error() and return code.
int fail(int code, const char* fmt, ...);
// Clear the message and return AS_OK.
int ok();
int pow2ceil(int x);
// LDS a workgroup may use on the current device (160 KiB on gfx950).
size_t shared_lds_limit();
// Compute units of the current device (cached per device).
int compute_units();
// Stream-ordered device allocation from the library's private memory pool
// (one per device, memory kept for reuse between calls); release with
// hipFreeAsync on a stream ordered after the last use.
hipError_t pool_alloc(void** p, size_t bytes, hipStream_t s);
// Checks shared by the simulate entry points; fill the model and placement
// part of a (placement arrays may be set later by the caller) and return the
// group count in W and the padded stage count in smax.
int check_common(const as_models_t* models, const as_placements_t* plc, KArgs& a, int& W, int& smax);
// Launch the batched simulation of a shared trace; a is complete except for
// the kernel shape, W is the group count on entry.  With scratch (device
// memory of scratch_bytes), the speculative kernels take their workspace
// from it and nothing is allocated; a call that would need more returns
// AS_E_LIMITS without launching.
int run_shared_trace(KArgs& a, int W, int smax, hipStream_t stream, void* scratch = nullptr,
                     size_t scratch_bytes = 0);
// Statistics launch of the shared-trace kernel (one SLO scale, no per-request
// output rows); returns AS_E_LIMITS without launching when that kernel cannot
// take the call (several scales, output rows, tables beyond the LDS).
int run_shared_stats(KArgs& a, int smax, hipStream_t stream);

// Shared-trace simulation on the segment-speculative kernels (one lane per
// job, the trace cut into segments simulated at once and reconciled);
// AS_E_LIMITS without launching when a wavefront's state does not fit in LDS
// or the segments would not pay.  With can_give_up, a reconciliation re-run
// that has not met the old results after a bounded number of requests stops
// the pipeline and sets *gave_up (device memory) to 1, else it stays 0: the
// caller then launches other kernels gated on it, which produce all results,
// and releases *workspace (stream-ordered, hipFreeAsync) after them.  Without
// it the workspace is released here and *gave_up is null.
// With caller_ws the workspace is carved from that device memory
// (caller_ws_bytes long) instead of being allocated, *workspace stays null,
// and a call that needs more returns kSpecScratchTooSmall (message set,
// nothing launched).
int run_spec(KArgs& a, int smax, hipStream_t stream, bool can_give_up, void* caller_ws,
             size_t caller_ws_bytes, void** workspace, const int32_t** gave_up);
// run_spec's return when a caller-given workspace is too small (internal).
constexpr int kSpecScratchTooSmall = -100;
// Whether a shared-trace call takes the segment-speculative kernels.
bool want_spec(const KArgs& a, int smax);
// Whether they would take it once wanted (sizes, LDS, segments that pay);
// nothing is launched.
bool spec_takes(const KArgs& a, int smax);

// One shape of a multi-shape shared-trace launch: lanes per job W (a power
// of two >= the group stride v.G), padded stages smax, and its jobs.
struct ShapeJobs {
  int W, smax;
  as_dev::JobSet v;
};
// The jobs of up to 16 shapes (one SLO scale, no per-request rows) in one
// dispatch, every job exactly as a launch of its own shape would simulate it
// (stats: the statistics outputs too).  Returns AS_E_LIMITS without
// launching when the jobs are too many for a multi-shape dispatch to pay
// (more than 2048 workgroups) or some shape would not take the shared-trace
// kernel as a launch of its own (the speculative kernels, LDS, the path
// switched off); the caller then launches the shapes one by one.
// dev_args: device memory of sizeof(KArgs) bytes for the common arguments,
// not used by other work until these launches have run.
int run_shared_multi(const KArgs& a, void* dev_args, const ShapeJobs* sh, int n, bool stats, hipStream_t stream);
// Whether ALPASERVE_PATH=spec forces them (even with a single segment).
bool spec_forced();

}  // namespace as_host
