// Kernel launchers, one translation unit per lanes-per-job width W (the
// build compiles sim_launch.hip once per W with -DAS_W=W and links them).
#pragma once

#include <hip/hip_runtime.h>

#include "sim_kernel.hpp"
#include "sim_shared.hpp"

namespace as_host {

using as_dev::KArgs;

// General LDS-staged kernel: GPL groups per lane, SEG = per-job segments.
template <int W>
hipError_t launch_lds(int gpl, int smax, bool seg, const KArgs& a, size_t lds, hipStream_t s);

// Shared-trace kernel: one group per lane, USIG = one SLO scale for all jobs;
// stats (one scale only): per-model served counts and per-group busy time.
template <int W>
hipError_t launch_shared(int smax, bool usig, bool stats, const KArgs& a, size_t lds, hipStream_t s);

// Several shapes of the shared-trace kernel (one SLO scale, no per-request
// rows) in one dispatch over `blocks` workgroups (sim_multi.hip); a_dev: the
// common arguments in device memory, unchanged until the launch has run.
hipError_t launch_shared_multi(bool stats, const KArgs* a_dev, const as_dev::MultiSegs& ms, int64_t blocks,
                               size_t lds, hipStream_t s);

// Segmented jobs with up to 64 groups, one job per wavefront at a time
// (built in the 64-lane unit): blocks workgroups of kWaves wavefronts, each
// wavefront running slot blockIdx * kWaves + w, or taking slots in turn
// from a.next_slot when that is set.
hipError_t launch_seg64(int smax, const KArgs& a, int64_t blocks, size_t lds, hipStream_t s);

#define AS_DECLARE_W(W)                                                                       \
  extern template hipError_t launch_lds<W>(int, int, bool, const KArgs&, size_t, hipStream_t); \
  extern template hipError_t launch_shared<W>(int, bool, bool, const KArgs&, size_t, hipStream_t);
AS_DECLARE_W(1)
AS_DECLARE_W(2)
AS_DECLARE_W(4)
AS_DECLARE_W(8)
AS_DECLARE_W(16)
AS_DECLARE_W(32)
AS_DECLARE_W(64)
#undef AS_DECLARE_W

}  // namespace as_host
