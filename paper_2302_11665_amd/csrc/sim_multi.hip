// Multi-shape launches of the shared-trace kernel: a search step scores the
// jobs of several kernel shapes (lanes per job, padded stages) at once.  Run
// as separate launches on separate streams, they queue behind each other
// whenever the streams share a hardware queue, and a step then costs several
// trace passes of latency.  Here one dispatch carries them all: each block
// finds its shape segment from a table in the kernel arguments and runs that
// shape's instantiation of the shared-trace body.  The arguments common to
// all segments are read from device memory (a by-value copy of them would be
// copied to scratch in a kernel this large).
#include <hip/hip_runtime.h>

#include "sim_kernel.hpp"
#include "sim_launch.hpp"
#include "sim_shared.hpp"

namespace as_dev {
namespace {

template <bool USIG, bool STATS, int WL>
__device__ __forceinline__ void multi_w(const KArgs& a, const JobSet& v, int64_t blk, int sl) {
  switch (sl) {
    case 0: shared_body<1 << WL, 1, USIG, STATS, false>(a, v, blk); break;
    case 1: shared_body<1 << WL, 2, USIG, STATS, false>(a, v, blk); break;
    case 2: shared_body<1 << WL, 4, USIG, STATS, false>(a, v, blk); break;
    default: shared_body<1 << WL, 8, USIG, STATS, false>(a, v, blk); break;
  }
}

template <bool USIG, bool STATS>
__global__ __launch_bounds__(kThreads) void shared_multi(const KArgs* __restrict__ ap, const MultiSegs ms) {
  const KArgs& a = *ap;
  // this block's segment, with static indices only (the table stays in the
  // kernel arguments)
  int wl = ms.s[0].wl, sl = ms.s[0].sl;
  int64_t b0 = ms.s[0].block0;
  JobSet v = ms.s[0].v;
  const int64_t bx = blockIdx.x;
#pragma unroll
  for (int k = 1; k < kMaxShapeSegs; ++k) {
    if (k < ms.n && bx >= ms.s[k].block0) {
      wl = ms.s[k].wl;
      sl = ms.s[k].sl;
      b0 = ms.s[k].block0;
      v = ms.s[k].v;
    }
  }
  const int64_t blk = bx - b0;
  switch (wl) {
    case 0: multi_w<USIG, STATS, 0>(a, v, blk, sl); break;
    case 1: multi_w<USIG, STATS, 1>(a, v, blk, sl); break;
    case 2: multi_w<USIG, STATS, 2>(a, v, blk, sl); break;
    case 3: multi_w<USIG, STATS, 3>(a, v, blk, sl); break;
    case 4: multi_w<USIG, STATS, 4>(a, v, blk, sl); break;
    case 5: multi_w<USIG, STATS, 5>(a, v, blk, sl); break;
    default: multi_w<USIG, STATS, 6>(a, v, blk, sl); break;
  }
}

}  // namespace
}  // namespace as_dev

namespace as_host {

hipError_t launch_shared_multi(bool stats, const KArgs* a_dev, const as_dev::MultiSegs& ms, int64_t blocks,
                               size_t lds, hipStream_t s) {
  if (stats)
    hipLaunchKernelGGL((as_dev::shared_multi<true, true>), dim3((unsigned)blocks), dim3(as_dev::kThreads), lds, s,
                       a_dev, ms);
  else
    hipLaunchKernelGGL((as_dev::shared_multi<true, false>), dim3((unsigned)blocks), dim3(as_dev::kThreads), lds, s,
                       a_dev, ms);
  return hipGetLastError();
}

}  // namespace as_host
