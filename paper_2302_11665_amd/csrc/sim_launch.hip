// Kernel launchers for one lanes-per-job width W = AS_W (see sim_launch.hpp).
#include <hip/hip_runtime.h>

#include "sim_kernel.hpp"
#include "sim_launch.hpp"
#include "sim_shared.hpp"

#ifndef AS_W
#error "compile with -DAS_W=<lanes per job>"
#endif

namespace as_host {
namespace {

template <int W, int GPL, int SMAX, bool SEG>
hipError_t lds_t(const KArgs& a, size_t lds, hipStream_t s) {
  if constexpr (W * GPL > 64) {
    return hipErrorInvalidValue;
  } else {
    constexpr int slots = (64 / W) * as_dev::kWaves;
    const int grid = (a.J + slots - 1) / slots;
    hipLaunchKernelGGL((as_dev::sim_kernel<W, GPL, SMAX, SEG>), dim3(grid), dim3(as_dev::kThreads), lds,
                       s, a);
    return hipGetLastError();
  }
}

template <int W, int GPL, bool SEG>
hipError_t lds_s(int smax, const KArgs& a, size_t lds, hipStream_t s) {
  switch (smax) {
    case 1: return lds_t<W, GPL, 1, SEG>(a, lds, s);
    case 2: return lds_t<W, GPL, 2, SEG>(a, lds, s);
    case 4: return lds_t<W, GPL, 4, SEG>(a, lds, s);
    default: return lds_t<W, GPL, 8, SEG>(a, lds, s);
  }
}

template <int W, int SMAX>
hipError_t shared_t(bool usig, bool stats, const KArgs& a, size_t lds, hipStream_t s) {
  constexpr int slots = (64 / W) * as_dev::kWaves;
  const int grid = (a.J + slots - 1) / slots;
  if (stats)
    hipLaunchKernelGGL((as_dev::shared_kernel<W, SMAX, true, true>), dim3(grid), dim3(as_dev::kThreads),
                       lds, s, a);
  else if (usig)
    hipLaunchKernelGGL((as_dev::shared_kernel<W, SMAX, true>), dim3(grid), dim3(as_dev::kThreads),
                       lds, s, a);
  else
    hipLaunchKernelGGL((as_dev::shared_kernel<W, SMAX, false>), dim3(grid), dim3(as_dev::kThreads),
                       lds, s, a);
  return hipGetLastError();
}

}  // namespace

template <int W>
hipError_t launch_lds(int gpl, int smax, bool seg, const KArgs& a, size_t lds, hipStream_t s) {
  switch (gpl) {
    case 1: return seg ? lds_s<W, 1, true>(smax, a, lds, s) : lds_s<W, 1, false>(smax, a, lds, s);
    case 2: return seg ? lds_s<W, 2, true>(smax, a, lds, s) : lds_s<W, 2, false>(smax, a, lds, s);
    default: return seg ? lds_s<W, 4, true>(smax, a, lds, s) : lds_s<W, 4, false>(smax, a, lds, s);
  }
}

template <int W>
hipError_t launch_shared(int smax, bool usig, bool stats, const KArgs& a, size_t lds, hipStream_t s) {
  switch (smax) {
    case 1: return shared_t<W, 1>(usig, stats, a, lds, s);
    case 2: return shared_t<W, 2>(usig, stats, a, lds, s);
    case 4: return shared_t<W, 4>(usig, stats, a, lds, s);
    default: return shared_t<W, 8>(usig, stats, a, lds, s);
  }
}

#if AS_W == 64
hipError_t launch_seg64(int smax, const KArgs& a, int64_t blocks, size_t lds, hipStream_t s) {
  const unsigned grid = (unsigned)blocks;
  switch (smax) {
    case 1:
      hipLaunchKernelGGL((as_dev::seg_kernel<1>), dim3(grid), dim3(as_dev::kThreads), lds, s, a);
      break;
    case 2:
      hipLaunchKernelGGL((as_dev::seg_kernel<2>), dim3(grid), dim3(as_dev::kThreads), lds, s, a);
      break;
    case 4:
      hipLaunchKernelGGL((as_dev::seg_kernel<4>), dim3(grid), dim3(as_dev::kThreads), lds, s, a);
      break;
    default:
      hipLaunchKernelGGL((as_dev::seg_kernel<8>), dim3(grid), dim3(as_dev::kThreads), lds, s, a);
      break;
  }
  return hipGetLastError();
}
#endif

template hipError_t launch_lds<AS_W>(int, int, bool, const KArgs&, size_t, hipStream_t);
template hipError_t launch_shared<AS_W>(int, bool, bool, const KArgs&, size_t, hipStream_t);

}  // namespace as_host
