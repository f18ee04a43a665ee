// Peak probes for gfx950: the two ceilings the simulator's roofline figures
// are quoted against, measured on the machine at hand.
//
//   as_probe_valu_f64  fp64 vector lane-operations per second, issued as the
//                      simulator issues them: v_max_f64 and v_add_f64 (no FMA),
//                      eight independent chains per lane, enough wavefronts to
//                      fill every SIMD several times over.
//   as_probe_hbm_read  bytes per second read from device memory: a buffer
//                      far larger than the caches, read once with 16-byte
//                      loads by a grid-stride loop.
//
// Measurement helpers only (bench.py calls them); they allocate their own
// device buffers and synchronise.  Return 0 on success, -1 on a HIP error.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ double probe_max(double a, double b) {
  double r;
  asm volatile("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

constexpr int kChains = 8;

__global__ __launch_bounds__(256) void valu_f64_kernel(double* out, int iters, double x, double y) {
  const int gid = blockIdx.x * blockDim.x + threadIdx.x;
  double acc[kChains];
#pragma unroll
  for (int k = 0; k < kChains; ++k) acc[k] = (double)gid * 1e-12 + k;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < kChains; ++k) acc[k] = probe_max(acc[k], x) + y;
  }
  double s = 0.0;
#pragma unroll
  for (int k = 0; k < kChains; ++k) s += acc[k];
  out[gid] = s;
}

// Four independent 16-byte loads in flight per lane and step, then the tail.
__global__ __launch_bounds__(256) void hbm_read_kernel(const uint4* in, size_t n, uint32_t* out) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  uint32_t x = 0;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const uint4 v0 = in[i], v1 = in[i + stride], v2 = in[i + 2 * stride], v3 = in[i + 3 * stride];
    x ^= v0.x ^ v0.y ^ v0.z ^ v0.w ^ v1.x ^ v1.y ^ v1.z ^ v1.w;
    x ^= v2.x ^ v2.y ^ v2.z ^ v2.w ^ v3.x ^ v3.y ^ v3.z ^ v3.w;
  }
  for (; i < n; i += stride) {
    const uint4 v = in[i];
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

int elapsed_ms(hipEvent_t a, hipEvent_t b, float* ms) {
  return hipEventElapsedTime(ms, a, b) == hipSuccess ? 0 : -1;
}

}  // namespace

// lane_ops: fp64 lane-operations per second (two per chain step: max and add);
// blocks of 256 threads; the best of `reps` timed launches after one warm-up.
extern "C" int as_probe_valu_f64(int blocks, int iters, int reps, double* lane_ops) {
  if (blocks <= 0 || iters <= 0 || reps <= 0 || !lane_ops) return -1;
  double* out = nullptr;
  if (hipMalloc(reinterpret_cast<void**>(&out), (size_t)blocks * 256 * sizeof(double)) != hipSuccess) return -1;
  hipEvent_t e0, e1;
  hipEventCreate(&e0);
  hipEventCreate(&e1);
  int rc = 0;
  float best = 0.0f;
  for (int r = 0; r <= reps && rc == 0; ++r) {
    hipEventRecord(e0, 0);
    hipLaunchKernelGGL(valu_f64_kernel, dim3(blocks), dim3(256), 0, 0, out, iters, 0.5, 1e-9);
    hipEventRecord(e1, 0);
    if (hipEventSynchronize(e1) != hipSuccess) rc = -1;
    float ms = 0.0f;
    if (rc == 0) rc = elapsed_ms(e0, e1, &ms);
    if (r > 0 && (best == 0.0f || ms < best)) best = ms;
  }
  if (hipGetLastError() != hipSuccess) rc = -1;
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  hipFree(out);
  if (rc == 0) *lane_ops = (double)blocks * 256.0 * iters * kChains * 2.0 / (best * 1e-3);
  return rc;
}

// bytes_per_s: device-memory read rate over a buffer of `bytes` (rounded
// down to 16 bytes); the best of `reps` timed launches after one warm-up.
extern "C" int as_probe_hbm_read(size_t bytes, int reps, double* bytes_per_s) {
  if (bytes < 16 || reps <= 0 || !bytes_per_s) return -1;
  const size_t n = bytes / 16;
  int dev = 0, cus = 256;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const int blocks = cus * 16;
  uint4* in = nullptr;
  uint32_t* out = nullptr;
  if (hipMalloc(reinterpret_cast<void**>(&in), n * 16) != hipSuccess) return -1;
  if (hipMalloc(reinterpret_cast<void**>(&out), (size_t)blocks * 256 * 4) != hipSuccess) {
    hipFree(in);
    return -1;
  }
  hipMemset(in, 1, n * 16);
  hipEvent_t e0, e1;
  hipEventCreate(&e0);
  hipEventCreate(&e1);
  int rc = hipDeviceSynchronize() == hipSuccess ? 0 : -1;
  float best = 0.0f;
  for (int r = 0; r <= reps && rc == 0; ++r) {
    hipEventRecord(e0, 0);
    hipLaunchKernelGGL(hbm_read_kernel, dim3(blocks), dim3(256), 0, 0, in, n, out);
    hipEventRecord(e1, 0);
    if (hipEventSynchronize(e1) != hipSuccess) rc = -1;
    float ms = 0.0f;
    if (rc == 0) rc = elapsed_ms(e0, e1, &ms);
    if (r > 0 && (best == 0.0f || ms < best)) best = ms;
  }
  if (hipGetLastError() != hipSuccess) rc = -1;
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  hipFree(in);
  hipFree(out);
  if (rc == 0) *bytes_per_s = (double)n * 16.0 / (best * 1e-3);
  return rc;
}
