// hb_probe.hip -- a measurement aid for the benchmark, built as its own small
// library (libhb_probe.so) beside libhb.so and not part of the scoring path:
// the dense int8 matrix-core rate this device sustains, so that the GEMM
// strategy's throughput can be stated against a measured peak as well as
// the published one. Every wave keeps sixteen independent accumulators busy
// with v_mfma_i32_16x16x64_i8 on register operands (2 * 16 * 16 * 64 = 32,768
// integer operations per instruction).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kChains = 16;
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void mfma_i8_loop(int iters, int *sink) {
  const int lane = threadIdx.x & 63;
  v4i a = {lane, lane + 1, lane + 2, lane + 3};
  v4i b = {3 * lane, lane ^ 5, lane + 7, 11};
  v4i acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = v4i{c, 0, 0, 0};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[c], 0, 0, 0);
  }
  int s = 0;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  sink[blockIdx.x * kThreads + threadIdx.x] = s;  // keeps the products live
}

}  // namespace

extern "C" {

// Measures the sustained rate on `device`: *ops_per_s receives integer
// operations per second. Returns 0, or a HIP error code (the probe allocates
// a small result buffer and two events of its own).
__attribute__((visibility("default"))) int hb_probe_mfma_i8(int device, double *ops_per_s) {
  if (!ops_per_s) return (int)hipErrorInvalidValue;
  hipError_t e = hipSetDevice(device);
  int cus = 0;
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) return (int)e;
  const int blocks = cus * 8;  // eight waves per SIMD: eight workgroups of four waves per CU
  const int iters = 4096;
  int *sink = nullptr;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  e = hipMalloc(&sink, (size_t)blocks * kThreads * sizeof(int));
  if (e == hipSuccess) e = hipEventCreate(&t0);
  if (e == hipSuccess) e = hipEventCreate(&t1);
  float ms = 0.0f;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(mfma_i8_loop, dim3(blocks), dim3(kThreads), 0, nullptr, 64, sink);  // warm-up
    (void)hipEventRecord(t0, nullptr);
    hipLaunchKernelGGL(mfma_i8_loop, dim3(blocks), dim3(kThreads), 0, nullptr, iters, sink);
    (void)hipEventRecord(t1, nullptr);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipEventSynchronize(t1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, t0, t1);
  }
  if (t0) (void)hipEventDestroy(t0);
  if (t1) (void)hipEventDestroy(t1);
  if (sink) (void)hipFree(sink);
  if (e != hipSuccess) return (int)e;
  const double ops = (double)blocks * (kThreads / 64) * iters * kChains * 2.0 * 16 * 16 * 64;
  *ops_per_s = ops / (ms * 1e-3);
  return 0;
}

}  // extern "C"
