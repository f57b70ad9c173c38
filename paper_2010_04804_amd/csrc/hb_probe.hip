// hb_probe.hip -- measurement aids for the benchmark, built as their own small
// library (libhb_probe.so) beside libhb.so and not part of the scoring path:
//  * the dense int8 matrix-core rate this device sustains, so that the GEMM
//    strategy's throughput can be stated against a measured peak as well as
//    the published one. Every wave keeps sixteen independent accumulators
//    busy with v_mfma_i32_16x16x64_i8 on register operands (2 * 16 * 16 * 64
//    = 32,768 integer operations per instruction);
//  * the rate at which a CU's LDS serves wave-wide reads of the shapes the
//    traversal walks issue (a lane's own word of a feature column, node
//    records at data-dependent slots of a tree), which bounds those walks.
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

// LDS reads: 16 waves per CU, eight independent reads in flight per wave
// (issued back to back, then one wait), each wave in its own 8 KiB of a
// 128 KiB array. Modes: 0 b32 at the lane's own word, 1 b32 at a hashed slot
// of 256 (a 1 KiB region), 2 b64 own, 3 b64 hashed of 256 (2 KiB), 4 u16 own,
// 5 b128 own, 6 b128 hashed of 64 (1 KiB), 7 alternately b64 hashed of 256
// and b32 own (a tree walk's node and feature reads).
__device__ __forceinline__ unsigned probe_hash(unsigned x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kLdsWords = 32768;  // 128 KiB

#define PROBE_READ8(OP, T)                                                                                      \
  T v0, v1, v2, v3, v4, v5, v6, v7;                                                                             \
  asm volatile(OP " %0, %8\n" OP " %1, %9\n" OP " %2, %10\n" OP " %3, %11\n" OP " %4, %12\n" OP " %5, %13\n" OP \
               " %6, %14\n" OP " %7, %15\ns_waitcnt lgkmcnt(0)"                                                 \
               : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3), "=v"(v4), "=v"(v5), "=v"(v6), "=v"(v7)                  \
               : "v"(addr[0]), "v"(addr[1]), "v"(addr[2]), "v"(addr[3]), "v"(addr[4]), "v"(addr[5]), "v"(addr[6]), \
                 "v"(addr[7]));

template <int M>
__global__ __launch_bounds__(1024) void lds_read_loop(int iters, unsigned *sink) {
  __shared__ __align__(16) unsigned lds[kLdsWords];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < kLdsWords; i += 1024) lds[i] = (unsigned)i;
  __syncthreads();
  constexpr int W = (M == 0 || M == 1) ? 4 : (M == 2 || M == 3) ? 8 : M == 4 ? 2 : 16;
  constexpr bool HASHED = M == 1 || M == 3 || M == 6;
  constexpr unsigned S = M == 6 ? 64 : 256;
  // largest byte offset: 15 * 8192 + 3 * 2048 + 8 * 255 + 8 = 131,072 (the array's end)
  unsigned addr[8];
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const unsigned h = probe_hash((unsigned)lane * 131u + (unsigned)g * 7919u + blockIdx.x);
    unsigned w = W, slot = HASHED ? h % S : (unsigned)lane;
    if (M == 7) {
      w = (g & 1) ? 4u : 8u;
      slot = (g & 1) ? (unsigned)lane : h % 256u;
    }
    addr[g] = (unsigned)(uintptr_t)lds + (unsigned)wave * 8192u + (unsigned)(g & 3) * 2048u + w * slot;
  }
  unsigned acc = 0;
  for (int it = 0; it < iters; ++it) {
    if constexpr (M == 0 || M == 1) {
      PROBE_READ8("ds_read_b32", unsigned)
      acc += v0 ^ v1 ^ v2 ^ v3 ^ v4 ^ v5 ^ v6 ^ v7;
    } else if constexpr (M == 2 || M == 3) {
      PROBE_READ8("ds_read_b64", unsigned long long)
      acc += (unsigned)(v0 ^ v1 ^ v2 ^ v3 ^ v4 ^ v5 ^ v6 ^ v7);
    } else if constexpr (M == 4) {
      PROBE_READ8("ds_read_u16", unsigned)
      acc += v0 ^ v1 ^ v2 ^ v3 ^ v4 ^ v5 ^ v6 ^ v7;
    } else if constexpr (M == 5 || M == 6) {
      PROBE_READ8("ds_read_b128", u32x4)
      acc += v0.x ^ v1.y ^ v2.z ^ v3.w ^ v4.x ^ v5.y ^ v6.z ^ v7.w;
    } else {
      unsigned long long a0, a2, a4, a6;
      unsigned b1, b3, b5, b7;
      asm volatile(
          "ds_read_b64 %0, %8\nds_read_b32 %1, %9\nds_read_b64 %2, %10\nds_read_b32 %3, %11\nds_read_b64 %4, %12\n"
          "ds_read_b32 %5, %13\nds_read_b64 %6, %14\nds_read_b32 %7, %15\ns_waitcnt lgkmcnt(0)"
          : "=v"(a0), "=v"(b1), "=v"(a2), "=v"(b3), "=v"(a4), "=v"(b5), "=v"(a6), "=v"(b7)
          : "v"(addr[0]), "v"(addr[1]), "v"(addr[2]), "v"(addr[3]), "v"(addr[4]), "v"(addr[5]), "v"(addr[6]),
            "v"(addr[7]));
      acc += (unsigned)(a0 ^ a2 ^ a4 ^ a6) ^ b1 ^ b3 ^ b5 ^ b7;
    }
  }
  sink[blockIdx.x * 1024 + tid] = acc;  // keeps the reads live
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

// LDS read rate on `device` for read shape `mode` (0..7, see lds_read_loop):
// *ns_per_read receives nanoseconds per wave-wide read instruction per CU
// (one 1024-thread workgroup per CU). Returns 0, or a HIP error code.
__attribute__((visibility("default"))) int hb_probe_lds_read(int device, int mode, double *ns_per_read) {
  if (!ns_per_read || mode < 0 || mode > 7) return (int)hipErrorInvalidValue;
  hipError_t e = hipSetDevice(device);
  int cus = 0;
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess) return (int)e;
  void (*fn)(int, unsigned *) = nullptr;
  switch (mode) {
    case 0: fn = lds_read_loop<0>; break;
    case 1: fn = lds_read_loop<1>; break;
    case 2: fn = lds_read_loop<2>; break;
    case 3: fn = lds_read_loop<3>; break;
    case 4: fn = lds_read_loop<4>; break;
    case 5: fn = lds_read_loop<5>; break;
    case 6: fn = lds_read_loop<6>; break;
    default: fn = lds_read_loop<7>; break;
  }
  const int iters = 4000;
  unsigned *sink = nullptr;
  hipEvent_t t0 = nullptr, t1 = nullptr;
  e = hipMalloc(&sink, (size_t)cus * 1024 * sizeof(unsigned));
  if (e == hipSuccess) e = hipEventCreate(&t0);
  if (e == hipSuccess) e = hipEventCreate(&t1);
  float ms = 0.0f;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(fn, dim3(cus), dim3(1024), 0, nullptr, 64, sink);  // warm-up
    (void)hipEventRecord(t0, nullptr);
    hipLaunchKernelGGL(fn, dim3(cus), dim3(1024), 0, nullptr, iters, sink);
    (void)hipEventRecord(t1, nullptr);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipEventSynchronize(t1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, t0, t1);
  }
  if (t0) (void)hipEventDestroy(t0);
  if (t1) (void)hipEventDestroy(t1);
  if (sink) (void)hipFree(sink);
  if (e != hipSuccess) return (int)e;
  *ns_per_read = (double)ms * 1e6 / (16.0 * iters * 8.0);
  return 0;
}

}  // extern "C"
