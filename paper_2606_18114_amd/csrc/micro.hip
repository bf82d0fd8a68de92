// Measured denominators for the rooflines (not part of the hot path; built
// into libtm_micro.so, separate from libtmamba.so).
//
//   tmm_mfma_loop: every wave of a full-occupancy grid (two 8-wave
//     workgroups per CU, so four waves per SIMD) runs `iters` rounds of four
//     independent v_mfma_f32_32x32x16_bf16 on operands it loaded from
//     `operands` (64 lanes x 16 bfloat16: the lane's A then B values), so the
//     matrix cores see the caller's data, e.g. random values, which draw more
//     power than zeros.  flops = 2 * 32 * 32 * 16 * 4 * iters * waves.
//   tmm_read_stream: a grid of four 512-thread workgroups per CU (the most
//     waves a CU holds) reads `bytes` from `buf` in 16-byte pieces, four
//     loads in flight per thread (128 KiB per CU), and folds them into one
//     word per thread (written to `out`) so the loads cannot be dropped.
//     `bytes` must be a multiple of 64 * tmm_grid_threads().
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 mbf16x8 __attribute__((ext_vector_type(8)));
typedef float mf32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t mu32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;

__global__ __launch_bounds__(kThreads) void mfma_loop_kernel(const uint16_t* __restrict__ operands,
                                                             int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  mbf16x8 a, b;
  const mu32x4 va = *reinterpret_cast<const mu32x4*>(operands + 16 * lane);
  const mu32x4 vb = *reinterpret_cast<const mu32x4*>(operands + 16 * lane + 8);
  a = __builtin_bit_cast(mbf16x8, va);
  b = __builtin_bit_cast(mbf16x8, vb);
  mf32x16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[j][i];
  out[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void read_stream_kernel(const mu32x4* __restrict__ buf,
                                                               int64_t pieces,
                                                               uint32_t* __restrict__ out) {
  const int64_t nthreads = (int64_t)gridDim.x * kThreads;
  const int64_t tid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  uint32_t acc = 0;
  for (int64_t i = tid; i < pieces; i += 4 * nthreads) {
    const mu32x4 v0 = buf[i];
    const mu32x4 v1 = buf[i + nthreads];
    const mu32x4 v2 = buf[i + 2 * nthreads];
    const mu32x4 v3 = buf[i + 3 * nthreads];
    acc ^= (v0.x ^ v1.y) ^ (v2.z ^ v3.w);
  }
  out[tid] = acc;
}

int cu_count() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
    return 256;
  return v;
}

}  // namespace

extern "C" {

// Threads of the largest grid below (4 workgroups of 512 per CU): the length
// of `out` in elements.
int tmm_grid_threads(void) { return 4 * cu_count() * kThreads; }

// operands: 1024 bfloat16 (device); out: tmm_grid_threads() floats (device;
// the first half is written).
// Returns 0 or the HIP error code of the launch.
int tmm_mfma_loop(const uint16_t* operands, int iters, float* out, void* stream) {
  if (!operands || !out || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(2 * cu_count()), dim3(kThreads), 0,
                     (hipStream_t)stream, operands, iters, out);
  return (int)hipGetLastError();
}

// buf: `bytes` of device memory, bytes % (64 * tmm_grid_threads()) == 0;
// out: tmm_grid_threads() words (device).
int tmm_read_stream(const void* buf, int64_t bytes, uint32_t* out, void* stream) {
  const int64_t threads = tmm_grid_threads();
  if (!buf || !out || bytes <= 0 || bytes % (64 * threads) != 0 ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(read_stream_kernel, dim3(4 * cu_count()), dim3(kThreads), 0,
                     (hipStream_t)stream, reinterpret_cast<const mu32x4*>(buf), bytes / 16, out);
  return (int)hipGetLastError();
}

}  // extern "C"
