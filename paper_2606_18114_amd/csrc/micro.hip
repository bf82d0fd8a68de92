// Measured denominators for the rooflines (not part of the hot path; built
// into libtm_micro.so, separate from libtmamba.so).
//
//   tmm_mfma_loop: every wave of a full-occupancy grid (two 8-wave
//     workgroups per CU, so four waves per SIMD) runs `iters` rounds of
//     independent bf16 MFMAs on operands it loaded from `operands` (64 lanes
//     x 16 bfloat16: the lane's A then B values), so the matrix cores see the
//     caller's data, e.g. random values, which draw more power than zeros.
//     shape 32: four v_mfma_f32_32x32x16_bf16 per round, shape 16: eight
//     v_mfma_f32_16x16x32_bf16; either way 131072 flops per wave and round.
//   tmm_read_stream: a grid of two 512-thread workgroups per CU reads `bytes`
//     from `buf` in contiguous 16 KiB chunks, one chunk per wave at a time
//     (sixteen 1 KiB loads in flight per wave, 256 KiB per CU), and folds the
//     data into one word per thread (written to `out`) so the loads cannot
//     be dropped.  Of the access patterns tried (grid-stride 16-byte pieces,
//     4 KiB or 16 KiB per wave, 32 rows x 128 bytes at a 512-byte pitch) the
//     contiguous chunks were fastest.  `bytes` must be a multiple of 16 KiB.
//   tmm_decode_stream: the same stream, with every 16-byte piece of packed
//     ternary codes decoded into the FP4 operand nibbles (2q: 0100, 1100,
//     0000) the decode GEMV hands to the matrix cores: format 2 is the 2-bit
//     code format (64 codes per piece, one 64-bit shift and four ANDs per 32
//     codes), format 3 base-3 packing (five codes per byte, 80 per piece,
//     one LDS table read per byte giving its five nibbles, placed into the
//     nibble stream by shifts).  It measures what decoding costs per code
//     against the bytes a format saves.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 mbf16x8 __attribute__((ext_vector_type(8)));
typedef float mf32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t mu32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 512;

typedef float mf32x4 __attribute__((ext_vector_type(4)));

template <int SHAPE>
__global__ __launch_bounds__(kThreads) void mfma_loop_kernel(const uint16_t* __restrict__ operands,
                                                             int iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const mu32x4 va = *reinterpret_cast<const mu32x4*>(operands + 16 * lane);
  const mu32x4 vb = *reinterpret_cast<const mu32x4*>(operands + 16 * lane + 8);
  const mbf16x8 a = __builtin_bit_cast(mbf16x8, va);
  const mbf16x8 b = __builtin_bit_cast(mbf16x8, vb);
  float s = 0.f;
  if constexpr (SHAPE == 32) {
    mf32x16 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[j][i] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) s += acc[j][i];
  } else {
    mf32x4 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[j][i] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) s += acc[j][i];
  }
  out[blockIdx.x * kThreads + threadIdx.x] = s;
}

__global__ __launch_bounds__(kThreads) void read_stream_kernel(const mu32x4* __restrict__ buf,
                                                               int64_t chunks,
                                                               uint32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t nwaves = (int64_t)gridDim.x * (kThreads / 64);
  uint32_t acc = 0;
  for (int64_t ch = wave; ch < chunks; ch += nwaves) {  // chunk: 1024 pieces of 16 bytes
    const mu32x4* p = buf + ch * 1024 + lane;
    mu32x4 v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = p[64 * j];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc ^= v[j].x ^ v[j].w;
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

// keeps a decoded operand word alive (as the matrix-core operand would) at
// no instruction cost, so the decode cannot be folded away
__device__ __forceinline__ void sink(uint32_t v) { asm volatile("" ::"v"(v)); }

template <int FMT>
__global__ __launch_bounds__(kThreads) void decode_stream_kernel(const mu32x4* __restrict__ buf,
                                                                 int64_t chunks,
                                                                 uint32_t* __restrict__ out) {
  __shared__ uint32_t lut[256];  // base 3: byte -> its five codes' FP4 nibbles
  if constexpr (FMT == 3) {
    for (int b = threadIdx.x; b < 256; b += kThreads) {
      uint32_t t = 0, v = (uint32_t)b;
      for (int i = 0; i < 5; ++i) {
        const uint32_t c = v % 3u;  // code + 1
        v /= 3u;
        t |= (c == 2u ? 0x4u : c == 0u ? 0xCu : 0u) << (4 * i);
      }
      lut[b] = b < 243 ? t : 0u;
    }
    __syncthreads();
  }
  const int lane = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * kThreads + threadIdx.x) >> 6;
  const int64_t nwaves = (int64_t)gridDim.x * (kThreads / 64);
  uint32_t acc = 0;
  for (int64_t ch = wave; ch < chunks; ch += nwaves) {
    const mu32x4* p = buf + ch * 1024 + lane;
    mu32x4 v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = p[64 * j];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
      acc ^= w[0];
      if constexpr (FMT == 2) {
        constexpr uint32_t kNib = 0xCCCCCCCCu;
#pragma unroll
        for (int k = 0; k < 4; k += 2) {
          const uint64_t ww = ((uint64_t)w[k + 1] << 32) | w[k];
          const uint64_t sh = ww << 2;
          sink(w[k] & kNib);
          sink((uint32_t)sh & kNib);
          sink(w[k + 1] & kNib);
          sink((uint32_t)(sh >> 32) & kNib);
        }
      } else {
        uint32_t o[10] = {};
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const uint32_t t = lut[(w[b / 4] >> (8 * (b % 4))) & 0xFFu];
          const int pos = 5 * b, d = pos / 8, sh = 4 * (pos % 8);
          o[d] |= t << sh;
          if (sh + 20 > 32) o[d + 1] |= t >> (32 - sh);
        }
#pragma unroll
        for (int i = 0; i < 10; ++i) sink(o[i]);
      }
    }
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
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

// Threads of the grids below (2 workgroups of 512 per CU): the length of
// `out` in elements.
int tmm_grid_threads(void) { return 2 * cu_count() * kThreads; }

// operands: 1024 bfloat16 (device); shape: 32 or 16 (the MFMA);
// out: tmm_grid_threads() floats (device).
// Returns 0 or the HIP error code of the launch.
int tmm_mfma_loop(const uint16_t* operands, int iters, int shape, float* out, void* stream) {
  if (!operands || !out || iters < 1 || (shape != 32 && shape != 16))
    return (int)hipErrorInvalidValue;
  if (shape == 32)
    hipLaunchKernelGGL(mfma_loop_kernel<32>, dim3(2 * cu_count()), dim3(kThreads), 0,
                       (hipStream_t)stream, operands, iters, out);
  else
    hipLaunchKernelGGL(mfma_loop_kernel<16>, dim3(2 * cu_count()), dim3(kThreads), 0,
                       (hipStream_t)stream, operands, iters, out);
  return (int)hipGetLastError();
}

// buf: `bytes` of device memory, bytes % 16384 == 0, 16-byte aligned;
// out: tmm_grid_threads() words (device).
int tmm_read_stream(const void* buf, int64_t bytes, uint32_t* out, void* stream) {
  if (!buf || !out || bytes <= 0 || bytes % 16384 != 0 ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(read_stream_kernel, dim3(2 * cu_count()), dim3(kThreads), 0,
                     (hipStream_t)stream, reinterpret_cast<const mu32x4*>(buf), bytes / 16384,
                     out);
  return (int)hipGetLastError();
}

// The read stream with each piece decoded as packed ternary codes: format 2
// (2-bit codes) or 3 (base-3, five codes per byte).  Same contract as
// tmm_read_stream.
int tmm_decode_stream(const void* buf, int64_t bytes, int format, uint32_t* out, void* stream) {
  if (!buf || !out || bytes <= 0 || bytes % 16384 != 0 || (format != 2 && format != 3) ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0)
    return (int)hipErrorInvalidValue;
  const auto* b = reinterpret_cast<const mu32x4*>(buf);
  if (format == 2)
    hipLaunchKernelGGL(decode_stream_kernel<2>, dim3(2 * cu_count()), dim3(kThreads), 0,
                       (hipStream_t)stream, b, bytes / 16384, out);
  else
    hipLaunchKernelGGL(decode_stream_kernel<3>, dim3(2 * cu_count()), dim3(kThreads), 0,
                       (hipStream_t)stream, b, bytes / 16384, out);
  return (int)hipGetLastError();
}

}  // extern "C"
