// Gradient of a per-group magnitude that multiplies the ternary codes:
//   out[n, j] = sum_{i < g} q[n, j g + i] * dW[n, j g + i]
// (the appendix's decoupled quantization, What = alpha_g * q, and the
// magnitude path of a learnable scale, Sec. 4), where dW is the gradient with
// respect to the dequantized weights (dY^T X, the straight-through dW).
//
// HBM bound: one pass over dW (4 bytes per weight) and the packed codes
// (1/4 byte).  A persistent grid walks 1024-weight units per wave with four
// coalesced 1 KiB loads of dW; each lane holds 4 consecutive weights of a
// load and reads the code word holding their codes (the four lanes of a word
// read it together).  Products are summed in float64 (exact for the 4 terms
// of a lane, then a butterfly over the g / 4 lanes of a group, two loads for
// g = 512) and rounded to float32 once.
#include "common.hpp"

namespace tmk {

constexpr int kGcdUnit = 1024;
constexpr int kGcdWaves = 16;

template <int G>
__global__ __launch_bounds__(64 * kGcdWaves) void group_code_dot_kernel(
    const uint32_t* __restrict__ codes, const float* __restrict__ dW, int64_t total,
    float* __restrict__ out) {
  constexpr int L = G / 4 < 64 ? G / 4 : 64;  // lanes holding one group within a load
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t nunits = (total + kGcdUnit - 1) / kGcdUnit;
  for (int64_t u = (int64_t)blockIdx.x * kGcdWaves + wave; u < nunits;
       u += (int64_t)gridDim.x * kGcdWaves) {
    const int64_t base = u * kGcdUnit;
    double ps[4];
    bool ok[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t off = base + 256 * i + 4 * lane;
      ok[i] = off < total;
      u32x4 v = {0u, 0u, 0u, 0u};
      uint32_t w = 0u;
      if (ok[i]) {
        v = ld16(dW + off);
        w = codes[off / 16];
      }
      const uint32_t dv[4] = {v.x, v.y, v.z, v.w};
      double t = 0.0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int e = 4 * (lane & 3) + j;  // element within its 16-code word
        const uint32_t c = (w >> (2 * (e / 2) + 16 * (e % 2))) & 3u;
        // 01 -> +dW, 11 -> -dW, 00 (and the unused 10) -> 0
        const float f = __uint_as_float(dv[j] ^ ((c >> 1) << 31));
        t += (c & 1u) ? (double)f : 0.0;
      }
      ps[i] = t;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) ps[i] = group_sum_f64<L>(ps[i]);
    if constexpr (G == 512) {  // a group spans two loads
      ps[0] += ps[1];
      ps[2] += ps[3];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t off = base + 256 * i + 4 * lane;
      if (ok[i] && (lane % L) == 0 && (G != 512 || (i & 1) == 0)) out[off / G] = (float)ps[i];
    }
  }
}

hipError_t launch_group_code_dot(const uint8_t* codes, const float* dW, int64_t N, int64_t K,
                                 int g, float* out, hipStream_t stream) {
  const int64_t total = N * K;
  int64_t blocks = (total / kGcdUnit + kGcdWaves) / kGcdWaves;
  if (blocks > 512) blocks = 512;
  const dim3 grid((unsigned)blocks), block(64 * kGcdWaves);
  auto* cw = reinterpret_cast<const uint32_t*>(codes);
  switch (g) {
    case 32:  hipLaunchKernelGGL(group_code_dot_kernel<32>, grid, block, 0, stream, cw, dW, total, out); break;
    case 64:  hipLaunchKernelGGL(group_code_dot_kernel<64>, grid, block, 0, stream, cw, dW, total, out); break;
    case 128: hipLaunchKernelGGL(group_code_dot_kernel<128>, grid, block, 0, stream, cw, dW, total, out); break;
    case 256: hipLaunchKernelGGL(group_code_dot_kernel<256>, grid, block, 0, stream, cw, dW, total, out); break;
    case 512: hipLaunchKernelGGL(group_code_dot_kernel<512>, grid, block, 0, stream, cw, dW, total, out); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
