// Gradient of a per-group magnitude that multiplies the ternary codes:
//   out[n, j] = sum_{i < g} q[n, j g + i] * dW[n, j g + i]
// (the appendix's decoupled quantization, What = alpha_g * q, and the
// magnitude path of a learnable scale, Sec. 4), where dW is the gradient with
// respect to the dequantized weights (dY^T X, the straight-through dW).
//
// HBM bound: one pass over dW (4 bytes per weight) and the packed codes
// (1/4 byte).  A persistent grid walks 1024-weight units per wave; each lane
// owns 16 consecutive weights, i.e. one packed code word (all in one group,
// g >= 32), and reads their dW as four 16-byte loads.  Products are summed
// in float64 (16 terms per lane, then a butterfly over the g / 16 lanes of a
// group) and rounded to float32 once; float64 holds these sums exactly
// unless a group's terms span more than about 2^20 in magnitude.
#include "common.hpp"

namespace tmk {

constexpr int kGcdUnit = 1024;
constexpr int kGcdWaves = 16;

template <int G>
__global__ __launch_bounds__(64 * kGcdWaves) void group_code_dot_kernel(
    const uint32_t* __restrict__ codes, const float* __restrict__ dW, int64_t total,
    float* __restrict__ out) {
  constexpr int L = G / 16;  // lanes holding one group
  static_assert(L >= 2 && L <= 32, "16 weights per lane, groups of 32 .. 512");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t nunits = (total + kGcdUnit - 1) / kGcdUnit;
  for (int64_t u = (int64_t)blockIdx.x * kGcdWaves + wave; u < nunits;
       u += (int64_t)gridDim.x * kGcdWaves) {
    // wave-uniform unit base, 32-bit lane offset kept opaque so that the
    // compiler does not hoist the derived addresses out of the loop
    const int64_t base = u * kGcdUnit;
    const int64_t rem = total - base;
    const int lim = rem < kGcdUnit ? (int)rem : kGcdUnit;
    int lo = 16 * lane;
    asm volatile("" : "+v"(lo));
    const bool ok = lo < lim;  // total % 16 == 0: all 16 weights valid or none
    u32x4 v[4] = {};
    uint32_t w = 0u;
    if (ok) {
      const float* p = dW + base + lo;
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = ld16(p + 4 * i);
      w = codes[(base + lo) / 16];
    }
    double ps = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t dv[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = 4 * i + k;  // element within the word
        const uint32_t c = (w >> (2 * (j / 2) + 16 * (j % 2))) & 3u;
        // 01 -> +dW, 11 -> -dW, 00 (and the unused 10) -> 0
        const float f = __uint_as_float(dv[k] ^ ((c >> 1) << 31));
        ps += (c & 1u) ? (double)f : 0.0;
      }
    }
    ps = group_sum_f64<L>(ps);
    if (ok && (lane % L) == 0) out[(base + lo) / G] = (float)ps;
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
