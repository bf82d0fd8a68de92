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

// Learnable scale with the rounding straight-through (clip keeps its
// derivative):  What = s * round(clip(w / d, -1, 1)),  d = fl32(s + eps),
//   ds[n, j] = sum_i dWhat_i * (q_i - m_i * w_i * s / d^2),
//   dw_i     = dWhat_i * m_i * s / d,
// where m_i = 1 iff the float32 quotient |w_i| / d is at most 1, i.e. iff
// |w_i| <= d (1 + 2^-24) exactly (round-to-nearest-even sends (1, 1 + 2^-24]
// to 1); the product d (1 + 2^-24) is exact in float64.  Same layout as
// above: one code word and its 16 weights per lane; the per-element terms
// and the group sums are float64, each result rounded once to float32.
// dw may be the dWhat array itself (each lane reads its 16 values before it
// writes them), so neither pointer is declared restrict.
template <int G>
__global__ __launch_bounds__(64 * kGcdWaves) void scale_ste_grad_kernel(
    const float* __restrict__ W, const uint32_t* __restrict__ codes,
    const float* __restrict__ scale, const float* dWhat, int64_t total, float eps,
    float* __restrict__ ds, float* dw) {
  constexpr int L = G / 16;
  static_assert(L >= 2 && L <= 32, "16 weights per lane, groups of 32 .. 512");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t nunits = (total + kGcdUnit - 1) / kGcdUnit;
  for (int64_t u = (int64_t)blockIdx.x * kGcdWaves + wave; u < nunits;
       u += (int64_t)gridDim.x * kGcdWaves) {
    const int64_t base = u * kGcdUnit;
    const int64_t rem = total - base;
    const int lim = rem < kGcdUnit ? (int)rem : kGcdUnit;
    int lo = 16 * lane;
    asm volatile("" : "+v"(lo));
    const bool ok = lo < lim;
    u32x4 wv[4] = {}, gv[4] = {};
    uint32_t cw = 0u;
    float sc = 1.f;
    if (ok) {
      const int64_t e0 = base + lo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        wv[i] = ld16(W + e0 + 4 * i);
        gv[i] = ld16(dWhat + e0 + 4 * i);
      }
      cw = codes[e0 / 16];
      sc = scale[e0 / G];
    }
    const float d = sc + eps;                        // float32, as the codes use it
    const double dd = (double)d;
    const double bound = dd * (1.0 + 0x1p-24);       // exact
    const double fs = (double)sc / (dd * dd);        // s / d^2
    const double fw = (double)sc / dd;               // s / d
    double ps = 0.0;
    float out[16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t wa[4] = {wv[i].x, wv[i].y, wv[i].z, wv[i].w};
      const uint32_t ga[4] = {gv[i].x, gv[i].y, gv[i].z, gv[i].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = 4 * i + k;
        const uint32_t c = (cw >> (2 * (j / 2) + 16 * (j % 2))) & 3u;
        const double q = (c & 1u) ? ((c & 2u) ? -1.0 : 1.0) : 0.0;
        const double w = (double)__uint_as_float(wa[k]);
        const double gr = (double)__uint_as_float(ga[k]);
        const bool m = fabs(w) <= bound;
        ps += gr * (m ? q - w * fs : q);
        out[j] = m ? (float)(gr * fw) : 0.f;
      }
    }
    if (ok && dw != nullptr) {
      float* p = dw + base + lo;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st16(p + 4 * i, u32x4{__float_as_uint(out[4 * i]), __float_as_uint(out[4 * i + 1]),
                              __float_as_uint(out[4 * i + 2]), __float_as_uint(out[4 * i + 3])});
    }
    ps = group_sum_f64<L>(ps);
    if (ok && (lane % L) == 0) ds[(base + lo) / G] = (float)ps;
  }
}

hipError_t launch_scale_ste_grad(const float* W, const uint8_t* codes, const float* scale,
                                 const float* dWhat, int64_t N, int64_t K, int g, float eps,
                                 float* ds, float* dw, hipStream_t stream) {
  const int64_t total = N * K;
  int64_t blocks = (total / kGcdUnit + kGcdWaves) / kGcdWaves;
  if (blocks > 512) blocks = 512;
  const dim3 grid((unsigned)blocks), block(64 * kGcdWaves);
  auto* cw = reinterpret_cast<const uint32_t*>(codes);
#define TM_SSG(G_)                                                                          \
  hipLaunchKernelGGL(scale_ste_grad_kernel<G_>, grid, block, 0, stream, W, cw, scale, dWhat, \
                     total, eps, ds, dw)
  switch (g) {
    case 32:  TM_SSG(32); break;
    case 64:  TM_SSG(64); break;
    case 128: TM_SSG(128); break;
    case 256: TM_SSG(256); break;
    case 512: TM_SSG(512); break;
    default: return hipErrorInvalidValue;
  }
#undef TM_SSG
  return hipGetLastError();
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
