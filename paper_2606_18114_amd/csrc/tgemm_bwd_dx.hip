// Straight-through backward w.r.t. the input (paper Sec. 3.1):
//   dX[M, K] = dY[M, N] . What[N, K],  What = s * q,
// a contraction over N on the gfx950 matrix cores (32x32x16 bf16 MFMA).
//
// The scale varies along the contraction, so it cannot be applied after the
// MFMA as in the forward kernel.  Folding it into one bfloat16 operand would
// cost about 2e-3 relative error; instead every dequantized weight is split
// exactly into two bfloat16 terms, q*s_hi + q*s_lo with s_hi = bf16(s) and
// s_lo = bf16(s - s_hi) (together 16 significant bits of s), and both terms
// run on the matrix cores against the same dY operand and accumulator.
//
// Tile: 256 (M) x 256 (K) outputs per workgroup of 8 waves (2 x 4), 128 x 64
// per wave; the contraction advances 32 rows of N per stage.  Per stage:
//   * dY [256 x 32] bf16 goes to LDS as loaded (rows padded to 80 bytes);
//   * the codes of [32 x 256] weights are decoded by all threads into the
//     two bfloat16 planes q*s_hi and q*s_lo in LDS, in natural [n][k] order;
//   * each MFMA B operand (eight consecutive n of one column k) is gathered
//     from the planes with 16-bit LDS reads.
#include "common.hpp"

namespace tmk {

constexpr int kDxBM = 256, kDxBK = 256, kDxBN = 32;
constexpr int kDxYStride = kDxBN + 8;   // bf16 per LDS row of the dY tile
constexpr int kDxWStride = kDxBK + 8;   // bf16 per LDS row of a weight plane

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <int G>
__global__ __launch_bounds__(512) void tgemm_bwd_dx_kernel(
    const uint16_t* __restrict__ dY, const uint32_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    float* __restrict__ dX, uint32_t tiles_k) {
  __shared__ __attribute__((aligned(16))) uint16_t ys[kDxBM][kDxYStride];
  __shared__ __attribute__((aligned(16))) uint16_t whi[kDxBN][kDxWStride];
  __shared__ __attribute__((aligned(16))) uint16_t wlo[kDxBN][kDxWStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 2, wk = wave & 3;
  const int h = lane >> 5;
  const int l32 = lane & 31;

  const uint32_t bid = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(bid / tiles_k) * kDxBM;
  const int64_t k0 = (int64_t)(bid % tiles_k) * kDxBK;
  const int64_t kw = K / 16;
  const int64_t ng = K / G;
  const int64_t nchunks = (N + kDxBN - 1) / kDxBN;

  // dY staging: 256 rows x 4 pieces of 16 bytes, 2 per thread
  int yrow[2], ycol[2];
  const uint16_t* ysrc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int idx = tid + 512 * i;
    yrow[i] = idx >> 2;
    ycol[i] = (idx & 3) * 8;
    int64_t m = m0 + yrow[i];
    m = m < M ? m : M - 1;
    ysrc[i] = dY + m * N + ycol[i];
  }
  // code decode: 32 rows x 16 words, one word per thread
  const int drow = tid >> 4;       // n within the stage
  const int dword_ = tid & 15;     // word within the 256-wide K tile
  const int64_t kd = k0 + 16 * dword_;
  const bool kd_ok = kd < K;

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t nb = c * kDxBN;
    // ---- stage dY ----
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (nb + ycol[i] < N) v = ld16(ysrc[i] + nb);
      st16(&ys[yrow[i]][ycol[i]], v);
    }
    // ---- decode 16 codes of row n into the hi / lo planes ----
    {
      const int64_t n = nb + drow;
      uint32_t w = 0u;
      float s = 0.f;
      if (n < N && kd_ok) {
        w = codes[n * kw + kd / 16];
        s = scales[n * ng + kd / G];
      }
      const uint32_t shi = f32_to_bf16_rne(s);
      const float rem = s - __builtin_bit_cast(float, shi << 16);
      const uint32_t slo = f32_to_bf16_rne(rem);
      const uint32_t hi2 = shi | (shi << 16), lo2 = slo | (slo << 16);
      u32x4 ph[2], pl[2];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t d = (w << (14 - 2 * i)) & kPairMask;  // 2q as bf16 pair
        // 0xFFFF in each half whose code is nonzero (bit 14 / 30 of d)
        const uint32_t nz = ((d >> 14) & 0x00010001u) * 0xFFFFu;
        const uint32_t sg = d & 0x80008000u;
        const uint32_t vh = (nz & hi2) ^ sg, vl = (nz & lo2) ^ sg;
        ph[i / 4][i % 4] = vh;
        pl[i / 4][i % 4] = vl;
      }
      st16(&whi[drow][16 * dword_], ph[0]);
      st16(&whi[drow][16 * dword_ + 8], ph[1]);
      st16(&wlo[drow][16 * dword_], pl[0]);
      st16(&wlo[drow][16 * dword_ + 8], pl[1]);
    }
    __syncthreads();

    // ---- MFMA: two 16-row steps of the contraction ----
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      bf16x8 bh[2], bl[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int kk = wk * 64 + b * 32 + l32;
        u32x4 vh, vl;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 16 * t + 8 * h + 2 * e;
          vh[e] = (uint32_t)whi[r][kk] | ((uint32_t)whi[r + 1][kk] << 16);
          vl[e] = (uint32_t)wlo[r][kk] | ((uint32_t)wlo[r + 1][kk] << 16);
        }
        bh[b] = as_bf16x8(vh);
        bl[b] = as_bf16x8(vl);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const u32x4 av = *reinterpret_cast<const u32x4*>(&ys[wm * 128 + a * 32 + l32][16 * t + 8 * h]);
        const bf16x8 aop = as_bf16x8(av);
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          acc[a][b] = mfma32(aop, bh[b], acc[a][b]);
          acc[a][b] = mfma32(aop, bl[b], acc[a][b]);
        }
      }
    }
    __syncthreads();
  }

#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int64_t k = k0 + wk * 64 + b * 32 + l32;
    if (k >= K) continue;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t m = m0 + wm * 128 + a * 32 + 8 * (i / 4) + 4 * h + (i % 4);
        if (m < M) dX[m * K + k] = acc[a][b][i];
      }
    }
  }
}

hipError_t launch_tgemm_bwd_dx(const uint16_t* dY, const uint8_t* codes, const float* scales,
                               int64_t M, int64_t N, int64_t K, int g, float* dX,
                               hipStream_t stream) {
  const int64_t tm = (M + kDxBM - 1) / kDxBM, tk = (K + kDxBK - 1) / kDxBK;
  const dim3 grid((unsigned)(tm * tk)), block(512);
  const auto* cw = reinterpret_cast<const uint32_t*>(codes);
  const uint32_t t_k = (uint32_t)tk;
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemm_bwd_dx_kernel<32>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k); break;
    case 64:  hipLaunchKernelGGL(tgemm_bwd_dx_kernel<64>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k); break;
    case 128: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<128>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k); break;
    case 256: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<256>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k); break;
    case 512: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<512>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
