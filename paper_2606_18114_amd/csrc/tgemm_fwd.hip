// Ternary forward GEMM (paper Sec. 3.1): Y[M, N] = X[M, K] . What[N, K]^T,
// What = s * q, on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// Tile: 256 x 256 outputs per workgroup of 8 waves (2 x 4), 128 x 64 per
// wave (4 x 2 MFMA blocks), K advanced 64 columns per pipeline stage.
//   * X (bf16) goes global -> registers -> LDS (double buffered, rows padded
//     to 144 bytes so the 32-row MFMA reads are bank-conflict free).
//   * The packed codes never touch LDS: every lane loads the 16 bytes (64
//     codes) of its own weight row per stage and decodes its MFMA operand
//     in registers, one shift and one AND per two codes, to the exact
//     bfloat16 values 2*q.
//   * The group scale is applied in float32, not folded into the bfloat16
//     operand (folding would cost about 2e-3 relative error).  Instead of a
//     second set of partial accumulators, the accumulator is kept in units
//     of the current group's scale c: when the next group (scale s) starts,
//     the accumulator is multiplied by c / s and c becomes s, so the matrix
//     cores keep adding exact products into one register set.  At the end
//     Y = c * acc / 2.  Groups with s = 0 are masked out of the operand.
#include "common.hpp"

namespace tmk {

constexpr int kFwdBM = 256, kFwdBN = 256, kFwdBK = 64;
constexpr int kFwdLdsStride = kFwdBK + 8;  // bf16 elements per LDS row

template <int G>
__global__ __launch_bounds__(512) void tgemm_fwd_kernel(
    const uint16_t* __restrict__ X, const uint32_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    float* __restrict__ Y, uint32_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][kFwdBM][kFwdLdsStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const uint32_t h = (uint32_t)(lane >> 5);  // k half of the MFMA operand
  const int l32 = lane & 31;

  const uint32_t bid = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t m0 = (int64_t)(bid / tiles_n) * kFwdBM;
  const int64_t n0 = (int64_t)(bid % tiles_n) * kFwdBN;
  const int64_t kw = K / 16;
  const int64_t ng = K / G;
  const int nchunks = (int)(K / kFwdBK);

  // weight rows (MFMA columns) of this lane, clamped for the ragged edge
  int64_t nrow[2];
  const uint32_t* crow[2];
  const float* srow[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    int64_t n = n0 + wn * 64 + b * 32 + l32;
    nrow[b] = n;
    n = n < N ? n : N - 1;
    crow[b] = codes + n * kw;
    srow[b] = scales + n * ng;
  }

  // X tile staging: 2048 16-byte pieces, 4 per thread
  const uint16_t* xsrc[4];
  int xrow[4], xcol[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int idx = tid + 512 * i;
    xrow[i] = idx >> 3;
    xcol[i] = (idx & 7) * 8;
    int64_t m = m0 + xrow[i];
    m = m < M ? m : M - 1;
    xsrc[i] = X + m * K + xcol[i];
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  float cref[2] = {0.f, 0.f};
  uint32_t msk[2] = {0u, 0u};

  // Group scales run one stage ahead: the scales used by the boundaries of
  // stage kc are loaded at the start of stage kc - 1, before that stage's
  // operand prefetch, so waiting for them never waits for the prefetch.  A
  // 64-column stage holds at most two group starts (g = 32).  Every load in
  // the loop is unconditional (the last stage reloads itself) so the
  // compiler can count outstanding loads exactly.
  constexpr int kStarts = G == 32 ? 2 : 1;
  float snext[kStarts][2], scur[kStarts][2];
  auto load_scales = [&](int kc_) {
#pragma unroll
    for (int q = 0; q < kStarts; ++q) {
      int64_t j = ((int64_t)kc_ * kFwdBK + 32 * q) / G;
      j = j < ng ? j : ng - 1;
#pragma unroll
      for (int b = 0; b < 2; ++b) snext[q][b] = srow[b][j];
    }
  };
  load_scales(0);

  // prologue: stage chunk 0
  u32x4 xv[4], cv[2], cvn[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) xv[i] = ld16(xsrc[i]);
#pragma unroll
  for (int b = 0; b < 2; ++b) cv[b] = ld16(crow[b]);
#pragma unroll
  for (int i = 0; i < 4; ++i) st16(&xs[0][xrow[i]][xcol[i]], xv[i]);
  __syncthreads();

  for (int kc = 0; kc < nchunks; ++kc) {
    const int buf = kc & 1;
    const int kn = kc + 1 < nchunks ? kc + 1 : kc;
#pragma unroll
    for (int q = 0; q < kStarts; ++q)
#pragma unroll
      for (int b = 0; b < 2; ++b) scur[q][b] = snext[q][b];
    load_scales(kn);
    {
      const int64_t ko = (int64_t)kn * kFwdBK;
#pragma unroll
      for (int i = 0; i < 4; ++i) xv[i] = ld16(xsrc[i] + ko);
#pragma unroll
      for (int b = 0; b < 2; ++b) cvn[b] = ld16(crow[b] + ko / 16);
    }

#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t kcol = (int64_t)kc * kFwdBK + 16 * t;
      const bool boundary = (t == 0 && (kcol % G) == 0) || (G == 32 && t == 2);
      if (boundary) {
        const int q = (G == 32 && t == 2) ? kStarts - 1 : 0;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const float sv = scur[q][b];
          msk[b] = sv != 0.f ? 0xFFFFFFFFu : 0u;
          const float r = (sv != 0.f && cref[b] != 0.f) ? cref[b] / sv : 1.f;
          cref[b] = sv != 0.f ? sv : cref[b];
#pragma unroll
          for (int a = 0; a < 4; ++a) acc[a][b] *= r;
        }
      }
      bf16x8 bop[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const uint32_t w = (t == 0 ? cv[b].x : t == 1 ? cv[b].y : t == 2 ? cv[b].z : cv[b].w) & msk[b];
        bop[b] = decode_half_rt(w, h);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const u32x4 av = *reinterpret_cast<const u32x4*>(&xs[buf][wm * 128 + a * 32 + l32][16 * t + 8 * h]);
        const bf16x8 aop = as_bf16x8(av);
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(aop, bop[b], acc[a][b]);
      }
    }

#pragma unroll
    for (int i = 0; i < 4; ++i) st16(&xs[buf ^ 1][xrow[i]][xcol[i]], xv[i]);
#pragma unroll
    for (int b = 0; b < 2; ++b) cv[b] = cvn[b];
    __syncthreads();
  }

  // epilogue: lane holds column l32 of each block, rows 8*(i/4) + 4*h + i%4
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int64_t n = nrow[b];
    if (n >= N) continue;
    const float f = 0.5f * cref[b];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t m = m0 + wm * 128 + a * 32 + 8 * (i / 4) + 4 * h + (i % 4);
        if (m < M) Y[m * N + n] = f * acc[a][b][i];
      }
    }
  }
}

hipError_t launch_tgemm_fwd(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int g, float* Y,
                            hipStream_t stream) {
  const int64_t tm = (M + kFwdBM - 1) / kFwdBM, tn = (N + kFwdBN - 1) / kFwdBN;
  const dim3 grid((unsigned)(tm * tn)), block(512);
  const auto* cw = reinterpret_cast<const uint32_t*>(codes);
  const uint32_t t_n = (uint32_t)tn;
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemm_fwd_kernel<32>, grid, block, 0, stream, X, cw, scales, M, N, K, Y, t_n); break;
    case 64:  hipLaunchKernelGGL(tgemm_fwd_kernel<64>, grid, block, 0, stream, X, cw, scales, M, N, K, Y, t_n); break;
    case 128: hipLaunchKernelGGL(tgemm_fwd_kernel<128>, grid, block, 0, stream, X, cw, scales, M, N, K, Y, t_n); break;
    case 256: hipLaunchKernelGGL(tgemm_fwd_kernel<256>, grid, block, 0, stream, X, cw, scales, M, N, K, Y, t_n); break;
    case 512: hipLaunchKernelGGL(tgemm_fwd_kernel<512>, grid, block, 0, stream, X, cw, scales, M, N, K, Y, t_n); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
