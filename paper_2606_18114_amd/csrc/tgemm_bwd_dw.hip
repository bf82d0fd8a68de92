// Straight-through backward w.r.t. the latent weight (paper Sec. 3.1,
// identity estimator: the gradient of What passes to W unchanged):
//   dW[N, K] = dY[M, N]^T . X[M, K],
// a contraction over the M tokens on the gfx950 matrix cores.
//
// Both operands arrive token-major, so each MFMA operand (eight consecutive
// tokens of one column) is gathered from LDS tiles kept in their natural
// [token][column] order.  Tile: 256 (N) x 256 (K) outputs per workgroup of
// 8 waves (2 x 4), 128 x 64 per wave, 32 tokens per stage.  The token range
// is split across workgroups (split-K) so that the grid fills the chip; the
// partial tiles are added into dW with float32 atomics.
#include "common.hpp"

namespace tmk {

constexpr int kDwBN = 256, kDwBK = 256, kDwBM = 32;
constexpr int kDwStride = 256 + 8;  // bf16 per LDS row

__global__ void fill_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 3 < n) {
    *reinterpret_cast<f32x4*>(p + i) = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
    for (int64_t j = i; j < n; ++j) p[j] = 0.f;
  }
}

__global__ __launch_bounds__(512) void tgemm_bwd_dw_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X, int64_t M,
    int64_t N, int64_t K, float* __restrict__ dW, uint32_t tiles_k,
    uint32_t tiles_nk, int64_t m_per_split) {
  __shared__ __attribute__((aligned(16))) uint16_t ys[kDwBM][kDwStride];
  __shared__ __attribute__((aligned(16))) uint16_t xs[kDwBM][kDwStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave >> 2, wk = wave & 3;
  const int h = lane >> 5;
  const int l32 = lane & 31;

  const uint32_t bid = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t split = bid / tiles_nk;
  const uint32_t t = bid % tiles_nk;
  const int64_t n0 = (int64_t)(t / tiles_k) * kDwBN;
  const int64_t k0 = (int64_t)(t % tiles_k) * kDwBK;
  const int64_t mbeg = (int64_t)split * m_per_split;
  const int64_t mend = mbeg + m_per_split < M ? mbeg + m_per_split : M;

  // staging: each operand tile is 32 rows x 32 pieces of 16 bytes; thread
  // tid loads piece (tid & 31) of rows (tid >> 5) and (tid >> 5) + 16
  const int prow = tid >> 5;
  const int pcol = (tid & 31) * 8;
  const bool y_ok = n0 + pcol < N;
  const bool x_ok = k0 + pcol < K;

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

  for (int64_t mb = mbeg; mb < mend; mb += kDwBM) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int row = prow + 16 * r;
      const int64_t m = mb + row;
      u32x4 vy = {0u, 0u, 0u, 0u}, vx = {0u, 0u, 0u, 0u};
      if (m < mend) {
        if (y_ok) vy = ld16(dY + m * N + n0 + pcol);
        if (x_ok) vx = ld16(X + m * K + k0 + pcol);
      }
      st16(&ys[row][pcol], vy);
      st16(&xs[row][pcol], vx);
    }
    __syncthreads();

#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8 bop[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int kk = wk * 64 + b * 32 + l32;
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 16 * s + 8 * h + 2 * e;
          v[e] = (uint32_t)xs[r][kk] | ((uint32_t)xs[r + 1][kk] << 16);
        }
        bop[b] = as_bf16x8(v);
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int nn = wn * 128 + a * 32 + l32;
        u32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 16 * s + 8 * h + 2 * e;
          v[e] = (uint32_t)ys[r][nn] | ((uint32_t)ys[r + 1][nn] << 16);
        }
        const bf16x8 aop = as_bf16x8(v);
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = mfma32(aop, bop[b], acc[a][b]);
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
        const int64_t n = n0 + wn * 128 + a * 32 + 8 * (i / 4) + 4 * h + (i % 4);
        if (n < N) atomicAdd(dW + n * K + k, acc[a][b][i]);
      }
    }
  }
}

hipError_t launch_tgemm_bwd_dw(const uint16_t* dY, const uint16_t* X, int64_t M, int64_t N,
                               int64_t K, float* dW, int accumulate, hipStream_t stream) {
  if (!accumulate) {
    const int64_t n = N * K;
    const int64_t threads = (n + 3) / 4;
    hipLaunchKernelGGL(fill_zero_f32, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                       stream, dW, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t tn = (N + kDwBN - 1) / kDwBN, tk = (K + kDwBK - 1) / kDwBK;
  const int64_t tiles = tn * tk;
  // enough splits of the token range for about eight workgroups per CU in
  // total, each split at least 256 tokens long
  int64_t splits = (2048 + tiles - 1) / tiles;
  const int64_t max_splits = (M + 255) / 256;
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  int64_t mps = (M + splits - 1) / splits;
  mps = (mps + kDwBM - 1) / kDwBM * kDwBM;
  splits = (M + mps - 1) / mps;
  const dim3 grid((unsigned)(tiles * splits)), block(512);
  hipLaunchKernelGGL(tgemm_bwd_dw_kernel, grid, block, 0, stream, dY, X, M, N, K, dW,
                     (uint32_t)tk, (uint32_t)tiles, mps);
  return hipGetLastError();
}

}  // namespace tmk
