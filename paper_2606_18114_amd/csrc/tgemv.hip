// Decode-time ternary GEMV (batch B <= 16), strided-batched over matrices.
//
// Batch-1 decoding is bound by the weight bytes (paper Sec. 8), so the
// kernel streams the packed codes once from HBM and does the arithmetic on
// the matrix cores, where it costs nothing: one v_mfma_f32_16x16x32_bf16
// takes the (zero-padded) activations x as the A operand (rows = batch) and
// sixteen weight rows, decoded to exact bfloat16 2*q, as the B operand.
// Decoding is one shift and one AND per two codes (common.hpp).
//
// Work split: a workgroup (4 waves) owns 64 weight rows of one matrix; each
// wave takes every fourth 512-wide slice of K and keeps partial sums for its
// 64 rows; the four partials are added through LDS at the end.
//
// Within a K chunk of C = min(g, 128) columns the 4 lane groups of the MFMA
// own C/4 contiguous columns each and MFMA step t uses octet t of every lane
// group's range, so each step stays inside one quantization group and the
// float16 scale can be applied per chunk in float32:
//   acc += s * sum_t mfma(x_t, 2q_t) ,  y = acc / 2.
#include "common.hpp"

namespace tmk {

constexpr int kGemvRows = 64;    // rows per workgroup (4 MFMA row blocks)
constexpr int kGemvSlice = 512;  // K columns per wave pass

template <int G>
__global__ __launch_bounds__(256) void tgemv_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales_f16, int B, int64_t N, int64_t K,
    float* __restrict__ y) {
  constexpr int C = G < 128 ? G : 128;  // chunk width
  constexpr int SPC = C / 32;           // MFMA steps per chunk
  constexpr int CPS = kGemvSlice / C;   // chunks per full slice
  __shared__ float red[4][4][4][64];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;  // weight row within a 16-row block; batch row for x
  const int lg = lane >> 4;   // MFMA lane group (k octet group)
  const int64_t mat = blockIdx.y;
  const int64_t n0 = (int64_t)blockIdx.x * kGemvRows;
  const int64_t kw = K / 16;  // words per code row
  const int64_t ng = K / G;   // groups per row

  const uint32_t* cw = reinterpret_cast<const uint32_t*>(codes) + mat * N * kw;
  const uint16_t* sm = scales_f16 + mat * N * ng;
  const uint16_t* xm = x + mat * (int64_t)B * K;
  const bool xrow = col < B;
  const uint16_t* xr = xm + (int64_t)(xrow ? col : 0) * K;

  int64_t rows[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    int64_t n = n0 + rb * 16 + col;
    rows[rb] = n < N ? n : N - 1;
  }

  f32x4 acc[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nslices = (K + kGemvSlice - 1) / kGemvSlice;
  for (int64_t sl = wave; sl < nslices; sl += 4) {
    const int64_t kbase = sl * kGemvSlice;
    const int64_t krem = K - kbase;
    const int nch = krem >= kGemvSlice ? CPS : (int)(krem / C);
    for (int ch = 0; ch < nch; ++ch) {
      const int64_t k0 = kbase + (int64_t)ch * C;
      // x operand for the SPC steps of this chunk
      bf16x8 xa[SPC];
#pragma unroll
      for (int t = 0; t < SPC; ++t) {
        const int64_t kx = k0 + 8 * (lg * SPC + t);
        u32x4 v = ld16(xr + kx);
        if (!xrow) v = u32x4{0u, 0u, 0u, 0u};
        xa[t] = as_bf16x8(v);
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        const uint32_t* crow = cw + rows[rb] * kw + k0 / 16;
        const float s = (float)__builtin_bit_cast(_Float16, sm[rows[rb] * ng + k0 / G]);
        f32x4 p = {0.f, 0.f, 0.f, 0.f};
        if constexpr (C == 128) {
          const u32x2 wv = *reinterpret_cast<const u32x2*>(crow + 2 * lg);
          p = mfma16(xa[0], decode_half<0>(wv.x), p);
          p = mfma16(xa[1], decode_half<1>(wv.x), p);
          p = mfma16(xa[2], decode_half<0>(wv.y), p);
          p = mfma16(xa[3], decode_half<1>(wv.y), p);
        } else if constexpr (C == 64) {
          const uint32_t w = crow[lg];
          p = mfma16(xa[0], decode_half<0>(w), p);
          p = mfma16(xa[1], decode_half<1>(w), p);
        } else {
          const uint32_t w = crow[lg >> 1];
          p = mfma16(xa[0], decode_half_rt(w, lg & 1), p);
        }
        acc[rb] += s * p;
      }
    }
  }

#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    red[wave][rb][0][lane] = acc[rb].x;
    red[wave][rb][1][lane] = acc[rb].y;
    red[wave][rb][2][lane] = acc[rb].z;
    red[wave][rb][3][lane] = acc[rb].w;
  }
  __syncthreads();

  // thread t sums the four waves' partials for (row block t/64, lane t%64)
  const int rb = threadIdx.x >> 6;
  const int l = threadIdx.x & 63;
  const int64_t n = n0 + rb * 16 + (l & 15);
  if (n < N) {
    float* ym = y + mat * (int64_t)B * N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int b = 4 * (l >> 4) + i;
      if (b < B) {
        const float v = red[0][rb][i][l] + red[1][rb][i][l] + red[2][rb][i][l] + red[3][rb][i][l];
        ym[(int64_t)b * N + n] = 0.5f * v;
      }
    }
  }
}

hipError_t launch_tgemv(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                        int B, int64_t N, int64_t K, int g, float* y, hipStream_t stream) {
  const dim3 grid((unsigned)((N + kGemvRows - 1) / kGemvRows), (unsigned)count), block(256);
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemv_kernel<32>, grid, block, 0, stream, x, codes, s16, B, N, K, y); break;
    case 64:  hipLaunchKernelGGL(tgemv_kernel<64>, grid, block, 0, stream, x, codes, s16, B, N, K, y); break;
    case 128: hipLaunchKernelGGL(tgemv_kernel<128>, grid, block, 0, stream, x, codes, s16, B, N, K, y); break;
    case 256: hipLaunchKernelGGL(tgemv_kernel<256>, grid, block, 0, stream, x, codes, s16, B, N, K, y); break;
    case 512: hipLaunchKernelGGL(tgemv_kernel<512>, grid, block, 0, stream, x, codes, s16, B, N, K, y); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
