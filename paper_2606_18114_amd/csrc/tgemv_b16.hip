// Decode-time ternary GEMV for batches of 9 to 16 rows (paper Sec. 8: decode
// reads every weight once per step; with more tokens per step the products
// grow and the vector ALUs of the FP8-split form become the bound).
//
// The batch rows fill the 16 A rows of v_mfma_f32_16x16x32_bf16 as they are
// (bfloat16, rows past B zero), and the codes of 16 weight rows are the B
// operand, decoded to bfloat16 2q by one shift and one AND per two codes, so
// the products are exact and the sums float32.  A lane with column n (its
// weight row, also its A row) and k quarter kq takes, for each 64-column
// chunk of a row, the chunk's code word kq: its first half gives the chunk's
// first k step (columns 16 kq + 0..7) and its second half the second (16 kq
// + 8..15); the A operand carries the same columns of x.  Each group's sum is
// scaled by its float16 scale into a float32 total.
//
// One workgroup of four waves per (matrix, four consecutive 16-row blocks),
// or per single block when a launch has few blocks; wave w takes a
// contiguous quarter of the rows' groups, with the loads of eight chunks in
// flight at a time (each chunk's x, from L2, shared by the workgroup's
// blocks), and the four waves' totals are added in LDS in wave order
// (deterministic).
#include "common.hpp"
#include "launchers.hpp"
#include "mixer_dev.hpp"

namespace tmk {

constexpr int kB16Chunks = 8;  // 64-column chunks whose loads are in flight together

// NB: 16-row blocks per workgroup (consecutive), sharing each chunk of x
template <int G, int NB>
__global__ __launch_bounds__(256) void tgemv_b16_kernel(const uint16_t* __restrict__ x,
                                                        const uint8_t* __restrict__ codes,
                                                        const uint16_t* __restrict__ s16,
                                                        int B, int N, int K, int nblk,
                                                        float* __restrict__ y) {
  static_assert(G % 64 == 0 && kB16Chunks % (G / 64 > 0 ? G / 64 : 1) == 0,
                "groups of whole chunks, whole groups per round");
  constexpr int kWpg = G / 64;                // chunks per group
  constexpr int kScales = kB16Chunks / kWpg;  // groups per round
  __shared__ float red[4 * NB * 64 * 4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, kq = lane >> 4;
  const int c = blockIdx.x / nblk, j0 = NB * (blockIdx.x % nblk);
  const bool xok = n < B;
  const int ngr = K / G, gpw = (ngr + 3) / 4, g0 = wave * gpw;
  const int gw = ngr - g0 < gpw ? (ngr - g0 > 0 ? ngr - g0 : 0) : gpw;  // groups of this wave
  const int nch = gw * kWpg;
  const uint32_t* crow[NB];
  const uint16_t* srow[NB];
  bool rok[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int row = 16 * (j0 + b) + n;
    rok[b] = row < N;
    crow[b] = reinterpret_cast<const uint32_t*>(codes +
                                                ((int64_t)c * N + (rok[b] ? row : 0)) * (K / 4));
    srow[b] = s16 + ((int64_t)c * N + (rok[b] ? row : 0)) * (K / G);
  }
  const uint16_t* xrow = x + ((int64_t)c * B + (xok ? n : 0)) * K;

  float tot[NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < 4; ++e) tot[b][e] = 0.f;
  for (int i0 = 0; i0 < nch; i0 += kB16Chunks) {
    uint32_t cw[kB16Chunks][NB];
    u32x4 xa[kB16Chunks][2];
    uint16_t sc[NB][kScales];
#pragma unroll
    for (int t = 0; t < kB16Chunks; ++t) {
      const int i = i0 + t;
      const int col = g0 * G + 64 * i + 16 * kq;
      xa[t][0] = xa[t][1] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int b = 0; b < NB; ++b) cw[t][b] = 0u;
      if (i < nch) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
          if (rok[b]) cw[t][b] = crow[b][col / 16];
        if (xok) {
          xa[t][0] = ld16(xrow + col);
          xa[t][1] = ld16(xrow + col + 8);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < kScales; ++r) {
        const int gi = i0 / kWpg + r;
        sc[b][r] = rok[b] && gi < gw ? srow[b][g0 + gi] : (uint16_t)0;
      }
    f32x4 acc[NB];
#pragma unroll
    for (int t = 0; t < kB16Chunks; ++t) {
      if (i0 + t < nch) {  // uniform
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          if (t % kWpg == 0) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
          const uint32_t w = cw[t][b];
          const u32x4 b0 = {(w << 14) & kPairMask, (w << 12) & kPairMask, (w << 10) & kPairMask,
                            (w << 8) & kPairMask};
          const u32x4 b1 = {(w << 6) & kPairMask, (w << 4) & kPairMask, (w << 2) & kPairMask,
                            w & kPairMask};
          acc[b] = mfma16(as_bf16x8(xa[t][0]), as_bf16x8(b0), acc[b]);
          acc[b] = mfma16(as_bf16x8(xa[t][1]), as_bf16x8(b1), acc[b]);
          if (t % kWpg == kWpg - 1) {
            const float s = h2f(sc[b][t / kWpg]);
#pragma unroll
            for (int e = 0; e < 4; ++e) tot[b][e] = __builtin_fmaf(acc[b][e], s, tot[b][e]);
          }
        }
      }
    }
  }
  // lane (kq, n) holds batch rows 4 kq + e of weight row n of each block; the
  // waves meet in LDS
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[((wave * NB + b) * 64 + lane) * 4 + e] = tot[b][e];
  __syncthreads();
  {
    const int b = wave;  // wave b writes block b (NB <= 4)
    if (b < NB) {
      const int row = 16 * (j0 + b) + n;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = 4 * kq + e;
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) sum += red[((w * NB + b) * 64 + lane) * 4 + e];
        // the codes decode to 2q
        if (m < B && row < N) y[((int64_t)c * B + m) * N + row] = 0.5f * sum;
      }
    }
  }
}

// four blocks per workgroup (x read once per 64 rows) when that still gives
// two workgroups per CU, else one
template <int G>
static hipError_t launch_b16_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                               int count, int B, int64_t N, int64_t K, float* y,
                               hipStream_t stream) {
  if (N > 0x7FFFFFFF || K > 0x7FFFFFFF) return hipErrorInvalidValue;
  const int64_t nb4 = (N + 63) / 64;
  if ((int64_t)count * nb4 >= 2 * current_cu_count() && (int64_t)count * nb4 <= 0x7FFFFFFF) {
    hipLaunchKernelGGL((tgemv_b16_kernel<G, 4>), dim3((unsigned)(count * nb4)), dim3(256), 0,
                       stream, x, codes, s16, B, (int)N, (int)K, (int)nb4, y);
    return hipGetLastError();
  }
  const int64_t nb1 = (N + 15) / 16, grid = (int64_t)count * nb1;
  if (grid < 1 || grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL((tgemv_b16_kernel<G, 1>), dim3((unsigned)grid), dim3(256), 0, stream, x,
                     codes, s16, B, (int)N, (int)K, (int)nb1, y);
  return hipGetLastError();
}

bool tgemv_b16_takes(int B, int g) { return B >= 9 && B <= 16 && g >= 64 && g <= 512; }

hipError_t launch_tgemv_b16(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                            int count, int B, int64_t N, int64_t K, int g, float* y,
                            hipStream_t stream) {
  if (!tgemv_b16_takes(B, g) || K % 64 != 0 || K % g != 0) return hipErrorInvalidValue;
  switch (g) {
    case 64:  return launch_b16_g<64>(x, codes, s16, count, B, N, K, y, stream);
    case 128: return launch_b16_g<128>(x, codes, s16, count, B, N, K, y, stream);
    case 256: return launch_b16_g<256>(x, codes, s16, count, B, N, K, y, stream);
    case 512: return launch_b16_g<512>(x, codes, s16, count, B, N, K, y, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tmk
