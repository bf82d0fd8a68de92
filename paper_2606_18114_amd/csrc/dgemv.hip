// Decode product of a layer kept in FP16 (layer-selective quantization,
// paper Sec. 7: the first and last blocks stay unquantized):
//   y[c, b, n] = sum_k x[c, b, k] * W[c, n, k],  W float16, x bfloat16,
// strided-batched over `count` same-shape matrices, float32 out.
//
// HBM bound: 2 bytes per weight against 1/4 + 2/g for a ternary matrix, so a
// kept in_proj layer streams 34.9 MB where its ternary form streams 4.6 MB.
// Each lane streams 16-byte pieces (8 weights) of its wave's rows, R rows at
// a time with SEG pieces of each row in flight (R * SEG = 16 loads of 16
// bytes per lane, issued together), and multiplies them on the vector ALUs
// in float32: a float16 weight times the float32 value of its bfloat16
// activation is exact, and the products are summed by fused multiply-adds.
// x is staged once per workgroup in LDS as float32 [B][K]; one 32-byte LDS
// read per lane and chunk serves all R rows.  The per-lane partial sums of a
// row meet in a butterfly over the wave.
#include "common.hpp"
#include "launchers.hpp"

namespace tmk {

constexpr int kDgWaves = 4;
constexpr int kDgChunk = 512;  // columns one wave load covers (64 lanes x 8)

__device__ __forceinline__ float wave_sum_f32(float v) {
  v += __uint_as_float(lane_xchg<1>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<2>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<4>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<8>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<16>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<32>(__float_as_uint(v)));
  return v;
}

__device__ __forceinline__ float half_lo(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
}
__device__ __forceinline__ float half_hi(uint32_t w) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// Grid: (ceil(N / (R * kDgWaves)), count); wave w of workgroup i owns rows
// (i * kDgWaves + w) * R .. + R - 1.  LDS: x as B * K floats, or for more
// than one batch row as bfloat16 (half the LDS reads per weight piece, which
// otherwise bound a batch of 4: 8 reads of 16 bytes per 16 bytes of weights;
// the values widen with a shift or an AND per element), then B row factors.
// RMS (one matrix; a decoding block's normalization fused into the staging):
// x[b, k] = bf16(xr[b, k] / sqrt(mean_k xr[b, k]^2 + eps) * nw[k]), the row
// sums taken by one wave per row in a fixed order.  accum: y += instead of =.
template <int BMAX, int R, int SEG, bool RMS>
__global__ __launch_bounds__(64 * kDgWaves) void dgemv_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ W, int B, int64_t N,
    int64_t K, float* __restrict__ y, const float* __restrict__ xr,
    const float* __restrict__ nw, float eps, int accum) {
  constexpr bool XB = BMAX > 1;  // x in LDS as bfloat16
  extern __shared__ __attribute__((aligned(16))) float xs[];
  uint16_t* const xh = reinterpret_cast<uint16_t*>(xs);
  float* const rfac = reinterpret_cast<float*>(
      reinterpret_cast<uint8_t*>(xs) + ((int64_t)B * K * (XB ? 2 : 4) + 15) / 16 * 16);
  const int64_t mat = blockIdx.y;
  const uint16_t* xm = x + mat * (int64_t)B * K;
  const uint16_t* Wm = W + mat * N * K;
  float* ym = y + mat * (int64_t)B * N;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;

  // this wave's rows (one batch row: the first pass's weight loads go out
  // before x is staged, so their latency overlaps the staging; with more
  // batch rows that costs more than it gains, measured)
  const int64_t row0 = ((int64_t)blockIdx.x * kDgWaves + wave) * R;
  u32x4 wv[R][SEG];
  // all loads of a pass at once (rows past N and columns past K re-read an
  // in-bounds piece and are not used)
  auto load_pass = [&](int64_t k0) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t n = row0 + r < N ? row0 + r : N - 1;
#pragma unroll
      for (int j = 0; j < SEG; ++j) {
        int64_t col = k0 + (int64_t)kDgChunk * j + 8 * lane;
        col = col < K ? col : K - 8;
        wv[r][j] = ld16(Wm + n * K + col);
      }
    }
  };
  if constexpr (!XB) load_pass(0);

  if constexpr (RMS) {
    for (int b = wave; b < B; b += kDgWaves) {
      float sq = 0.f;
      for (int64_t k = 4 * lane; k < K; k += 256) {
        const u32x4 v = ld16(xr + (int64_t)b * K + k);
        sq = __builtin_fmaf(__uint_as_float(v.x), __uint_as_float(v.x), sq);
        sq = __builtin_fmaf(__uint_as_float(v.y), __uint_as_float(v.y), sq);
        sq = __builtin_fmaf(__uint_as_float(v.z), __uint_as_float(v.z), sq);
        sq = __builtin_fmaf(__uint_as_float(v.w), __uint_as_float(v.w), sq);
      }
      sq = wave_sum_f32(sq);
      if (lane == 0) rfac[b] = 1.f / sqrtf(sq / (float)K + eps);
    }
    __syncthreads();
    for (int64_t i = threadIdx.x; i < (int64_t)B * K / 4; i += 64 * kDgWaves) {
      const int64_t b = 4 * i / K, k = 4 * i % K;
      const u32x4 v = ld16(xr + 4 * i);
      const u32x4 w = ld16(nw + k);
      const float r = rfac[b];
      const uint32_t a[4] = {v.x, v.y, v.z, v.w}, c[4] = {w.x, w.y, w.z, w.w};
      uint32_t o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint32_t bits = __float_as_uint(__uint_as_float(a[t]) * r * __uint_as_float(c[t]));
        o[t] = (bits + 0x7FFFu + ((bits >> 16) & 1u)) >> 16;  // bf16, nearest even
      }
      if constexpr (XB)
        *reinterpret_cast<u32x2*>(xh + 4 * i) = u32x2{o[0] | (o[1] << 16), o[2] | (o[3] << 16)};
      else
        st16(xs + 4 * i, u32x4{o[0] << 16, o[1] << 16, o[2] << 16, o[3] << 16});
    }
  }
  // x -> LDS (8 values per thread and step; K % 8 == 0), as float32 or as is
  for (int64_t i = threadIdx.x; !RMS && i < (int64_t)B * K / 8; i += 64 * kDgWaves) {
    const u32x4 v = ld16(xm + 8 * i);
    if constexpr (XB) {
      st16(xh + 8 * i, v);
      continue;
    }
    const uint32_t a[4] = {v.x, v.y, v.z, v.w};
    float f[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      f[2 * t] = __uint_as_float(a[t] << 16);
      f[2 * t + 1] = __uint_as_float(a[t] & 0xFFFF0000u);
    }
    st16(xs + 8 * i, u32x4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                           __float_as_uint(f[3])});
    st16(xs + 8 * i + 4, u32x4{__float_as_uint(f[4]), __float_as_uint(f[5]),
                               __float_as_uint(f[6]), __float_as_uint(f[7])});
  }
  __syncthreads();

  float acc[R][BMAX];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b) acc[r][b] = 0.f;

  for (int64_t k0 = 0; k0 < K; k0 += (int64_t)kDgChunk * SEG) {
    if (XB || k0 > 0) load_pass(k0);
#pragma unroll
    for (int j = 0; j < SEG; ++j) {
      const int64_t col = k0 + (int64_t)kDgChunk * j + 8 * lane;
      if (col >= K) continue;
#pragma unroll
      for (int b = 0; b < BMAX; ++b) {
        if (b >= B) break;
        float xv[8];
        if constexpr (XB) {
          const u32x4 h = *reinterpret_cast<const u32x4*>(xh + (int64_t)b * K + col);
          const uint32_t hv[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            xv[2 * t] = __uint_as_float(hv[t] << 16);
            xv[2 * t + 1] = __uint_as_float(hv[t] & 0xFFFF0000u);
          }
        } else {
          const u32x4 x0 = *reinterpret_cast<const u32x4*>(xs + (int64_t)b * K + col);
          const u32x4 x1 = *reinterpret_cast<const u32x4*>(xs + (int64_t)b * K + col + 4);
          xv[0] = __uint_as_float(x0.x); xv[1] = __uint_as_float(x0.y);
          xv[2] = __uint_as_float(x0.z); xv[3] = __uint_as_float(x0.w);
          xv[4] = __uint_as_float(x1.x); xv[5] = __uint_as_float(x1.y);
          xv[6] = __uint_as_float(x1.z); xv[7] = __uint_as_float(x1.w);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const uint32_t wa[4] = {wv[r][j].x, wv[r][j].y, wv[r][j].z, wv[r][j].w};
          float a = acc[r][b];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            a = __builtin_fmaf(half_lo(wa[t]), xv[2 * t], a);
            a = __builtin_fmaf(half_hi(wa[t]), xv[2 * t + 1], a);
          }
          acc[r][b] = a;
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b) acc[r][b] = wave_sum_f32(acc[r][b]);
  // lane r * BMAX + b stores row r, batch row b
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b)
      if (lane == r * BMAX + b && b < B && row0 + r < N) {
        float* o = ym + (int64_t)b * N + row0 + r;
        *o = accum ? *o + acc[r][b] : acc[r][b];
      }
}

template <int BMAX, bool RMS>
static hipError_t launch_dgemv_b(const uint16_t* x, const uint16_t* W, int count, int B,
                                 int64_t N, int64_t K, float* y, hipStream_t stream,
                                 const float* xr, const float* nw, float eps, int accum) {
  const size_t lds = ((size_t)B * K * (BMAX > 1 ? 2 : 4) + 15) / 16 * 16 + (RMS ? 16 * 4 : 0);
  // four rows per wave, or two when the launch has few rows per CU or (one
  // batch row) the rows are long: K > 2048 takes a row in one pass, 8
  // pieces per lane
  const int64_t blocks4 = (N + 4 * kDgWaves - 1) / (4 * kDgWaves) * count;
  if (blocks4 >= 2 * (int64_t)current_cu_count() && (BMAX > 1 || K <= 4 * kDgChunk)) {
    const dim3 grid((unsigned)((N + 4 * kDgWaves - 1) / (4 * kDgWaves)), (unsigned)count);
    hipLaunchKernelGGL((dgemv_kernel<BMAX, 4, 4, RMS>), grid, dim3(64 * kDgWaves), lds, stream, x,
                       W, B, N, K, y, xr, nw, eps, accum);
  } else {
    const dim3 grid((unsigned)((N + 2 * kDgWaves - 1) / (2 * kDgWaves)), (unsigned)count);
    hipLaunchKernelGGL((dgemv_kernel<BMAX, 2, 8, RMS>), grid, dim3(64 * kDgWaves), lds, stream, x,
                       W, B, N, K, y, xr, nw, eps, accum);
  }
  return hipGetLastError();
}

template <bool RMS>
static hipError_t launch_dgemv_any(const uint16_t* x, const uint16_t* W16, int count, int B,
                                   int64_t N, int64_t K, float* y, hipStream_t stream,
                                   const float* xr, const float* nw, float eps, int accum) {
  if (B <= 1) return launch_dgemv_b<1, RMS>(x, W16, count, B, N, K, y, stream, xr, nw, eps, accum);
  if (B <= 2) return launch_dgemv_b<2, RMS>(x, W16, count, B, N, K, y, stream, xr, nw, eps, accum);
  if (B <= 4) return launch_dgemv_b<4, RMS>(x, W16, count, B, N, K, y, stream, xr, nw, eps, accum);
  return launch_dgemv_b<8, RMS>(x, W16, count, B, N, K, y, stream, xr, nw, eps, accum);
}

hipError_t launch_dgemv(const uint16_t* x, const uint16_t* W16, int count, int B, int64_t N,
                        int64_t K, float* y, hipStream_t stream) {
  return launch_dgemv_any<false>(x, W16, count, B, N, K, y, stream, nullptr, nullptr, 0.f, 0);
}

hipError_t launch_dgemv_rms(const float* src, const float* nw, float eps, const uint16_t* W16,
                            int B, int64_t N, int64_t K, float* y, int accum,
                            hipStream_t stream) {
  return launch_dgemv_any<true>(nullptr, W16, 1, B, N, K, y, stream, src, nw, eps, accum);
}

}  // namespace tmk
