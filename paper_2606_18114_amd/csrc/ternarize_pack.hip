// Grouped-absmean ternarizer (paper Sec. 3.1) with 2-bit packing (Sec. 8)
// and the zero-code count (Sec. 3.1, Table 1), in one pass over W.
//
// A wave reads 1024 consecutive weights per iteration as four fully
// coalesced 1 KiB loads; each lane holds 4 weights of a load, so a group of g
// weights sits on g/4 adjacent lanes (two loads for g = 512) and its sum of
// |w| is a float64 butterfly over those lanes.  With the sum in float64 the
// mean rounds once to float32, which is what the float64 oracle produces.
// Four adjacent lanes OR their codes into one packed 32-bit word.  The grid
// is persistent and each workgroup adds its zero count to the output once.
//
// Code decision, identical to the float32 expression
//   q = round_half_even(clip(fl32(w / fl32(s + eps)), -1, 1)):
// the float32 quotient rounds to at most 1/2 exactly when the real quotient
// is at most 1/2 + 2^-25 (the midpoint between 1/2 and the next float32 is a
// tie and goes to the even 1/2), and half-to-even rounding sends 1/2 to 0.
// So q != 0  <=>  |w| > d * (1/2 + 2^-25),  d = fl32(s + eps).  The product
// of a 24-bit and a 25-bit significand is exact in float64, so the test is a
// single exact float64 compare per weight and no division is needed.
#include "common.hpp"

namespace tmk {

__global__ void zero_u64_kernel(unsigned long long* p) { *p = 0ull; }

constexpr int kTernUnit = 1024;  // weights per wave iteration (4 loads x 64 lanes x 4)
constexpr int kTernWaves = 16;   // waves per workgroup

// row_mult (optional, [N]): the code of row n divides by fl32(row_mult[n] * s)
// + eps instead of s + eps (the appendix's asymmetric gate thresholds); the
// stored scale is the absmean either way.
// tau_in (optional, [N, K/g]): the caller's per-group thresholds replace the
// absmean (a learned scale, Sec. 4); no scales are written then.
template <int G>
__global__ __launch_bounds__(64 * kTernWaves) void ternarize_pack_kernel(
    const float* __restrict__ W, int64_t total, int64_t K, float eps,
    const float* __restrict__ row_mult, const float* __restrict__ tau_in,
    uint32_t* __restrict__ codes,
    float* __restrict__ scales, uint16_t* __restrict__ scales_f16,
    unsigned long long* __restrict__ zero_count) {
  constexpr int L = G / 4 < 64 ? G / 4 : 64;  // lanes holding one group within a load
  __shared__ uint32_t wave_zeros[kTernWaves];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t nunits = (total + kTernUnit - 1) / kTernUnit;
  uint32_t zeros = 0;

  for (int64_t u = (int64_t)blockIdx.x * kTernWaves + wave; u < nunits;
       u += (int64_t)gridDim.x * kTernWaves) {
    const int64_t base = u * kTernUnit;
    // load i covers weights [base + 256 i, base + 256 i + 256); lane l holds 4 of them
    float w[4][4];
    bool ok[4];
    double ps[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t off = base + 256 * i + 4 * lane;
      ok[i] = off < total;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (ok[i]) v = ld16(W + off);
      // __uint_as_float, not __builtin_bit_cast: this compiler reads every
      // element of a vector as its first one when bit-casting v.y, v.z, v.w
      w[i][0] = __uint_as_float(v.x);
      w[i][1] = __uint_as_float(v.y);
      w[i][2] = __uint_as_float(v.z);
      w[i][3] = __uint_as_float(v.w);
      ps[i] = ((double)fabsf(w[i][0]) + (double)fabsf(w[i][1])) +
              ((double)fabsf(w[i][2]) + (double)fabsf(w[i][3]));
    }
    // group sums: butterfly over the L lanes of each group (float64, exact)
#pragma unroll
    for (int i = 0; i < 4; ++i) ps[i] = group_sum_f64<L>(ps[i]);
    if constexpr (G == 512) {  // a group spans two loads
      ps[0] += ps[1];
      ps[1] = ps[0];
      ps[2] += ps[3];
      ps[3] = ps[2];
    }

#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float sc = (float)(ps[i] / (double)G);
      if (tau_in) sc = tau_in[(ok[i] ? base + 256 * i + 4 * lane : 0) / G];  // uniform branch
      float tau = sc;
      if (row_mult) {  // (uniform branch) the threshold of this element's row
        const int64_t off = base + 256 * i + 4 * lane;
        const int64_t row = (ok[i] ? off : 0) / K;
        tau = __fmul_rn(row_mult[row], sc);  // rounded on its own: no fused m * s + eps
      }
      const float d = __fadd_rn(tau, eps);
      const double thr = (double)d * (0.5 + 0x1p-25);
      uint32_t part = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int e = 4 * (lane & 3) + j;  // element within its 16-weight word
        const bool nz = (double)fabsf(w[i][j]) > thr;
        const uint32_t code = nz ? ((__float_as_uint(w[i][j]) >> 31) ? 3u : 1u) : 0u;
        part |= code << (2 * (e / 2) + 16 * (e % 2));
        zeros += (nz || !ok[i]) ? 0u : 1u;
      }
      part |= lane_xchg<1>(part);
      part |= lane_xchg<2>(part);
      const int64_t off = base + 256 * i + 4 * lane;
      if (ok[i] && (lane & 3) == 0) codes[off / 16] = part;
      if (!tau_in && ok[i] && (lane % L) == 0 && (G != 512 || (i & 1) == 0)) {
        const int64_t grp = off / G;
        scales[grp] = sc;
        if (scales_f16) scales_f16[grp] = __builtin_bit_cast(uint16_t, (_Float16)sc);
      }
    }
  }

  if (zero_count) {
    uint32_t z = zeros;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o, 64);
    if (lane == 0) wave_zeros[wave] = z;
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long t = 0;
#pragma unroll
      for (int i = 0; i < kTernWaves; ++i) t += wave_zeros[i];
      if (t) atomicAdd(zero_count, t);
    }
  }
}

hipError_t launch_ternarize_pack(const float* W, int64_t N, int64_t K, int g, float eps,
                                 const float* row_mult, const float* tau_in, uint8_t* codes,
                                 float* scales,
                                 uint16_t* scales_f16, uint64_t* zero_count,
                                 hipStream_t stream) {
  const int64_t total = N * K;
  auto* zc = reinterpret_cast<unsigned long long*>(zero_count);
  if (zc) {
    // a fill kernel rather than a memset node, so the call can be captured
    hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(1), 0, stream, zc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // a persistent grid: at most 512 workgroups, each adding its zero count once
  int64_t blocks = (total / kTernUnit + kTernWaves) / kTernWaves;
  if (blocks > 512) blocks = 512;
  const dim3 grid((unsigned)blocks), block(64 * kTernWaves);
  auto* cw = reinterpret_cast<uint32_t*>(codes);
  switch (g) {
    case 32:  hipLaunchKernelGGL(ternarize_pack_kernel<32>, grid, block, 0, stream, W, total, K, eps, row_mult, tau_in, cw, scales, scales_f16, zc); break;
    case 64:  hipLaunchKernelGGL(ternarize_pack_kernel<64>, grid, block, 0, stream, W, total, K, eps, row_mult, tau_in, cw, scales, scales_f16, zc); break;
    case 128: hipLaunchKernelGGL(ternarize_pack_kernel<128>, grid, block, 0, stream, W, total, K, eps, row_mult, tau_in, cw, scales, scales_f16, zc); break;
    case 256: hipLaunchKernelGGL(ternarize_pack_kernel<256>, grid, block, 0, stream, W, total, K, eps, row_mult, tau_in, cw, scales, scales_f16, zc); break;
    case 512: hipLaunchKernelGGL(ternarize_pack_kernel<512>, grid, block, 0, stream, W, total, K, eps, row_mult, tau_in, cw, scales, scales_f16, zc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
