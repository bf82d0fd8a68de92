// Grouped-absmean ternarizer (paper Sec. 3.1) with 2-bit packing (Sec. 8)
// and the zero-code count (Sec. 3.1, Table 1), in one pass over W.
//
// One thread owns 16 consecutive weights of a row, i.e. one packed word.
// The g/16 threads of a group are adjacent lanes of one wave, so the group's
// sum of |w| is a float64 butterfly over those lanes.  With the sum in
// float64 the mean rounds once to float32, which is what the float64 oracle
// produces as well.
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

template <int G>
__global__ __launch_bounds__(256) void ternarize_pack_kernel(
    const float* __restrict__ W, int64_t n_words, float eps,
    uint32_t* __restrict__ codes, float* __restrict__ scales,
    uint16_t* __restrict__ scales_f16, unsigned long long* __restrict__ zero_count) {
  constexpr int kLanesPerGroup = G / 16;
  const int64_t word = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool live = word < n_words;

  float w[16];
  if (live) {
    const float* src = W + word * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // __uint_as_float, not __builtin_bit_cast: this compiler reads every
      // element of a vector as its first one when bit-casting v.y, v.z, v.w
      const u32x4 v = ld16(src + 4 * i);
      w[4 * i + 0] = __uint_as_float(v.x);
      w[4 * i + 1] = __uint_as_float(v.y);
      w[4 * i + 2] = __uint_as_float(v.z);
      w[4 * i + 3] = __uint_as_float(v.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = 0.0f;
  }

  double sum = 0.0;
#pragma unroll
  for (int i = 0; i < 16; ++i) sum += (double)fabsf(w[i]);
#pragma unroll
  for (int off = 1; off < kLanesPerGroup; off <<= 1) sum += __shfl_xor(sum, off, 64);

  const float s = (float)(sum / (double)G);
  const float d = s + eps;
  const double thr = (double)d * (0.5 + 0x1p-25);

  uint32_t packed = 0;
  int zeros = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const uint32_t bits = __float_as_uint(w[e]);
    const bool nz = (double)fabsf(w[e]) > thr;
    const uint32_t code = nz ? ((bits >> 31) ? 3u : 1u) : 0u;
    packed |= code << (2 * (e / 2) + 16 * (e % 2));
    zeros += nz ? 0 : 1;
  }

  if (live) {
    codes[word] = packed;
    if ((word % kLanesPerGroup) == 0) {
      const int64_t grp = word / kLanesPerGroup;
      scales[grp] = s;
      if (scales_f16) scales_f16[grp] = __builtin_bit_cast(uint16_t, (_Float16)s);
    }
  } else {
    zeros = 0;
  }

  if (zero_count) {
    // wave-wide sum, one 64-bit atomic per wave
    int z = zeros;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) z += __shfl_xor(z, off, 64);
    if ((threadIdx.x & 63) == 0 && z) atomicAdd(zero_count, (unsigned long long)z);
  }
}

hipError_t launch_ternarize_pack(const float* W, int64_t N, int64_t K, int g, float eps,
                                 uint8_t* codes, float* scales, uint16_t* scales_f16,
                                 uint64_t* zero_count, hipStream_t stream) {
  const int64_t n_words = N * (K / 16);
  auto* zc = reinterpret_cast<unsigned long long*>(zero_count);
  if (zc) {
    // a fill kernel rather than a memset node, so the call can be captured
    hipLaunchKernelGGL(zero_u64_kernel, dim3(1), dim3(1), 0, stream, zc);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)((n_words + 255) / 256)), block(256);
  auto* cw = reinterpret_cast<uint32_t*>(codes);
  switch (g) {
    case 32:  hipLaunchKernelGGL(ternarize_pack_kernel<32>, grid, block, 0, stream, W, n_words, eps, cw, scales, scales_f16, zc); break;
    case 64:  hipLaunchKernelGGL(ternarize_pack_kernel<64>, grid, block, 0, stream, W, n_words, eps, cw, scales, scales_f16, zc); break;
    case 128: hipLaunchKernelGGL(ternarize_pack_kernel<128>, grid, block, 0, stream, W, n_words, eps, cw, scales, scales_f16, zc); break;
    case 256: hipLaunchKernelGGL(ternarize_pack_kernel<256>, grid, block, 0, stream, W, n_words, eps, cw, scales, scales_f16, zc); break;
    case 512: hipLaunchKernelGGL(ternarize_pack_kernel<512>, grid, block, 0, stream, W, n_words, eps, cw, scales, scales_f16, zc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
