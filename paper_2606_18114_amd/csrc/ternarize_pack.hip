// Grouped-absmean ternarizer (paper Sec. 3.1) with 2-bit packing (Sec. 8)
// and the zero-code count (Sec. 3.1, Table 1), in one pass over W.
//
// A wave takes 1024 consecutive weights per iteration and each lane owns 16
// consecutive ones: the 16 codes of one packed 32-bit word, all in one group
// (g >= 32) and one row (K % 16 == 0).  The lane reads its 64 bytes as four
// 16-byte loads (together the wave's loads cover 4 KiB), sums |w| in float64,
// and a butterfly over the g/16 lanes of the group completes the group sum.
// With the sum in float64 the mean rounds once to float32, which is what the
// float64 oracle produces.  The lane then decides its 16 codes, stores its
// word and counts its zeros with one popcount; the grid is persistent and
// each workgroup adds its zero count to the output once.
//
// Code decision, identical to the float32 expression
//   q = round_half_even(clip(fl32(w / fl32(s + eps)), -1, 1)):
// the float32 quotient rounds to at most 1/2 exactly when the real quotient
// is at most 1/2 + 2^-25 (the midpoint between 1/2 and the next float32 is a
// tie and goes to the even 1/2), and half-to-even rounding sends 1/2 to 0.
// So q != 0  <=>  |w| > d * (1/2 + 2^-25),  d = fl32(s + eps) >= 0.  For d in
// [2^e, 2^(e+1)) the excess d * 2^-25 lies in [u/2, u), u = 2^(e-24) the
// spacing of float32 values at d/2, so no float32 lies strictly between d/2
// and the threshold: for a float32 |w| the test is  |w| > d/2  (d/2 exact),
// and  |w| > RZ(d/2)  when d/2 falls below the normal range (RZ: rounded
// toward zero).  One float32 compare per weight, no division.
#include "common.hpp"

namespace tmk {

__global__ void zero_u64_kernel(unsigned long long* p) { *p = 0ull; }

constexpr int kTernUnit = 1024;  // weights per wave iteration: 16 per lane
constexpr int kTernWaves = 16;  // waves per workgroup

// row_mult (optional, [N]): the code of row n divides by fl32(row_mult[n] * s)
// + eps instead of s + eps (the appendix's asymmetric gate thresholds); the
// stored scale is the absmean either way.
// tau_in (optional, [N, K/g]): the caller's per-group thresholds replace the
// absmean (a learned scale, Sec. 4); no scales are written then.
// MODE: 0 absmean, 1 absmean with row_mult, 2 tau_in (separate instances, so
// the plain pass carries no registers for the other two)
template <int G, int MODE>
__global__ __launch_bounds__(64 * kTernWaves) void ternarize_pack_kernel(
    const float* __restrict__ W, int64_t total, int64_t K, float eps,
    const float* __restrict__ row_mult, const float* __restrict__ tau_in,
    uint32_t* __restrict__ codes,
    float* __restrict__ scales, uint16_t* __restrict__ scales_f16,
    unsigned long long* __restrict__ zero_count) {
  constexpr int L = G / 16;  // lanes holding one group
  static_assert(L >= 2 && L <= 32, "16 weights per lane, groups of 32 .. 512");
  __shared__ uint32_t wave_zeros[kTernWaves];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t nunits = (total + kTernUnit - 1) / kTernUnit;
  uint32_t zeros = 0;

  for (int64_t u = (int64_t)blockIdx.x * kTernWaves + wave; u < nunits;
       u += (int64_t)gridDim.x * kTernWaves) {
    // The unit's base is wave-uniform; offsets inside it are 32-bit.  The
    // lane offset is made opaque per unit so that the compiler does not hoist
    // every derived address out of the loop (registers held for the whole
    // kernel would cost waves per SIMD).
    const int64_t base = u * kTernUnit;
    const int64_t rem = total - base;
    const int lim = rem < kTernUnit ? (int)rem : kTernUnit;  // valid weights in the unit
    int lo = 16 * lane;
    asm volatile("" : "+v"(lo));
    const bool ok = lo < lim;  // total % 16 == 0: a lane's 16 weights are all valid or none
    const float* Wl = W + base + lo;
    u32x4 v[4] = {};
    if (ok) {
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = ld16(Wl + 4 * i);
    }
    // __uint_as_float, not __builtin_bit_cast: this compiler reads every
    // element of a vector as its first one when bit-casting v.y, v.z, v.w
    float w[16];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      w[4 * i + 0] = __uint_as_float(v[i].x);
      w[4 * i + 1] = __uint_as_float(v[i].y);
      w[4 * i + 2] = __uint_as_float(v[i].z);
      w[4 * i + 3] = __uint_as_float(v[i].w);
    }
    double ps = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      ps += ((double)fabsf(w[4 * i]) + (double)fabsf(w[4 * i + 1])) +
            ((double)fabsf(w[4 * i + 2]) + (double)fabsf(w[4 * i + 3]));
    ps = group_sum_f64<L>(ps);  // float64, exact

    float sc = (float)(ps / (double)G);
    if constexpr (MODE == 2) sc = tau_in[(base + (ok ? lo : 0)) / G];
    float tau = sc;
    if constexpr (MODE == 1) {  // the threshold of this lane's row
      const int64_t row = (base + (ok ? lo : 0)) / K;
      tau = __fmul_rn(row_mult[row], sc);  // rounded on its own: no fused m * s + eps
    }
    const float d = __fadd_rn(tau, eps);
    // d / 2 rounded toward zero, exactly: a plain halving when d is normal
    // above 2^-125 (or inf, NaN), a truncating shift of the bits below
    const uint32_t db = __float_as_uint(d);
    const float thr = (db >> 23) >= 2u ? d * 0.5f : __uint_as_float(db >> 1);
    // element j of the word: bits 2j (j even) or 16 + 2(j - 1)/2 (j odd);
    // codes 01 = +1, 11 = -1
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t b = __float_as_uint(w[j]);
      const uint32_t code = fabsf(w[j]) > thr ? (((b >> 30) & 2u) | 1u) : 0u;
      word |= code << (2 * (j / 2) + 16 * (j % 2));
    }
    if (ok) {
      codes[(base + lo) / 16] = word;
      zeros += 16u - (uint32_t)__popc((word | (word >> 1)) & 0x55555555u);
      if (MODE != 2 && (lane % L) == 0) {
        const int64_t grp = (base + lo) / G;
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
  const int mode = tau_in ? 2 : (row_mult ? 1 : 0);
#define TM_TERN_CASE(GG, MM)                                                            \
  hipLaunchKernelGGL((ternarize_pack_kernel<GG, MM>), grid, block, 0, stream, W, total, K, \
                     eps, row_mult, tau_in, cw, scales, scales_f16, zc)
#define TM_TERN_G(GG)                  \
  case GG:                             \
    if (mode == 0)                     \
      TM_TERN_CASE(GG, 0);             \
    else if (mode == 1)                \
      TM_TERN_CASE(GG, 1);             \
    else                               \
      TM_TERN_CASE(GG, 2);             \
    break;
  switch (g) {
    TM_TERN_G(32)
    TM_TERN_G(64)
    TM_TERN_G(128)
    TM_TERN_G(256)
    TM_TERN_G(512)
    default: return hipErrorInvalidValue;
  }
#undef TM_TERN_G
#undef TM_TERN_CASE
  return hipGetLastError();
}

}  // namespace tmk
