// Decode-time ternary GEMV (batch B <= 16), strided-batched over matrices.
//
// Batch-1 decoding is bound by the weight bytes (paper Sec. 8), so the
// kernel streams the packed codes once from HBM and lets the matrix cores do
// the multiply-adds: one v_mfma_f32_32x32x16_bf16 takes the activations x as
// the A operand (rows = batch, padded to 32 with zeros) and 32 weight rows,
// decoded to exact bfloat16 2*q, as the B operand.  Decoding is one shift
// and one AND per two codes (common.hpp).  The decode of MFMA step t+1 is
// issued before the MFMA of step t into its own registers: when the vector
// ALU instead rewrites the registers an in-flight MFMA still reads, the two
// units serialize and the GEMV runs at half speed.
//
// Work split: each wave owns 32 consecutive weight rows of one matrix and
// walks the whole K range, so no cross-wave reduction is needed; a workgroup
// of 4 waves covers 128 rows and first copies x of its matrix into LDS.
// K is walked in chunks of C = min(g, 128) columns; within a chunk each half
// of the wave (lanes 0-31, 32-63) owns C/2 contiguous columns of its row, so
// a lane fetches its codes with one 16-byte load per chunk (g >= 128), and
// MFMA step t takes octet t of both halves' ranges: every step stays inside
// one quantization group and the float16 scale is applied per chunk in
// float32 (acc += s * sum_t mfma, y = acc / 2).  Code and scale loads run
// kGemvPf chunks ahead of the arithmetic through a register ring.
#include "common.hpp"

namespace tmk {

constexpr int kGemvWaves = 4;
constexpr int kGemvRows = 32 * kGemvWaves;  // rows per workgroup (32 per wave)
constexpr int kGemvPf = 8;                  // chunks of codes in flight per wave
constexpr int kGemvXBytes = 64 * 1024;      // LDS budget for x

template <int G, int NV>
__global__ __launch_bounds__(64 * kGemvWaves) void tgemv_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales_f16, int B, int64_t N, int64_t K, int64_t KP,
    float* __restrict__ y) {
  constexpr int C = G < 128 ? G : 128;  // chunk width
  constexpr int SPC = C / 16;           // MFMA steps per chunk
  constexpr int WPL = C / 32;           // code words a lane holds per chunk
  // NV: accumulator entries that can hold a batch row (4 when B <= 4)
  extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [B][KP] + zero pad

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int64_t mat = blockIdx.y;
  const int64_t kw = K / 16;
  const int64_t ng = K / G;

  int64_t n = (int64_t)blockIdx.x * kGemvRows + wave * 32 + l32;
  const bool nrow_ok = n < N;
  n = nrow_ok ? n : N - 1;
  const uint32_t* crow = reinterpret_cast<const uint32_t*>(codes) + (mat * N + n) * kw;
  const uint16_t* srow = scales_f16 + (mat * N + n) * ng;
  const uint16_t* xm = x + mat * (int64_t)B * K;
  const int zpad = B * (int)KP;  // element offset of the zero pad in xs
  // lanes whose batch row b = l32 exists read x; the others read the zero pad
  const bool xl = l32 < B;
  const int xbase = xl ? l32 * (int)KP + h * (C / 2) : zpad;
  const uint32_t kmask = xl ? 0xFFFFFFFFu : 0u;

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;

  for (int64_t kp0 = 0; kp0 < K; kp0 += KP) {
    const int kpl = (int)(K - kp0 < KP ? K - kp0 : KP);
    // ---- stage x[:, kp0 : kp0 + kpl] and the zero pad ----
    __syncthreads();
    for (int i = threadIdx.x; i < B * kpl / 8; i += 64 * kGemvWaves) {
      const int b = i / (kpl / 8), c8 = i % (kpl / 8);
      st16(&xs[b * (int)KP + 8 * c8], ld16(xm + (int64_t)b * K + kp0 + 8 * c8));
    }
    for (int i = threadIdx.x; i < C / 8; i += 64 * kGemvWaves)
      st16(&xs[zpad + 8 * i], u32x4{0u, 0u, 0u, 0u});
    __syncthreads();

    const int nch = kpl / C;
    // ---- code / scale ring, kGemvPf chunks ahead ----
    uint32_t cr[kGemvPf][WPL];
    uint16_t sr[kGemvPf];
    auto fetch = [&](int slot, int c) {
      const int cc = c < nch ? c : nch - 1;  // past the end: re-read the last chunk
      const int64_t k0 = kp0 + (int64_t)cc * C;
      const uint32_t* p = crow + k0 / 16 + h * WPL;
      if constexpr (WPL == 4) {
        const u32x4 v = ld16(p);
        cr[slot][0] = v.x;
        cr[slot][1 % WPL] = v.y;
        cr[slot][2 % WPL] = v.z;
        cr[slot][3 % WPL] = v.w;
      } else if constexpr (WPL == 2) {
        const u32x2 v = *reinterpret_cast<const u32x2*>(p);
        cr[slot][0] = v.x;
        cr[slot][1 % WPL] = v.y;
      } else {
        cr[slot][0] = *p;
      }
      sr[slot] = srow[k0 / G];
    };
    auto decode = [&](int slot, int t) {
      const uint32_t w = cr[slot][t / 2];
      return (t & 1) ? decode_half<1>(w) : decode_half<0>(w);
    };
    // Two partial-sum buffers alternate between chunks: the scale of chunk
    // c - 1 is applied after the MFMAs of chunk c are issued, so the vector
    // ALUs never wait for the MFMA chain they just started.
    f32x16 pb[2];
    float spend = 0.f;  // scale of the chunk whose partial sums are pending
    int pend = -1;      // buffer holding them (-1: none)
    auto retire = [&](int buf) {
#pragma unroll
      for (int i = 0; i < NV; ++i) acc[i] += spend * pb[buf][i];
    };
    // one chunk: x fragments first, then MFMA t while step t + 1 decodes
    auto chunk = [&](int slot, int c, int buf) {
      const uint32_t kb = (uint32_t)(c * C) & kmask;
      u32x4 xf[SPC];
#pragma unroll
      for (int t = 0; t < SPC; ++t)
        xf[t] = *reinterpret_cast<const u32x4*>(&xs[xbase + kb + 8 * t]);
#pragma unroll
      for (int i = 0; i < 16; ++i) pb[buf][i] = 0.f;
      bf16x8 bcur = decode(slot, 0);
#pragma unroll
      for (int t = 0; t < SPC; ++t) {
        const bf16x8 bnext = decode(slot, t + 1 < SPC ? t + 1 : t);
        pb[buf] = mfma32(as_bf16x8(xf[t]), bcur, pb[buf]);
        bcur = bnext;
      }
      if (pend >= 0) retire(buf ^ 1);
      spend = (float)__builtin_bit_cast(_Float16, sr[slot]);
      pend = buf;
    };
#pragma unroll
    for (int s = 0; s < kGemvPf; ++s) fetch(s, s);

    // steady state: whole ring periods, no branches inside
    int c0 = 0;
    for (; c0 + kGemvPf <= nch; c0 += kGemvPf) {
#pragma unroll
      for (int s = 0; s < kGemvPf; ++s) {
        chunk(s, c0 + s, s & 1);
        fetch(s, c0 + s + kGemvPf);
      }
    }
    // tail: fewer than kGemvPf chunks left, already in the ring
#pragma unroll
    for (int s = 0; s < kGemvPf; ++s)
      if (c0 + s < nch) chunk(s, c0 + s, s & 1);
    if (pend >= 0) retire(pend);
  }

  // lane holds column n and batch rows b = 8*(i/4) + 4*h + i%4
  if (nrow_ok) {
    float* ym = y + mat * (int64_t)B * N;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int b = 8 * (i / 4) + 4 * h + (i % 4);
      if (b < B) ym[(int64_t)b * N + n] = 0.5f * acc[i];
    }
  }
}

template <int G>
static void launch_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                     int B, int64_t N, int64_t K, float* y, hipStream_t stream) {
  constexpr int C = G < 128 ? G : 128;
  // x part staged in LDS: B * KP bf16 plus a C-wide zero pad, within 64 KiB
  int64_t KP = ((kGemvXBytes / 2 - C) / B) / C * C;
  if (KP > K) KP = K;
  const size_t lds = (size_t)(B * KP + C) * 2;
  const dim3 grid((unsigned)((N + kGemvRows - 1) / kGemvRows), (unsigned)count);
  const dim3 block(64 * kGemvWaves);
  if (B > 4)
    hipLaunchKernelGGL((tgemv_kernel<G, 16>), grid, block, lds, stream, x, codes, s16, B, N, K, KP, y);
  else
    hipLaunchKernelGGL((tgemv_kernel<G, 4>), grid, block, lds, stream, x, codes, s16, B, N, K, KP, y);
}

hipError_t launch_tgemv(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                        int B, int64_t N, int64_t K, int g, float* y, hipStream_t stream) {
  switch (g) {
    case 32:  launch_g<32>(x, codes, s16, count, B, N, K, y, stream); break;
    case 64:  launch_g<64>(x, codes, s16, count, B, N, K, y, stream); break;
    case 128: launch_g<128>(x, codes, s16, count, B, N, K, y, stream); break;
    case 256: launch_g<256>(x, codes, s16, count, B, N, K, y, stream); break;
    case 512: launch_g<512>(x, codes, s16, count, B, N, K, y, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
