// Decode-time ternary GEMV (batch B <= 16), strided-batched over matrices.
//
// Batch-1 decoding is bound by the weight bytes (paper Sec. 8).  The kernel
// streams the packed codes once, with every load instruction reading whole
// 128-byte lines, and lets the matrix cores do the multiply-adds: one
// v_mfma_f32_16x16x32_bf16 takes the activations x as the A operand (rows =
// batch, padded to 16 with zeros) and 16 weight rows, decoded to exact
// bfloat16 2*q, as the B operand.  Decoding is one shift and one AND per two
// codes (common.hpp).
//
// Work split: each wave owns 32 consecutive weight rows (two 16-row blocks)
// of one matrix and walks the whole K range; a workgroup of 4 waves covers
// 128 rows and first copies x of its matrix into LDS.
//
// Loads: the codes of a wave's 32 rows are staged through a wave-private,
// 2-deep LDS ring in slots of 512 columns (128 bytes per row), filled by
// direct-to-LDS loads (global_load_lds) that each read 8 whole rows' 128-byte
// pieces.  The eight 16-byte units of a row piece are stored XOR-permuted by
// gemv_swz(row), so the MFMA operand reads below are bank-conflict free.  The
// float16 group scales of the slot ride along (one 2-byte load per lane; the
// hardware writes each lane's value into its own 4-byte LDS word).  The loads
// are issued from inline assembly, so the compiler neither tracks them nor
// waits for them; each wave counts its own and waits with s_waitcnt before
// reading a slot.  No workgroup barrier is needed for the ring.
//
// Compute: K is walked in chunks of C = min(g, 128) columns, so a chunk lies
// inside one quantization group and its scale is applied in float32 once per
// chunk (acc += s * partial, y = acc / 2).  Inside a chunk the four 8-column
// lane groups of the MFMA take their codes as below, so that a lane reads 4
// or 8 contiguous bytes of its row per chunk and decodes them with shifts
// known at compile time:
//   C = 128: step t, lane group q -> word 2q + t/2, half t%2
//   C =  64: step t, lane group q -> word q, half t
//   C =  32: step 0, lane group q -> word q/2, half q%2
// (word = 16 codes, half = 8 of them); x is read from LDS with the same
// mapping.
#include <type_traits>

#include "common.hpp"

namespace tmk {

constexpr int kGemvWaves = 4;
constexpr int kGemvBlocks = 2;                             // 16-row MFMA blocks per wave
constexpr int kGemvWaveRows = 16 * kGemvBlocks;            // 32
constexpr int kGemvRows = kGemvWaveRows * kGemvWaves;      // rows per workgroup
constexpr int kGemvSlotK = 512;                            // columns per ring slot
constexpr int kGemvSlotCodes = kGemvWaveRows * kGemvSlotK / 4;  // 4 KiB per slot
constexpr int kGemvXBytes = 32 * 1024;                     // LDS budget for x

// scales per row per slot and their direct-to-LDS loads per slot
template <int G>
struct GemvCfg {
  static constexpr int kNs = kGemvSlotK / G > 1 ? kGemvSlotK / G : 1;
  static constexpr int kSLoads = (kGemvWaveRows * kNs + 63) / 64;
  static constexpr int kSlotScales = 256 * kSLoads;  // LDS bytes (4 per value)
  static constexpr int kSlotBytes = kGemvSlotCodes + kSlotScales;
  static constexpr int kWaveBytes = 2 * kSlotBytes;
  static constexpr int kLoads = 4 + kSLoads;  // direct-to-LDS loads per slot
};

// calls f(integral_constant<int, I>) for I in [I0, N), fully unrolled
template <int I, int N, typename F>
__device__ __forceinline__ void gemv_static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    gemv_static_for<I + 1, N>(f);
  }
}

__device__ __forceinline__ int gemv_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// lane i: 16 (2) bytes at base + voff -> LDS lds_base + 16 i (4 i, zero-extended)
__device__ __forceinline__ void gemv_dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
__device__ __forceinline__ void gemv_dma2(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_ushort %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int G>
__global__ __launch_bounds__(64 * kGemvWaves) void tgemv_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales_f16, int B, int64_t N, int64_t K, int64_t KP,
    float* __restrict__ y) {
  using Cfg = GemvCfg<G>;
  constexpr int C = G < 128 ? G : 128;   // chunk width
  constexpr int SPC = C / 32;            // MFMA steps per chunk
  constexpr int CPS = kGemvSlotK / C;    // chunks per slot
  constexpr int NB = kGemvBlocks;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  // [waves][2 slots][codes 4 KiB | scales], then x [B][KP] + zero pad

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15;
  const int q = lane >> 4;  // lane group: the MFMA's 8-column k slice
  const int64_t mat = blockIdx.y;
  const int64_t kb = K / 4;  // code bytes per row
  const int64_t ng = K / G;
  const int nslot = (int)((K + kGemvSlotK - 1) / kGemvSlotK);
  const int64_t row0 = (int64_t)blockIdx.x * kGemvRows + wave * kGemvWaveRows;  // wave's rows
  const uint32_t wlds = (uint32_t)(uintptr_t)smem + wave * Cfg::kWaveBytes;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + kGemvWaves * Cfg::kWaveBytes);

  // ---- load plan of one slot (uniform base + per-lane offsets) ----
  // codes: load j covers wave rows 8j .. 8j+7, lane -> row 8j + lane/8, unit
  // lane%8 of the LDS row, which holds logical unit (lane%8) ^ gemv_swz(row)
  const uint8_t* cbase = codes + (mat * N) * kb;
  uint32_t coff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = 8 * j + (lane >> 3);
    int64_t n = row0 + r;
    n = n < N ? n : N - 1;
    coff[j] = (uint32_t)(n * kb) + 16u * ((lane & 7) ^ gemv_swz(r));
  }
  // scales: load m, lane -> value 64m + lane = (row v / kNs, group v % kNs)
  const uint16_t* sbase = scales_f16 + (mat * N) * ng;
  int64_t srow[Cfg::kSLoads];
  int sgrp[Cfg::kSLoads];
#pragma unroll
  for (int m = 0; m < Cfg::kSLoads; ++m) {
    const int v = 64 * m + lane;
    const int r = (v / Cfg::kNs) % kGemvWaveRows;  // kNs == 1: lanes 32..63 repeat
    int64_t n = row0 + r;
    n = n < N ? n : N - 1;
    srow[m] = n * ng;
    sgrp[m] = v % Cfg::kNs;
  }
  auto issue = [&](int s) {  // loads of slot s (past the end: the last slot again)
    const int sc = s < nslot ? s : nslot - 1;
    const uint32_t dst = wlds + (s & 1) * Cfg::kSlotBytes;
    const int64_t kcol = (int64_t)sc * kGemvSlotK;
    // a row piece past K (last slot of a ragged K) re-reads its last unit
    const uint32_t units = (uint32_t)((K - kcol) / 64 < 8 ? (K - kcol) / 64 : 8);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t off = coff[j];
      const uint32_t u = (lane & 7) ^ gemv_swz(8 * j + (lane >> 3));
      if (u >= units) off -= 16u * (u - (units - 1));
      gemv_dma16(cbase + kcol / 4, off, dst + 1024 * j);
    }
#pragma unroll
    for (int m = 0; m < Cfg::kSLoads; ++m) {
      int64_t grp = kcol / G + sgrp[m];
      grp = grp < ng ? grp : ng - 1;
      gemv_dma2(sbase, (uint32_t)((srow[m] + grp) * 2), dst + kGemvSlotCodes + 256 * m);
    }
  };

  const uint16_t* xm = x + mat * (int64_t)B * K;
  const int zpad = B * (int)KP;  // element offset of the zero pad in xs
  // lanes whose batch row b = l16 exists read x; the others read the zero pad
  const bool xl = l16 < B;
  const int xbase = xl ? l16 * (int)KP : zpad;
  const uint32_t kmask = xl ? 0xFFFFFFFFu : 0u;

  f32x4 acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Partial sums alternate between two buffers: the scale of chunk c - 1 is
  // applied after the MFMAs of chunk c are issued, so the vector ALUs never
  // wait for the MFMA chain they just started.
  f32x4 pb[2][NB];
  float spend[NB] = {0.f, 0.f};

  int s = 0;  // next slot to compute; slots s, s + 1 are in flight
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
    if (kp0 == 0) {
      issue(0);
      issue(1);
    }

    // slots of this part (KP is a multiple of the slot width)
    const int send = (int)((kp0 + kpl + kGemvSlotK - 1) / kGemvSlotK);
    for (; s < send; ++s) {
      // slot s landed: only slot s + 1's loads may still be in flight
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"(Cfg::kLoads) : "memory");
      const uint8_t* cs = smem + wave * Cfg::kWaveBytes + (s & 1) * Cfg::kSlotBytes;
      const uint8_t* ss = cs + kGemvSlotCodes;
      const int64_t kcol = (int64_t)s * kGemvSlotK;
      const int cend = (int)((K - kcol) / C < CPS ? (K - kcol) / C : CPS);
      gemv_static_for<0, CPS>([&](auto c_tag) {
        constexpr int c = decltype(c_tag)::value;
        if (c >= cend) return;  // the last slot of a ragged K
        constexpr int buf = c & 1;
        // this chunk's code words and scale, per block
        uint32_t cw[NB][2];
        float sv[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int r = 16 * j + l16;
          const int byte = C == 128 ? 32 * c + 8 * q : (C == 64 ? 16 * c + 4 * q : 8 * c + 4 * (q >> 1));
          const uint8_t* p = cs + 128 * r + 16 * ((byte >> 4) ^ gemv_swz(r)) + (byte & 15);
          if constexpr (C == 128) {
            const u32x2 v = *reinterpret_cast<const u32x2*>(p);
            cw[j][0] = v.x;
            cw[j][1] = v.y;
          } else {
            cw[j][0] = *reinterpret_cast<const uint32_t*>(p);
            cw[j][1] = cw[j][0];
          }
          const int jj = (int)((c * C) / G);  // group of the chunk inside the slot
          const uint32_t sraw = *reinterpret_cast<const uint32_t*>(ss + 4 * (r * Cfg::kNs + jj));
          sv[j] = (float)__builtin_bit_cast(_Float16, (uint16_t)sraw);
        }
        const uint32_t kb0 = (uint32_t)(kcol - kp0 + (int64_t)c * C) & kmask;
#pragma unroll
        for (int t = 0; t < SPC; ++t) {
          const int word = C == 128 ? 2 * q + (t >> 1) : (C == 64 ? q : q >> 1);
          const int half = C == 32 ? (q & 1) : (C == 64 ? t : (t & 1));
          const bf16x8 af = as_bf16x8(
              *reinterpret_cast<const u32x4*>(&xs[xbase + kb0 + 16 * word + 8 * half]));
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const uint32_t w = cw[j][C == 128 ? (t >> 1) : 0];
            bf16x8 bop;
            if constexpr (C == 32)
              bop = decode_half_rt(w, (uint32_t)(q & 1));
            else
              bop = ((C == 64 ? t : t & 1) != 0) ? decode_half<1>(w) : decode_half<0>(w);
            pb[buf][j] = mfma16(af, bop, t == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : pb[buf][j]);
          }
        }
        if (c > 0) {
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[j] += spend[j] * pb[buf ^ 1][j];
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) spend[j] = sv[j];
        if (c + 1 == cend) {  // the slot's last chunk: nothing to overlap with
#pragma unroll
          for (int j = 0; j < NB; ++j) acc[j] += spend[j] * pb[buf][j];
        }
      });
      // this wave's reads of the slot are done: refill it with slot s + 2
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      issue(s + 2);
    }
  }
  // loads issued past the end must land before the workgroup's LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // lane holds column (row of W) l16 of each block and batch rows 4*q + i
  float* ym = y + mat * (int64_t)B * N;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int64_t n = row0 + 16 * j + l16;
    if (n >= N) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int b = 4 * q + i;
      if (b < B) ym[(int64_t)b * N + n] = 0.5f * acc[j][i];
    }
  }
}

template <int G>
static void launch_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                     int B, int64_t N, int64_t K, float* y, hipStream_t stream) {
  constexpr int C = G < 128 ? G : 128;
  // x part staged in LDS: B * KP bf16 plus a C-wide zero pad; KP is a
  // multiple of the slot width so that slots never straddle two parts
  int64_t KP = ((kGemvXBytes / 2 - C) / B) / kGemvSlotK * kGemvSlotK;
  if (KP > K) KP = K;
  const size_t lds = (size_t)kGemvWaves * GemvCfg<G>::kWaveBytes + (size_t)(B * KP + C) * 2;
  const dim3 grid((unsigned)((N + kGemvRows - 1) / kGemvRows), (unsigned)count);
  const dim3 block(64 * kGemvWaves);
  hipLaunchKernelGGL((tgemv_kernel<G>), grid, block, lds, stream, x, codes, s16, B, N, K, KP, y);
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
