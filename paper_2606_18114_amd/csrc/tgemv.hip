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
// Loads: the codes of a wave's 32 rows are staged through a wave-private LDS
// ring (kGemvRing slots) of 512 columns (128 bytes per row), filled by
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

// Launch shape: waves per workgroup, LDS ring depth (slots per wave) and
// slot width in columns.  One slot per wave (the next slot's loads are issued
// once the current one is consumed) measured faster than two or more: the
// smaller LDS footprint fits more workgroups per CU, and the other waves
// cover each wave's load latency.
constexpr int kGemvWaves = 4;
constexpr int kGemvRing = 1;
constexpr int kGemvSlotK = 512;
constexpr int kGemvBlocks = 2;                   // 16-row MFMA blocks per wave
constexpr int kGemvWaveRows = 16 * kGemvBlocks;  // 32
constexpr int kGemvXBytes = 32 * 1024;           // LDS budget for x

template <int G, int WAVES, int RING, int SK>
struct GemvCfg {
  static constexpr int kUnits = SK / 64;                   // 16-byte units per row piece
  static constexpr int kCodeLoads = kUnits / 2;            // 1 KiB loads per slot (32 rows)
  static constexpr int kSlotCodes = kGemvWaveRows * SK / 4;
  static constexpr int kNs = SK / G > 1 ? SK / G : 1;      // scales per row per slot
  static constexpr int kSLoads = (kGemvWaveRows * kNs + 63) / 64;
  static constexpr int kSlotScales = 256 * kSLoads;        // LDS bytes (4 per value)
  static constexpr int kSlotBytes = kSlotCodes + kSlotScales;
  static constexpr int kWaveBytes = RING * kSlotBytes;
  static constexpr int kLoads = kCodeLoads + kSLoads;      // direct-to-LDS loads per slot
  static constexpr int kRows = kGemvWaveRows * WAVES;      // rows per workgroup
};

// 16-byte unit permutation of wave row r inside a slot (units per row: U)
template <int U>
__device__ __forceinline__ int gemv_swz(int r) {
  if constexpr (U == 8)
    return (r & 7) ^ ((r >> 3) & 1);
  else
    return (((r >> 1) ^ (r >> 3)) & 1) | (((r >> 2) & 1) << 1);
}

// calls f(integral_constant<int, I>) for I in [I0, N), fully unrolled
template <int I, int N, typename F>
__device__ __forceinline__ void gemv_static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    gemv_static_for<I + 1, N>(f);
  }
}

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

template <int G, int WAVES, int RING, int SK, int NV>
__global__ __launch_bounds__(64 * WAVES) void tgemv_kernel(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ codes,
    const uint16_t* __restrict__ scales_f16, int B, int64_t N, int64_t K, int64_t KP,
    float* __restrict__ y) {
  using Cfg = GemvCfg<G, WAVES, RING, SK>;
  constexpr int C = G < 128 ? G : 128;   // chunk width
  constexpr int SPC = C / 32;            // MFMA steps per chunk
  constexpr int CPS = SK / C;            // chunks per slot
  constexpr int NB = kGemvBlocks;
  constexpr int U = Cfg::kUnits;
  // NV: batch rows a lane's partial sums can hold (1 when B == 1, else 4)
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  // [waves][RING slots][codes | scales], then x [B][KP] + zero pad

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15;
  const int q = lane >> 4;  // lane group: the MFMA's 8-column k slice
  const int64_t mat = blockIdx.y;
  const int64_t kb = K / 4;  // code bytes per row
  const int64_t ng = K / G;
  const int nslot = (int)((K + SK - 1) / SK);
  const int64_t row0 = (int64_t)blockIdx.x * Cfg::kRows + wave * kGemvWaveRows;  // wave's rows
  const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
  const uint32_t wlds = lds0 + wave * Cfg::kWaveBytes;
  const int xoff_b = WAVES * Cfg::kWaveBytes;  // byte offset of x in LDS
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + xoff_b);

  // ---- load plan of one slot (uniform base + per-lane offsets) ----
  // codes: load j covers wave rows (64/U) j .. +64/U - 1; lane -> row
  // (64/U) j + lane/U, unit lane%U of the LDS row piece, which holds logical
  // unit (lane%U) ^ gemv_swz(row)
  const uint8_t* cbase = codes + (mat * N) * kb;
  uint32_t coff[Cfg::kCodeLoads];
  int cunit[Cfg::kCodeLoads];
#pragma unroll
  for (int j = 0; j < Cfg::kCodeLoads; ++j) {
    const int r = (64 / U) * j + lane / U;
    int64_t n = row0 + r;
    n = n < N ? n : N - 1;
    cunit[j] = (lane % U) ^ gemv_swz<U>(r);
    coff[j] = (uint32_t)(n * kb) + 16u * cunit[j];
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
  int islot = 0;  // ring buffer of the next slot to issue
  auto issue = [&](int s) {  // loads of slot s (past the end: the last slot again)
    const int sc = s < nslot ? s : nslot - 1;
    const uint32_t dst = wlds + islot * Cfg::kSlotBytes;
    islot = islot == RING - 1 ? 0 : islot + 1;
    const int64_t kcol = (int64_t)sc * SK;
    // a row piece past K (last slot of a ragged K) re-reads its last unit
    const int units = (int)((K - kcol) / 64 < U ? (K - kcol) / 64 : U);
#pragma unroll
    for (int j = 0; j < Cfg::kCodeLoads; ++j) {
      uint32_t off = coff[j];
      if (cunit[j] >= units) off -= 16u * (uint32_t)(cunit[j] - (units - 1));
      gemv_dma16(cbase + kcol / 4, off, dst + 1024 * j);
    }
#pragma unroll
    for (int m = 0; m < Cfg::kSLoads; ++m) {
      int64_t grp = kcol / G + sgrp[m];
      grp = grp < ng ? grp : ng - 1;
      gemv_dma2(sbase, (uint32_t)((srow[m] + grp) * 2), dst + Cfg::kSlotCodes + 256 * m);
    }
  };
  // x part [B][kp0, kp0 + kpl) -> xs[B][KP]: 1 KiB loads spread over the waves
  // (a load past the part re-reads its last 16 bytes; those columns are
  // never used), then the zero pad
  const uint16_t* xm = x + mat * (int64_t)B * K;
  const int zpad = B * (int)KP;  // element offset of the zero pad in xs
  auto stage_x = [&](int64_t kp0, int kpl) {
    const int per_row = (kpl + 511) / 512;
    for (int i = wave; i < B * per_row; i += WAVES) {
      const int b = i / per_row, ch = i % per_row;
      int e = 512 * ch + 8 * lane;
      e = e < kpl - 8 ? e : kpl - 8;
      gemv_dma16(xm + (int64_t)b * K + kp0, (uint32_t)(2 * e),
                 lds0 + xoff_b + 2 * (b * (int)KP + 512 * ch));
    }
    for (int i = threadIdx.x; i < C / 8; i += 64 * WAVES)
      st16(&xs[zpad + 8 * i], u32x4{0u, 0u, 0u, 0u});
  };

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

  // prologue: x part 0 and the first RING code slots in flight together
  stage_x(0, (int)(K < KP ? K : KP));
  for (int p = 0; p < RING; ++p) issue(p);
  // own x loads landed (only code loads newer), zero pad written; then a plain
  // barrier, which unlike __syncthreads does not wait for the code loads
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(RING * Cfg::kLoads) : "memory");

  int s = 0;      // next slot to compute; slots s .. s + RING - 1 are in flight
  int cslot = 0;  // its ring buffer
  for (int64_t kp0 = 0; kp0 < K; kp0 += KP) {
    const int kpl = (int)(K - kp0 < KP ? K - kp0 : KP);
    if (kp0 > 0) {  // next x part: every wave is done with the previous one
      __syncthreads();
      stage_x(kp0, kpl);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
    // slots of this part (KP is a multiple of the slot width)
    const int send = (int)((kp0 + kpl + SK - 1) / SK);
    for (; s < send; ++s) {
      // slot s landed: only the RING - 1 slots after it may still be in flight
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"((RING - 1) * Cfg::kLoads) : "memory");
      const uint8_t* cs = smem + wave * Cfg::kWaveBytes + cslot * Cfg::kSlotBytes;
      const uint8_t* ss = cs + Cfg::kSlotCodes;
      cslot = cslot == RING - 1 ? 0 : cslot + 1;
      const int64_t kcol = (int64_t)s * SK;
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
          const uint8_t* p = cs + (SK / 4) * r + 16 * ((byte >> 4) ^ gemv_swz<U>(r)) + (byte & 15);
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
        // the chunk's B operands: step t takes word t / 2 (C = 128) or the
        // only word (C = 64), half t % 2; C = 32 picks its half per lane
        bf16x8 bops[NB][SPC];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          if constexpr (C == 128) {
            decode_words(u32x2{cw[j][0], cw[j][1]}, bops[j][0], bops[j][1], bops[j][2], bops[j][3]);
          } else if constexpr (C == 64) {
            bops[j][0] = decode_half<0>(cw[j][0]);
            bops[j][1] = decode_half<1>(cw[j][0]);
          } else {
            bops[j][0] = decode_half_rt(cw[j][0], (uint32_t)(q & 1));
          }
        }
        const uint32_t kb0 = (uint32_t)(kcol - kp0 + (int64_t)c * C) & kmask;
#pragma unroll
        for (int t = 0; t < SPC; ++t) {
          const int word = C == 128 ? 2 * q + (t >> 1) : (C == 64 ? q : q >> 1);
          const int half = C == 32 ? (q & 1) : (C == 64 ? t : (t & 1));
          const bf16x8 af = as_bf16x8(
              *reinterpret_cast<const u32x4*>(&xs[xbase + kb0 + 16 * word + 8 * half]));
#pragma unroll
          for (int j = 0; j < NB; ++j)
            pb[buf][j] = mfma16(af, bops[j][t], t == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : pb[buf][j]);
        }
        if (c > 0) {
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < NV; ++i) acc[j][i] += spend[j] * pb[buf ^ 1][j][i];
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) spend[j] = sv[j];
        if (c + 1 == cend) {  // the slot's last chunk: nothing to overlap with
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int i = 0; i < NV; ++i) acc[j][i] += spend[j] * pb[buf][j][i];
        }
      });
      // this wave's reads of the slot are done: refill its buffer
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      issue(s + RING);
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
    for (int i = 0; i < NV; ++i) {
      const int b = 4 * q + i;
      if (b < B) ym[(int64_t)b * N + n] = 0.5f * acc[j][i];
    }
  }
}

template <int G, int WAVES = kGemvWaves, int RING = kGemvRing, int SK = kGemvSlotK>
static void launch_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                     int B, int64_t N, int64_t K, float* y, hipStream_t stream) {
  using Cfg = GemvCfg<G, WAVES, RING, SK>;
  constexpr int C = G < 128 ? G : 128;
  // x part staged in LDS: B * KP bf16 plus a C-wide zero pad; KP is a
  // multiple of 512 columns (whole slots, whole x loads)
  int64_t KP = ((kGemvXBytes / 2 - C) / B) / 512 * 512;
  if (KP > K) KP = (K + 511) / 512 * 512;
  const size_t lds = (size_t)WAVES * Cfg::kWaveBytes + (size_t)(B * KP + C) * 2;
  const dim3 grid((unsigned)((N + Cfg::kRows - 1) / Cfg::kRows), (unsigned)count);
  const dim3 block(64 * WAVES);
  if (B == 1)
    hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, 1>), grid, block, lds, stream, x, codes,
                       s16, B, N, K, KP, y);
  else
    hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, 4>), grid, block, lds, stream, x, codes,
                       s16, B, N, K, KP, y);
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
