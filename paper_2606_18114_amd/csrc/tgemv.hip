// Decode-time ternary GEMV (batch B <= 16), strided-batched over matrices.
//
// Batch-1 decoding is bound by the weight bytes (paper Sec. 8), so the kernel
// is built to keep the vector ALUs nearly idle while the packed codes stream
// from HBM: the matrix cores take the codes almost as stored.
//
// Operands.  v_mfma_scale_f32_16x16x128_f8f6f4 multiplies 16 rows of FP8
// (e4m3) activations by 16 weight rows of FP4 (e2m1) codes over 128 columns.
// A code word's sixteen 2-bit two's-complement codes become FP4 values 2*q
// with one AND for the eight codes at bits 4j+2..4j+3 (already the sign and
// high exponent bit of an e2m1 nibble: 0100 = +2, 1100 = -2) and one shift
// and one AND for the eight at bits 4j..4j+1; the shift is done 64 bits wide
// for two words at once.  So one instruction decodes ~6.4 codes per lane,
// against ~1.4 for a bfloat16 operand.
//
// Activations.  A bfloat16 value has 8 significant bits, an e4m3 value 4, so
// each x is split into two FP8 terms at a power-of-two exponent e:
//   t1 = fp8(x * 2^-e),  t2 = fp8((x * 2^-e - t1) * 16),
// and x = (t1 + t2 / 16) * 2^e exactly whenever |x * 2^-e| >= 2^-6.  The
// exponent is chosen per 32-column block of a row (the 32 values one MFMA
// k block covers) and handed to the matrix core as the E8M0 scale of that
// block, so an outlier only sets the exponent of its own block.
//
// The matrix core adds the 32 products of a block at about 13 bits below
// the largest of them (measured: a product whose lowest bit lies further
// down is truncated; sums across blocks are float32-accurate).  So each A
// row of a block must keep its values within 2^8 of its largest one.  The
// values of a block are therefore cut into two magnitude classes: "large"
// values (|x| >= 2^(e-1), where e scales the block maximum into [128, 256))
// are split at e, the others at the exponent of their own maximum.  Each
// class and term is a row of the MFMA's A operand, four rows per batch
// item, with scales 2^e and 2^(e-4) for the two terms.  Every value of at
// least 2^-8 times the largest of its class is exact, which includes every
// value within 2^16 of its block maximum; smaller ones err by less than
// 2^-11 of the largest small value.  Blocks whose maximum lies under 2^-116
// keep the exponent -123 that the scale range allows.  The other rows of the
// operand hold other batch items and, for g < 128, the other groups inside
// the 128 columns (each row zero outside its group).
//
// Work split: one workgroup of 4 waves per (matrix, 128-row block); each wave
// owns 32 consecutive weight rows (two 16-row blocks) and walks the whole K
// range in 512-column slots.  Launches with few row blocks (one layer's
// matrix) use a split form instead: one workgroup per 32 rows, whose waves
// share the slots and add their partial sums in LDS (see the kernel).
//
// Loads: a wave's slot (32 rows x 128 bytes of codes, plus the rows' float16
// group scales) arrives in a wave-private LDS buffer by direct-to-LDS loads
// (global_load_lds) that each read 8 whole rows' 128-byte pieces.  The eight
// 16-byte units of a row piece are stored XOR-permuted by gemv_swz(row), so
// the reads below are bank-conflict free.  The loads are issued from inline
// assembly, so the compiler neither tracks them nor waits for them; each wave
// counts its own and waits with s_waitcnt.  When a slot has landed the wave
// copies its code words and scales into registers and refills the buffer
// with the next slot at once, so a slot is in flight while the wave computes:
// the bytes in flight are bounded by LDS (about 4 KiB per wave, up to seven
// workgroups per CU), and register-destination loads of the same bytes in
// the MFMA's lane layout were measured three times slower.
//
// Compute per 128-column chunk c and 16-row block: lane (row l16, lane group
// q) takes the two code words 2q, 2q+1 of the chunk (columns 32q .. 32q+31),
// decodes them into its 32 FP4 values (MFMA k = 32q + i), and the lane's A
// operand is the matching 32 FP8 values of its A row, laid out in LDS in the
// MFMA's k order when x is staged.  The partial sums of a chunk are scaled by
// their group's float16 scale in float32 (acc += s * partial), one chunk
// behind the MFMAs so the vector ALUs never wait on the matrix core.
#include <type_traits>

#include "common.hpp"
#include "launchers.hpp"

namespace tmk {

// Launch shape: waves per workgroup, LDS ring depth (slots per wave) and
// slot width in columns.
constexpr int kGemvWaves = 4;
constexpr int kGemvRing = 1;
constexpr int kGemvSlotK = 512;
constexpr int kGemvBlocks = 2;                   // 16-row MFMA blocks per wave
constexpr int kGemvWaveRows = 16 * kGemvBlocks;  // 32
// LDS budget for the split x: 36 KiB holds a whole in_proj row (K = 2048)
// for 16 A rows (batch 4 at g >= 128), three workgroups still fit a CU
constexpr int kGemvXBytes = 36 * 1024;
constexpr int kGemvXPad = 16;                    // bytes between A rows in LDS (bank spread)

typedef __attribute__((ext_vector_type(8))) int i32x8;

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
// lane i: 4 bytes at base + voff -> LDS lds_base + 4 i
__device__ __forceinline__ void gemv_dma4(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

// Two code words (32 codes, columns 0..31 of the pair) as 32 FP4 values 2*q.
// Value i of the result (MFMA k = 32 q + i) holds column fp4_col(i):
//   dwords 0, 2 (word 0, 1): nibble j -> column 4j + 2 (j < 4), 4(j-4) + 3
//   dwords 1, 3:             nibble j -> column 4j     (j < 4), 4(j-4) + 1
// (plus 16 for dwords 2, 3).  The 64-bit shift also moves two bits of word 0
// into the bottom of dword 3's source; the mask clears them.
__device__ __forceinline__ i32x8 decode_fp4(u32x2 w) {
  constexpr uint32_t kNib = 0xCCCCCCCCu;
  const u32x2 s = shl64(w, 2);
  i32x8 r;
  r[0] = (int)(w.x & kNib);
  r[1] = (int)(s.x & kNib);
  r[2] = (int)(w.y & kNib);
  r[3] = (int)(s.y & kNib);
  r[4] = 0;
  r[5] = 0;
  r[6] = 0;
  r[7] = 0;
  return r;
}

// This file is built without the VGPR form of the matrix instructions, so
// the result lands in accumulator registers and can never share registers
// with an operand: with the result allocated over part of the B operand's
// VGPRs, this instruction was measured to give wrong sums (the operand is
// evidently still being read while the result is written).
// A: FP8 e4m3 (cbsz 0) scaled per lane by the E8M0 byte OPSEL of `escale`
// (lane (row r, block q) holds row r's columns 32 q .. 32 q + 31 of the
// chunk); B: FP4 e2m1 (blgp 4) with the scale 2^-1, since the codes are 2 q.
template <int OPSEL>
__device__ __forceinline__ f32x4 mfma_f8f4(i32x8 a, i32x8 b, int escale) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 4,
                                                          OPSEL, escale, 0, 126);
}

// A rows per batch item and group: large/small magnitude class x two terms
constexpr int kTerms = 4;

// Order of a 16-column piece of x in the MFMA's k order (see decode_fp4):
// byte o of the piece holds column kFp4Col[o].
__device__ constexpr int kFp4Col[16] = {2, 6, 10, 14, 3, 7, 11, 15, 0, 4, 8, 12, 1, 5, 9, 13};


// ---------------------------------------------------------------------------
// Pieces shared by both kernels
// ---------------------------------------------------------------------------

// Exponent that scales a block maximum into [128, 256), 0 for an all-zero
// block, and at least -123 so that both terms' E8M0 scales (127 + e and
// 127 + e - 4) stay in range.
__device__ __forceinline__ int block_exp(float mx) {
  const int e = mx > 0.f ? __builtin_amdgcn_frexp_expf(mx) - 8 : 0;
  return e < -123 ? -123 : e;
}

// FP8 terms of four scaled values a[0..3] (byte j of the result: value j)
__device__ __forceinline__ void fp8_terms(const float (&a)[4], uint32_t& p1out, uint32_t& p2out) {
  int p1 = __builtin_amdgcn_cvt_pk_fp8_f32(a[0], a[1], 0, false);
  p1 = __builtin_amdgcn_cvt_pk_fp8_f32(a[2], a[3], p1, true);
  const float r0 = 16.f * (a[0] - __builtin_amdgcn_cvt_f32_fp8(p1, 0));
  const float r1 = 16.f * (a[1] - __builtin_amdgcn_cvt_f32_fp8(p1, 1));
  const float r2 = 16.f * (a[2] - __builtin_amdgcn_cvt_f32_fp8(p1, 2));
  const float r3 = 16.f * (a[3] - __builtin_amdgcn_cvt_f32_fp8(p1, 3));
  int p2 = __builtin_amdgcn_cvt_pk_fp8_f32(r0, r1, 0, false);
  p2 = __builtin_amdgcn_cvt_pk_fp8_f32(r2, r3, p2, true);
  p1out = (uint32_t)p1;
  p2out = (uint32_t)p2;
}

// Split the 32-column block held by a lane pair (lane and lane ^ 1, each with
// 16 bfloat16 values in wv; dead lanes pass zeros) into its four A rows in
// the MFMA's k order: t[0], t[1] the large class's terms, t[2], t[3] the
// small class's; e[u] is row u's scale exponent.  Both lanes of a pair must
// call this together (the block maxima are exchanged between them).
__device__ __forceinline__ void split_block(const uint32_t (&wv)[8], bool live, u32x4 (&t)[kTerms],
                                            int (&e)[kTerms]) {
  float v[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const uint32_t bits = (c & 1) ? (wv[c >> 1] & 0xFFFF0000u) : (wv[c >> 1] << 16);
    v[c] = live ? __uint_as_float(bits) : 0.f;
  }
  float m = 0.f;
#pragma unroll
  for (int c = 0; c < 16; ++c) m = fmaxf(m, fabsf(v[c]));
  m = fmaxf(m, __shfl_xor(m, 1));
  const int eb = block_exp(m);
  const float thr = __builtin_ldexpf(1.f, eb - 1);  // large: within 2^8 of the maximum
  float ms = 0.f;
#pragma unroll
  for (int c = 0; c < 16; ++c) ms = fabsf(v[c]) < thr ? fmaxf(ms, fabsf(v[c])) : ms;
  ms = fmaxf(ms, __shfl_xor(ms, 1));
  const int es = block_exp(ms);
  e[0] = eb;
  e[1] = eb - 4;
  e[2] = es;
  e[3] = es - 4;
  uint32_t o[kTerms][4];
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    float al[4], as[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const float x = v[kFp4Col[4 * d + jj]];
      const bool large = fabsf(x) >= thr;
      al[jj] = large ? __builtin_ldexpf(x, -eb) : 0.f;
      as[jj] = large ? 0.f : __builtin_ldexpf(x, -es);
    }
    fp8_terms(al, o[0][d], o[1][d]);
    fp8_terms(as, o[2][d], o[3][d]);
  }
#pragma unroll
  for (int u = 0; u < kTerms; ++u) t[u] = u32x4{o[u][0], o[u][1], o[u][2], o[u][3]};
}

// max |x| of bfloat16 pairs
__device__ __forceinline__ float absmax2(float m, uint32_t w) {
  m = fmaxf(m, fabsf(__uint_as_float(w << 16)));
  return fmaxf(m, fabsf(__uint_as_float(w & 0xFFFF0000u)));
}

// Write one split 16-column piece of batch row b at MFMA k offset koff of the
// A rows (kTerms b + u) H + hh: the piece's own group h gets the terms, the
// other groups of the chunk zeros.
template <int H>
__device__ __forceinline__ void put_piece(uint8_t* xs, int xstride, int b, int h, int koff,
                                          const u32x4 (&t)[kTerms]) {
  const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int u = 0; u < kTerms; ++u)
#pragma unroll
    for (int hh = 0; hh < H; ++hh)
      st16(xs + ((kTerms * b + u) * H + hh) * xstride + koff, hh == h ? t[u] : z);
}

// Byte of 32-column block blk (of an x part) in an A row's exponent bytes:
// one 32-bit word per (512-column slot, lane group q) holds the bytes of the
// slot's four 128-column chunks, so a lane reads its scales for a whole slot
// with one load and the MFMA picks the chunk's byte.
__device__ __forceinline__ int exp_index(int blk) {
  return (blk >> 4) * 16 + (blk & 3) * 4 + ((blk >> 2) & 3);
}

// E8M0 scale bytes of block blk for the A rows of batch row b (group h gets
// 127 + e[u]; the other groups' rows, which are zero there, get 2^0)
template <int H>
__device__ __forceinline__ void put_exps(uint8_t* es, int estride, int b, int h, int blk,
                                         const int (&e)[kTerms]) {
  const int idx = exp_index(blk);
#pragma unroll
  for (int u = 0; u < kTerms; ++u)
#pragma unroll
    for (int hh = 0; hh < H; ++hh)
      es[((kTerms * b + u) * H + hh) * estride + idx] = (uint8_t)(hh == h ? 127 + e[u] : 127);
}

// MFMA k offset of the first byte of the 16-column piece at column col
// (a multiple of 16) of a run of whole 128-column chunks
__device__ __forceinline__ int piece_koff(int col) {
  const int cic = col % 128;
  return (col - cic) + 32 * (cic / 32) + 16 * ((cic / 16) % 2);
}

// Store y for the wave's rows rowb .. rowb + 31.  Lane (row l16, group q)
// holds, per group hh, the scaled sum of its D rows 16 r + 4 q + i with
// i % H == hh; D row (kTerms b + u) H + hh belongs to batch item b.
template <int NR, int H>
__device__ __forceinline__ void store_rows(const float (&acc)[NR][kGemvBlocks][H], int B,
                                           int64_t N, int64_t rowb, int l16, int q, float* ym,
                                           bool accum) {
  auto put = [&](int64_t at, float v) {
    if (accum)
      ym[at] += v;  // each element has one owner lane: a plain read-modify-write
    else
      ym[at] = v;
  };
#pragma unroll
  for (int j = 0; j < kGemvBlocks; ++j) {
    const int64_t n = rowb + 16 * j + l16;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      float v = acc[r][j][0];
#pragma unroll
      for (int hh = 1; hh < H; ++hh) v += acc[r][j][hh];
      if constexpr (H == 1) {
        // rows 4b .. 4b+3 are lane group q's four rows
        const int b = 4 * r + q;
        if (n < N && b < B) put((int64_t)b * N + n, v);
      } else if constexpr (H == 2) {
        // rows 8b .. 8b+7: lane groups q = 2(b%2) and q + 1
        v += __shfl_xor(v, 16);
        const int b = 2 * r + (q >> 1);
        if ((q & 1) == 0 && n < N && b < B) put((int64_t)b * N + n, v);
      } else {
        // rows 16b .. 16b+15: all four lane groups of operand r
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (q == 0 && n < N && r < B) put((int64_t)r * N + n, v);
      }
    }
  }
}

// Per-lane load plan of a slot (32 rows x SK columns of one matrix): code
// offsets (16-byte units, XOR-permuted per row) and scale indices.  SW: the
// scales arrive as 4-byte words holding two float16 values (packed in LDS;
// needs an even number of groups per row and a 4-byte aligned array), else as
// one float16 per lane (each in its own 4-byte LDS word).
template <int G, int SK, bool SW>
struct SlotPlan {
  static constexpr int U = SK / 64;
  static constexpr int kCodeLoads = U / 2;
  static constexpr int kNs = SK / G > 1 ? SK / G : 1;        // scales per row per slot
  static constexpr int kPer = SW ? kNs / 2 : kNs;             // scale loads per row
  static constexpr int kSLoads = (kGemvWaveRows * kPer + 63) / 64;
  static constexpr int kCodeBytes = kGemvWaveRows * SK / 4;
  static constexpr int kSlotBytes = kCodeBytes + 256 * kSLoads;
  static constexpr int kLoads = kCodeLoads + kSLoads;
  static_assert(!SW || kNs % 2 == 0, "word scale loads need two groups per row and slot");
  int lane;
  __device__ __forceinline__ void init(int l) { lane = l; }
  // wave row and 16-byte unit of code load j, wave row and first group of
  // scale load m
  __device__ __forceinline__ int crow(int j) const { return (64 / U) * j + lane / U; }
  __device__ __forceinline__ int cunit(int j) const { return (lane % U) ^ gemv_swz<U>(crow(j)); }
  __device__ __forceinline__ int srow(int m) const {
    return ((64 * m + lane) / kPer) % kGemvWaveRows;  // lanes past 32 rows repeat
  }
  __device__ __forceinline__ int sgrp(int m) const { return ((64 * m + lane) % kPer) * (SW ? 2 : 1); }
  // loads of the slot at column kcol of rows rowb .. rowb + 31 of one matrix
  __device__ __forceinline__ void issue(const uint8_t* cmat, const uint16_t* smat, int64_t N,
                                        int64_t K, int64_t rowb, int64_t kcol,
                                        uint32_t dst) const {
    const int64_t kb = K / 4, ng = K / G;
    // a row piece past K (last slot of a ragged K) re-reads its last unit
    const int units = (int)((K - kcol) / 64 < U ? (K - kcol) / 64 : U);
#pragma unroll
    for (int j = 0; j < kCodeLoads; ++j) {
      int64_t n = rowb + crow(j);
      n = n < N ? n : N - 1;
      const int unit = cunit(j) < units ? cunit(j) : units - 1;
      gemv_dma16(cmat + kcol / 4, (uint32_t)(n * kb) + 16u * (uint32_t)unit, dst + 1024 * j);
    }
#pragma unroll
    for (int m = 0; m < kSLoads; ++m) {
      int64_t n = rowb + srow(m);
      n = n < N ? n : N - 1;
      int64_t grp = kcol / G + sgrp(m);
      grp = grp < ng ? grp : ng - (SW ? 2 : 1);
      if constexpr (SW)
        gemv_dma4(smat, (uint32_t)((n * ng + grp) * 2), dst + kCodeBytes + 256 * m);
      else
        gemv_dma2(smat, (uint32_t)((n * ng + grp) * 2), dst + kCodeBytes + 256 * m);
    }
  }
  // float16 scale of wave row r, group jj of the slot
  __device__ __forceinline__ static float scale(const uint8_t* ss, int r, int jj) {
    const int v = r * kNs + jj;
    const uint16_t raw = SW ? *reinterpret_cast<const uint16_t*>(ss + 2 * v)
                            : (uint16_t)*reinterpret_cast<const uint32_t*>(ss + 4 * v);
    return (float)__builtin_bit_cast(_Float16, raw);
  }
};

// A slot's code words and scales, read from LDS into registers so that the
// slot's buffer can be refilled before the slot is computed.
template <int G, int SK, int H>
struct SlotRegs {
  static constexpr int CPS = SK / 128;
  u32x2 cw[kGemvBlocks][CPS];
  float sv[kGemvBlocks][CPS][H];
  template <bool SW>
  __device__ __forceinline__ void fetch(const uint8_t* cs, int l16, int q) {
    constexpr int U = SK / 64;
#pragma unroll
    for (int j = 0; j < kGemvBlocks; ++j) {
      const int r = 16 * j + l16;
#pragma unroll
      for (int c = 0; c < CPS; ++c) {
        const int byte = 32 * c + 8 * q;
        cw[j][c] = *reinterpret_cast<const u32x2*>(cs + (SK / 4) * r +
                                                   16 * ((byte >> 4) ^ gemv_swz<U>(r)) +
                                                   (byte & 15));
#pragma unroll
        for (int hh = 0; hh < H; ++hh)
          sv[j][c][hh] = SlotPlan<G, SK, SW>::scale(cs + kGemvWaveRows * SK / 4, r,
                                                    (c * 128 + hh * (G < 128 ? G : 0)) / G);
      }
    }
  }
};

// acc[r][j][hh] += (group hh's float16 scale) x (the sum of the chunk's D
// rows of group hh): lane row i of a lane group is group i % H, and the
// rows of one group in a lane are the terms of one batch item.
template <int NR, int H, int CPS>
__device__ __forceinline__ void scale_add(const f32x4 (&pb)[NR][kGemvBlocks],
                                          const float (&sv)[kGemvBlocks][CPS][H], int c,
                                          float (&acc)[NR][kGemvBlocks][H]) {
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int j = 0; j < kGemvBlocks; ++j)
#pragma unroll
      for (int hh = 0; hh < H; ++hh) {
        float t = pb[r][j][hh];
#pragma unroll
        for (int i = hh + H; i < 4; i += H) t += pb[r][j][i];
        acc[r][j][hh] += sv[j][c][hh] * t;
      }
}

// One slot of a wave from registers: cend full 128-column chunks plus a final
// 64-column chunk when tail64, with the A rows at part column kb0 (a
// multiple of the slot width) and their exponent words at ebase.  Adds the
// scaled partial sums into acc.
template <int G, int SK, int NR, int H>
__device__ __forceinline__ void slot_compute(const uint8_t* smem, const SlotRegs<G, SK, H>& sr,
                                             const int (&abase)[NR],
                                             const uint32_t (&amask)[NR],
                                             const int (&ebase)[NR], uint32_t kb0, int cend,
                                             bool tail64, int q,
                                             float (&acc)[NR][kGemvBlocks][H]) {
  constexpr int CPS = SK / 128;
  constexpr int NB = kGemvBlocks;
  static_assert(CPS <= 4, "one exponent word covers four chunks");
  int esc[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r)
    esc[r] = *reinterpret_cast<const int*>(smem + ebase[r] + (kb0 / 512) * 16 + 4 * q);
  // partial sums alternate between two buffers: chunk c - 1 is scaled after
  // the MFMAs of chunk c are issued, so the vector ALUs never wait on them
  f32x4 pb[2][NR][NB];
  gemv_static_for<0, CPS>([&](auto c_tag) {
    constexpr int c = decltype(c_tag)::value;
    if (c > cend || (c == cend && !tail64)) return;
    constexpr int buf = c & 1;
    i32x8 bop[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)  // columns past K (g < 128, last chunk) decode to zero
      bop[j] = decode_fp4((G < 128 && c == cend && q >= 2) ? u32x2{0u, 0u} : sr.cw[j][c]);
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const uint8_t* ap = smem + abase[r] + ((kb0 + 128u * c) & amask[r]) + 16 * q;
      const u32x4 a0 = *reinterpret_cast<const u32x4*>(ap);
      const u32x4 a1 = *reinterpret_cast<const u32x4*>(ap + 64);
      const i32x8 aop = {(int)a0.x, (int)a0.y, (int)a0.z, (int)a0.w,
                         (int)a1.x, (int)a1.y, (int)a1.z, (int)a1.w};
#pragma unroll
      for (int j = 0; j < NB; ++j) pb[buf][r][j] = mfma_f8f4<c>(aop, bop[j], esc[r]);
    }
    if constexpr (c > 0) scale_add<NR, H, CPS>(pb[buf ^ 1], sr.sv, c - 1, acc);
    if (c == CPS - 1 || c + 1 > cend || (c + 1 == cend && !tail64))  // the slot's last chunk
      scale_add<NR, H, CPS>(pb[buf], sr.sv, c, acc);
  });
}

// ---------------------------------------------------------------------------
// The kernel
// ---------------------------------------------------------------------------
//
// One workgroup per (matrix, 128-row block); each of its 4 waves owns 32 rows
// and walks K in 512-column slots.  The split x (FP8 A rows and their E8M0
// exponent bytes) is staged in LDS in parts of KP columns (a multiple of the
// slot width) that fit the LDS budget, with up to NR = 4 A operands of 16
// rows per chunk (the launcher splits larger batches; x and y rows of matrix
// m start at m * xms and m * yms).
//
// XD (x by direct-to-LDS loads, one part only): the raw bfloat16 x of the
// matrix is fetched into the A-row area by direct-to-LDS loads issued before
// the first slot's codes, so both arrive within one memory latency; every
// thread then takes its (at most two) 16-column pieces into registers and,
// once all raw pieces are read, splits them in place.  Otherwise each part
// is split from global memory.
//
// KS (split K across the waves, for launches with few row blocks): all waves
// of the workgroup share its 32 rows, wave w takes slots w, w + WAVES, ...,
// and the partial sums are added in LDS in wave order (deterministic) before
// wave 0 stores y.  A single matrix of in_proj has only 67 blocks of 128
// rows, out_proj 16, so without the split most CUs would idle.
//
// RMS (XD only; a decoding block's normalization fused into the staging):
// x is not given; each batch row b of the float32 source xr is normalized,
//   x[b, k] = bf16(xr[b, k] / sqrt(mean_k xr[b, k]^2 + eps) * nw[k]),
// by every workgroup for itself: each thread loads its pieces of the source
// rows and of the weight into registers, the sums of squares are taken per
// 16-column piece and then per row in a fixed order (deterministic).
// accum: y += the product instead of y = (each element has one owner lane).
//
// PAIR (one launch over two stacks of matrices, e.g. the in_proj and the
// out_proj layers of a decode token): the grid is one-dimensional, the first
// pr.nb0 workgroups take the stack given by the regular arguments (pr.rb0 row
// blocks per matrix), the rest the stack in `pr`; the stacks share g, B and
// the launch shape, so the tail of the first overlaps the head of the second
// instead of draining the GPU between two launches.
struct GemvPair {
  const uint16_t* x;
  const uint8_t* codes;
  const uint16_t* s16;
  float* y;
  int64_t N, K, KP, xms, yms, nb0, rb0, rb1;
};

template <int G, int WAVES, int RING, int SK, int NR, bool SW, bool XD, bool KS, bool RMS,
          bool PAIR = false>
__global__ __launch_bounds__(64 * WAVES) void tgemv_kernel(
    const uint16_t* __restrict__ x_a, const uint8_t* __restrict__ codes_a,
    const uint16_t* __restrict__ scales_a, int B, int64_t N_a, int64_t K_a, int64_t KP_a,
    int64_t xms_a, int64_t yms_a, float* __restrict__ y_a, const float* __restrict__ xr,
    const float* __restrict__ nw, float eps, int accum, GemvPair pr = GemvPair{}) {
  static_assert(!RMS || XD, "the fused normalization stages x directly");
  static_assert(!PAIR || (XD && !KS && !RMS), "pairs take the plain staged-x form");
  // the stack of this workgroup (uniform), its matrix and its row block
  const uint16_t* x = x_a;
  const uint8_t* codes = codes_a;
  const uint16_t* scales_f16 = scales_a;
  float* y = y_a;
  int64_t N = N_a, K = K_a, KP = KP_a, xms = xms_a, yms = yms_a;
  int64_t mat = blockIdx.y, rblk = blockIdx.x;
  if constexpr (PAIR) {
    const int64_t bid = blockIdx.x;
    if (bid < pr.nb0) {
      mat = bid / pr.rb0;
      rblk = bid % pr.rb0;
    } else {
      x = pr.x;
      codes = pr.codes;
      scales_f16 = pr.s16;
      y = pr.y;
      N = pr.N;
      K = pr.K;
      KP = pr.KP;
      xms = pr.xms;
      yms = pr.yms;
      mat = (bid - pr.nb0) / pr.rb1;
      rblk = (bid - pr.nb0) % pr.rb1;
    }
  }
  using Plan = SlotPlan<G, SK, SW>;
  constexpr int H = G < 128 ? 128 / G : 1;
  constexpr int CPS = SK / 128;
  constexpr int kXPieces = 2;  // XD: 16-column x pieces per thread
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  // [waves][codes | scales] | A rows [R][KP + pad] (XD: raw x first) |
  // exponent bytes [R][KP / 32] | zero pad [128]

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l16 = lane & 15;
  const int q = lane >> 4;
  const int nslot = (int)((K + SK - 1) / SK);
  const int64_t rowb = KS ? rblk * kGemvWaveRows
                          : rblk * (kGemvWaveRows * WAVES) + wave * kGemvWaveRows;
  const int s0 = KS ? wave : 0;       // first slot of this wave
  const int sstep = KS ? WAVES : 1;   // slot stride
  const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
  const uint32_t wlds = lds0 + wave * RING * Plan::kSlotBytes;
  const int R = kTerms * B * H;
  const int xstride = (int)KP + kGemvXPad;
  const int estride = (int)(KP / 32);
  const int xoff = WAVES * RING * Plan::kSlotBytes;
  uint8_t* xs = smem + xoff;
  const int64_t KR = (K + 511) / 512 * 512;  // XD: raw x row length
  const int xarea = XD && !RMS && B * KR * 2 > R * xstride ? (int)(B * KR * 2) : R * xstride;
  const int eoff = xoff + xarea;
  uint8_t* es = smem + eoff;
  const int zoff = eoff + (R * estride + 15) / 16 * 16;
  // RMS: per-piece sums of squares [2 x 64 WAVES] | row factors [4]
  float* part = reinterpret_cast<float*>(smem + zoff + 128);
  float* rfac = part + 2 * 64 * WAVES;

  Plan plan;
  plan.init(lane);
  const uint8_t* cmat = codes + mat * N * (K / 4);
  const uint16_t* smat = scales_f16 + mat * N * (K / G);
  auto issue = [&](int s) {  // slot s (past the end: the last slot again) into its ring buffer
    const int sc = s < nslot ? s : nslot - 1;
    plan.issue(cmat, smat, N, K, rowb, (int64_t)sc * SK,
               wlds + ((s / sstep) % RING) * Plan::kSlotBytes);
  };
  const uint16_t* xm = x + mat * xms;

  // operand rows past R read the zero pad (and row 0's exponents, any valid
  // scale: their values are zero)
  int abase[NR], ebase[NR];
  uint32_t amask[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int gr = 16 * r + l16;
    abase[r] = gr < R ? xoff + gr * xstride : zoff;
    amask[r] = gr < R ? 0xFFFFFFFFu : 0u;
    ebase[r] = eoff + (gr < R ? gr : 0) * estride;
  }
  float acc[NR][kGemvBlocks][H];
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int j = 0; j < kGemvBlocks; ++j)
#pragma unroll
      for (int i = 0; i < H; ++i) acc[r][j][i] = 0.f;

  // split piece i (16 columns) of an x part whose pieces per row are
  // `pieces`; the lane pair i, i ^ 1 holds one 32-column block
  auto put_split = [&](int i, int pieces, int64_t kpl, const uint32_t (&wv)[8]) {
    const int b = i / pieces, col = 16 * (i % pieces);
    const bool live = col < kpl;
    u32x4 t[kTerms];
    int e[kTerms];
    split_block(wv, live, t, e);
    const int h = live ? (G < 128 ? (col % 128) / G : 0) : -1;
    put_piece<H>(xs, xstride, b, h, piece_koff(col), t);
    if ((i & 1) == 0) put_exps<H>(es, estride, b, h, col / 32, e);
  };

  if constexpr (XD) {
    // this thread's pieces (16 columns of one batch row, up to whole chunks)
    const int pieces = (int)((K + 127) / 128 * 8);
    uint32_t wv[kXPieces][8];
    if constexpr (RMS) {
      // the pieces of the source rows and the norm weight straight into
      // registers, issued before the slots' direct-to-LDS loads (the
      // compiler's own waits for them then also cover those slots)
      const float* xrm = xr + mat * xms;
      float v[kXPieces][16], wk[kXPieces][16];
#pragma unroll
      for (int m = 0; m < kXPieces; ++m) {
        const int i = threadIdx.x + 64 * WAVES * m;
        const int b = i / pieces, col = 16 * (i % pieces);
        const bool live = b < B && col < K;
#pragma unroll
        for (int c = 0; c < 16; c += 4) {
          u32x4 t = {0u, 0u, 0u, 0u}, u = {0u, 0u, 0u, 0u};
          if (live) {
            t = ld16(xrm + (int64_t)b * K + col + c);
            u = ld16(nw + col + c);
          }
          v[m][c] = __uint_as_float(t.x);
          v[m][c + 1] = __uint_as_float(t.y);
          v[m][c + 2] = __uint_as_float(t.z);
          v[m][c + 3] = __uint_as_float(t.w);
          wk[m][c] = __uint_as_float(u.x);
          wk[m][c + 1] = __uint_as_float(u.y);
          wk[m][c + 2] = __uint_as_float(u.z);
          wk[m][c + 3] = __uint_as_float(u.w);
        }
      }
      for (int p = 0; p < RING; ++p) issue(s0 + p * sstep);
#pragma unroll
      for (int m = 0; m < kXPieces; ++m) {
        const int i = threadIdx.x + 64 * WAVES * m;
        float sq = 0.f;
#pragma unroll
        for (int c = 0; c < 16; ++c) sq = __builtin_fmaf(v[m][c], v[m][c], sq);
        if (i / pieces < B) part[i] = sq;
      }
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"(RING * Plan::kLoads) : "memory");
      __syncthreads();
      // row factors: the pieces' sums in a fixed order, then across a wave;
      // one row: every wave takes it itself (no second barrier); more: wave
      // b takes row b and hands it over in LDS
      auto row_factor = [&](int b) {
        float sq = 0.f;
        for (int j = lane; j < pieces; j += 64) sq += part[b * pieces + j];
        sq += __uint_as_float(lane_xchg<1>(__float_as_uint(sq)));
        sq += __uint_as_float(lane_xchg<2>(__float_as_uint(sq)));
        sq += __uint_as_float(lane_xchg<4>(__float_as_uint(sq)));
        sq += __uint_as_float(lane_xchg<8>(__float_as_uint(sq)));
        sq += __uint_as_float(lane_xchg<16>(__float_as_uint(sq)));
        sq += __uint_as_float(lane_xchg<32>(__float_as_uint(sq)));
        return 1.f / sqrtf(sq / (float)K + eps);
      };
      float rf[4] = {0.f, 0.f, 0.f, 0.f};
      if (B == 1) {
        rf[0] = row_factor(0);
      } else {
        if (wave < B) {
          const float r = row_factor(wave);
          if (lane == 0) rfac[wave] = r;
        }
        __syncthreads();
#pragma unroll
        for (int b = 0; b < 4; ++b) rf[b] = b < B ? rfac[b] : 0.f;
      }
#pragma unroll
      for (int m = 0; m < kXPieces; ++m) {
        const int i = threadIdx.x + 64 * WAVES * m;
        const int b = i / pieces;
        const float r = b == 0 ? rf[0] : b == 1 ? rf[1] : b == 2 ? rf[2] : rf[3];
#pragma unroll
        for (int c = 0; c < 16; c += 2) {   // dead pieces hold zeros
          const uint32_t lo = __float_as_uint(v[m][c] * r * wk[m][c]);
          const uint32_t hi = __float_as_uint(v[m][c + 1] * r * wk[m][c + 1]);
          const uint32_t blo = (lo + 0x7FFFu + ((lo >> 16) & 1u)) >> 16;   // round to
          const uint32_t bhi = (hi + 0x7FFFu + ((hi >> 16) & 1u)) >> 16;   // nearest even
          wv[m][c / 2] = blo | (bhi << 16);
        }
      }
    } else {
      // raw x (row b, columns 512 p .. 512 p + 511 per load; a load past K
      // re-reads the row's last 16 bytes into the row's pad), then the codes
      const int xl = B * (int)(KR / 512);
      for (int pi = wave; pi < xl; pi += WAVES) {
        const int b = pi / (int)(KR / 512), p = pi % (int)(KR / 512);
        int64_t e = 512 * (int64_t)p + 8 * lane;
        e = e < K - 8 ? e : K - 8;
        gemv_dma16(xm + (int64_t)b * K, (uint32_t)(2 * e),
                   lds0 + xoff + 2 * (uint32_t)(b * KR + 512 * p));
      }
      for (int p = 0; p < RING; ++p) issue(s0 + p * sstep);
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"(RING * Plan::kLoads) : "memory");  // own x landed
      __syncthreads();
      const uint16_t* xraw = reinterpret_cast<const uint16_t*>(xs);
#pragma unroll
      for (int m = 0; m < kXPieces; ++m) {
        const int i = threadIdx.x + 64 * WAVES * m;
        const int b = i / pieces, col = 16 * (i % pieces);
        const bool live = b < B && col < K;
        const int e = live ? (int)(b * KR) + col : 0;
        const u32x4 v0 = *reinterpret_cast<const u32x4*>(xraw + e);
        const u32x4 v1 = *reinterpret_cast<const u32x4*>(xraw + e + 8);
        wv[m][0] = v0.x; wv[m][1] = v0.y; wv[m][2] = v0.z; wv[m][3] = v0.w;
        wv[m][4] = v1.x; wv[m][5] = v1.y; wv[m][6] = v1.z; wv[m][7] = v1.w;
      }
    }
    __syncthreads();  // every raw piece has been read: the A rows overwrite them
#pragma unroll
    for (int m = 0; m < kXPieces; ++m) {
      const int i = threadIdx.x + 64 * WAVES * m;
      if (i / pieces < B) put_split(i, pieces, K, wv[m]);  // a lane pair shares its row
    }
    for (int i = threadIdx.x; i < 128 / 16; i += 64 * WAVES)
      st16(smem + zoff + 16 * i, u32x4{0u, 0u, 0u, 0u});
    __syncthreads();
  } else {
    for (int p = 0; p < RING; ++p) issue(s0 + p * sstep);
  }

  // part [kp0, kp0 + kpl) of x -> A rows; pieces past kpl up to the end of
  // its last chunk are zeros (stale LDS bytes could be FP8 NaNs)
  auto stage_x = [&](int64_t kp0, int kpl) {
    const int pieces = (kpl + 127) / 128 * 8;
    for (int i = threadIdx.x; i < B * pieces; i += 64 * WAVES) {
      const int b = i / pieces, col = 16 * (i % pieces);
      uint32_t wv[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
      if (col < kpl) {
        const u32x4 v0 = ld16(xm + (int64_t)b * K + kp0 + col);
        const u32x4 v1 = ld16(xm + (int64_t)b * K + kp0 + col + 8);
        wv[0] = v0.x; wv[1] = v0.y; wv[2] = v0.z; wv[3] = v0.w;
        wv[4] = v1.x; wv[5] = v1.y; wv[6] = v1.z; wv[7] = v1.w;
      }
      put_split(i, pieces, kpl, wv);
    }
    for (int i = threadIdx.x; i < 128 / 16; i += 64 * WAVES)
      st16(smem + zoff + 16 * i, u32x4{0u, 0u, 0u, 0u});
  };

  int s = s0;
  for (int64_t kp0 = 0; kp0 < K; kp0 += KP) {
    const int kpl = (int)(K - kp0 < KP ? K - kp0 : KP);
    if constexpr (!XD) {
      if (kp0 > 0) __syncthreads();  // every wave is done with the previous part
      stage_x(kp0, kpl);
      __syncthreads();
    }
    const int send = (int)((kp0 + kpl + SK - 1) / SK);
    for (; s < send; s += sstep) {
      // slot s landed (only the RING - 1 slots after it may still be in flight)
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"((RING - 1) * Plan::kLoads) : "memory");
      SlotRegs<G, SK, H> sr;
      sr.template fetch<SW>(smem + (wave * RING + (s / sstep) % RING) * Plan::kSlotBytes, l16,
                            q);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the buffer is free again
      // (one slot in flight: nothing to issue past the end; deeper rings keep
      // their wait counts exact by reloading the last slot)
      if (RING > 1 || s + RING * sstep < nslot) issue(s + RING * sstep);
      const int64_t kcol = (int64_t)s * SK;
      const int cend = (int)((K - kcol) / 128 < CPS ? (K - kcol) / 128 : CPS);
      const bool tail64 = G < 128 && (K - kcol) % 128 != 0 && (K - kcol) < SK;
      slot_compute<G, SK, NR, H>(smem, sr, abase, amask, ebase, (uint32_t)(kcol - kp0), cend,
                                 tail64, q, acc);
    }
  }
  // loads issued past the end must land before the workgroup's LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if constexpr (KS) {
    // each wave parks its partial sums in its own slot buffer (free now),
    // then wave 0 adds them in wave order
    constexpr int kAcc = NR * kGemvBlocks * H;
    static_assert(kAcc * 64 * 4 <= RING * Plan::kSlotBytes, "partial sums fit the slot buffer");
    float* mine = reinterpret_cast<float*>(smem + wave * RING * Plan::kSlotBytes);
    int t = 0;
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int j = 0; j < kGemvBlocks; ++j)
#pragma unroll
        for (int i = 0; i < H; ++i, ++t) mine[64 * t + lane] = acc[r][j][i];
    __syncthreads();
    if (wave != 0) return;
    for (int w = 1; w < WAVES; ++w) {
      const float* other = reinterpret_cast<const float*>(smem + w * RING * Plan::kSlotBytes);
      t = 0;
#pragma unroll
      for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int j = 0; j < kGemvBlocks; ++j)
#pragma unroll
          for (int i = 0; i < H; ++i, ++t) acc[r][j][i] += other[64 * t + lane];
    }
  }
  store_rows<NR, H>(acc, B, N, rowb, l16, q, y + mat * yms, accum != 0);
}

// ---------------------------------------------------------------------------
// Launch
// ---------------------------------------------------------------------------

template <int G, int WAVES, bool KS>
static hipError_t launch_gw(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                            int count, int B, int64_t N, int64_t K, float* y, hipStream_t stream,
                            const float* xr = nullptr, const float* nw = nullptr, float eps = 0.f,
                            int accum = 0) {
  constexpr int H = G < 128 ? 128 / G : 1;
  constexpr int SK = kGemvSlotK;
  constexpr int RING = kGemvRing;
  const int R = kTerms * B * H;
  const int rmax = R < 64 ? R : 64;  // A rows of one pass
  int budget = kGemvXBytes;
  if (budget < rmax * (SK + kGemvXPad)) budget = rmax * (SK + kGemvXPad);
  int64_t KP = (int64_t)(budget / rmax - kGemvXPad) / SK * SK;
  if (KP > K) KP = (K + SK - 1) / SK * SK;
  const int64_t KR = (K + 511) / 512 * 512;
  // x by direct-to-LDS loads: one part, at most two 16-column pieces per thread
  const bool xd = KP >= K && R <= 16 && B * ((K + 127) / 128 * 8) <= 2 * 64 * WAVES;
  // scales as 4-byte words: an even number of groups per row (so every row
  // and matrix starts 4-byte aligned) and two groups per slot
  const bool sw = (K / G) % 2 == 0 && SK / G >= 2 && ((uintptr_t)s16 & 3) == 0;
  constexpr int kRowsPerBlock = KS ? kGemvWaveRows : kGemvWaveRows * WAVES;
  const dim3 grid((unsigned)((N + kRowsPerBlock - 1) / kRowsPerBlock), (unsigned)count);
  const dim3 block(64 * WAVES);
  auto lds_of = [&](int slot_bytes, int rows, bool with_raw) {
    size_t xa = (size_t)rows * (KP + kGemvXPad);
    if (with_raw && (size_t)B * KR * 2 > xa) xa = (size_t)B * KR * 2;
    const size_t ea = ((size_t)rows * (KP / 32) + 15) / 16 * 16;
    return (size_t)WAVES * slot_bytes + xa + ea + 128;
  };
  if (xr) {  // fused normalization: x staged directly, one part over all of K
    const int pieces = (int)((K + 127) / 128 * 8);
    if (R > 16 || B * pieces > 2 * 64 * WAVES) return hipErrorInvalidValue;
    KP = (K + SK - 1) / SK * SK;
    const size_t xa = (size_t)R * (KP + kGemvXPad);
    const size_t ea = ((size_t)R * (KP / 32) + 15) / 16 * 16;
    const size_t aux = 2 * 64 * WAVES * 4 + 16;
#define TM_GEMV_RMS(SW_)                                                                     \
  do {                                                                                        \
    const size_t lds = (size_t)WAVES * RING * SlotPlan<G, SK, SW_>::kSlotBytes + xa + ea + 128 + \
                       aux;                                                                   \
    if (lds > 160 * 1024) return hipErrorInvalidValue;                                        \
    hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, 1, SW_, true, KS, true>), grid, block, \
                       lds, stream, nullptr, codes, s16, B, N, K, KP, (int64_t)B * K,         \
                       (int64_t)B * N, y, xr, nw, eps, accum);                                \
  } while (0)
    if constexpr (SK / G >= 2) {
      if (sw) {
        TM_GEMV_RMS(true);
        return hipGetLastError();
      }
    }
    TM_GEMV_RMS(false);
#undef TM_GEMV_RMS
    return hipGetLastError();
  }
#define TM_GEMV_LAUNCH(NR_, SW_, BP, B0)                                                      \
  hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, NR_, SW_, false, KS, false>), grid,     \
                     block,                                                                   \
                     lds_of(RING * SlotPlan<G, SK, SW_>::kSlotBytes, kTerms * (BP) * H, false), \
                     stream, x + (int64_t)(B0) * K, codes, s16, BP, N, K, KP, (int64_t)B * K,  \
                     (int64_t)B * N, y + (int64_t)(B0) * N, nullptr, nullptr, 0.f, 0)
  if (xd) {  // the common decode case: R <= 16
#define TM_GEMV_XD(SW_)                                                                       \
  hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, 1, SW_, true, KS, false>), grid, block, \
                     lds_of(RING * SlotPlan<G, SK, SW_>::kSlotBytes, R, true), stream, x,     \
                     codes, s16, B, N, K, KP, (int64_t)B * K, (int64_t)B * N, y, nullptr,      \
                     nullptr, 0.f, 0)
    if constexpr (SK / G >= 2) {
      if (sw) {
        TM_GEMV_XD(true);
        return hipGetLastError();
      }
    }
    TM_GEMV_XD(false);
#undef TM_GEMV_XD
    return hipGetLastError();
  }
  // at most 64 A rows per launch: batches beyond 64 / (kTerms H) go in passes
  const int bmax = 64 / (kTerms * H);
  for (int b0 = 0; b0 < B; b0 += bmax) {
    const int bp = B - b0 < bmax ? B - b0 : bmax;
    const int rp = kTerms * bp * H;
    if (rp <= 16) {
      if constexpr (SK / G >= 2) {
        if (sw) {
          TM_GEMV_LAUNCH(1, true, bp, b0);
          continue;
        }
      }
      TM_GEMV_LAUNCH(1, false, bp, b0);
    } else if constexpr (!KS) {  // the split form is only chosen for R <= 16
      if (rp <= 32)
        TM_GEMV_LAUNCH(2, false, bp, b0);
      else
        TM_GEMV_LAUNCH(4, false, bp, b0);
    }
  }
#undef TM_GEMV_LAUNCH
  return hipGetLastError();
}

// Few row blocks in all (a single matrix: one layer's projection) leave most
// CUs idle, so the slots of each 32-row block are split across the waves of
// its workgroup instead (eight waves once K has eight slots), for batches
// whose A rows fit one 16-row operand.
template <int G>
static hipError_t launch_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                           int count, int B, int64_t N, int64_t K, float* y, hipStream_t stream,
                           const float* xr, const float* nw, float eps, int accum) {
  const int64_t blocks = (int64_t)count * ((N + 127) / 128);
  const int64_t nslot = (K + kGemvSlotK - 1) / kGemvSlotK;
  const int R = kTerms * B * (G < 128 ? 128 / G : 1);  // A rows: one 16-row operand when <= 16
  // the fused form (one matrix) takes the split form whenever K has two slots
  if ((xr || blocks < 2 * (int64_t)current_cu_count()) && nslot >= 2 && R <= 16) {
    if (nslot >= 8)
      return launch_gw<G, 8, true>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    return launch_gw<G, kGemvWaves, true>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps,
                                          accum);
  }
  // many A rows (batch 4 at g >= 128): the split x fills much of a
  // workgroup's LDS, so eight waves share it (twice the rows per staging)
  // where the grid still gives every CU several workgroups
  if (R > 8 && (int64_t)count * ((N + 255) / 256) >= 4 * (int64_t)current_cu_count())
    return launch_gw<G, 8, false>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
  return launch_gw<G, kGemvWaves, false>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps,
                                         accum);
}

static hipError_t launch_any_g(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                               int count, int B, int64_t N, int64_t K, int g, float* y,
                               hipStream_t stream, const float* xr, const float* nw, float eps,
                               int accum) {
  switch (g) {
    case 32:  return launch_g<32>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    case 64:  return launch_g<64>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    case 128: return launch_g<128>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    case 256: return launch_g<256>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    case 512: return launch_g<512>(x, codes, s16, count, B, N, K, y, stream, xr, nw, eps, accum);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_tgemv(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                        int B, int64_t N, int64_t K, int g, float* y, hipStream_t stream) {
  return launch_any_g(x, codes, s16, count, B, N, K, g, y, stream, nullptr, nullptr, 0.f, 0);
}

// Two stacks in one launch (PAIR) when both take the plain staged-x form
// with the same scale-load form; otherwise two launches.  (Measured on the
// decode token: out_proj's 128 KiB workgroups first, then in_proj's 64 KiB
// ones, 59.2 us cold against 60.2 us in the other order.)
template <int G>
static hipError_t launch_pair_g(const uint16_t* x0, const uint8_t* c0, const uint16_t* s0,
                                int n0, int64_t N0, int64_t K0, float* y0, const uint16_t* x1,
                                const uint8_t* c1, const uint16_t* s1, int n1, int64_t N1,
                                int64_t K1, float* y1, int B, hipStream_t stream) {
  constexpr int H = G < 128 ? 128 / G : 1;
  constexpr int SK = kGemvSlotK, RING = kGemvRing, WAVES = kGemvWaves;
  const int R = kTerms * B * H;
  auto kp_of = [&](int64_t K) { return (K + SK - 1) / SK * SK; };
  auto staged = [&](int64_t K) {  // the XD condition of launch_gw with KP covering K
    const int rmax = R < 64 ? R : 64;
    int budget = kGemvXBytes;
    if (budget < rmax * (SK + kGemvXPad)) budget = rmax * (SK + kGemvXPad);
    const int64_t kp = (int64_t)(budget / rmax - kGemvXPad) / SK * SK;
    return kp >= K && R <= 16 && B * ((K + 127) / 128 * 8) <= 2 * 64 * WAVES;
  };
  auto words = [&](int64_t K, const uint16_t* sp) {
    return (K / G) % 2 == 0 && SK / G >= 2 && ((uintptr_t)sp & 3) == 0;
  };
  // the stack with the longer rows (more bytes per workgroup) goes first, so
  // the grid ends on the smaller workgroups, which even out the tail
  if (K1 > K0)
    return launch_pair_g<G>(x1, c1, s1, n1, N1, K1, y1, x0, c0, s0, n0, N0, K0, y0, B, stream);
  const bool sw0 = words(K0, s0), sw1 = words(K1, s1);
  const int64_t rb0 = (N0 + 127) / 128, rb1 = (N1 + 127) / 128;
  const int64_t nb0 = (int64_t)n0 * rb0, nb1 = (int64_t)n1 * rb1;
  if (!staged(K0) || !staged(K1) || sw0 != sw1 || nb0 + nb1 > 0x7FFFFFFF) {
    const hipError_t e = launch_g<G>(x0, c0, s0, n0, B, N0, K0, y0, stream, nullptr, nullptr,
                                     0.f, 0);
    if (e != hipSuccess) return e;
    return launch_g<G>(x1, c1, s1, n1, B, N1, K1, y1, stream, nullptr, nullptr, 0.f, 0);
  }
  const int64_t KP0 = kp_of(K0), KP1 = kp_of(K1);
  auto lds_of = [&](int slot_bytes, int64_t KP, int64_t K) {
    const int64_t KR = (K + 511) / 512 * 512;
    size_t xa = (size_t)R * (KP + kGemvXPad);
    if ((size_t)B * KR * 2 > xa) xa = (size_t)B * KR * 2;
    const size_t ea = ((size_t)R * (KP / 32) + 15) / 16 * 16;
    return (size_t)WAVES * slot_bytes + xa + ea + 128;
  };
  GemvPair pr;
  pr.x = x1;
  pr.codes = c1;
  pr.s16 = s1;
  pr.y = y1;
  pr.N = N1;
  pr.K = K1;
  pr.KP = KP1;
  pr.xms = (int64_t)B * K1;
  pr.yms = (int64_t)B * N1;
  pr.nb0 = nb0;
  pr.rb0 = rb0;
  pr.rb1 = rb1;
  const dim3 grid((unsigned)(nb0 + nb1)), block(64 * WAVES);
#define TM_GEMV_PAIR(SW_)                                                                      \
  do {                                                                                         \
    constexpr int kSlot = RING * SlotPlan<G, SK, SW_>::kSlotBytes;                             \
    const size_t la = lds_of(kSlot, KP0, K0), lb = lds_of(kSlot, KP1, K1);                     \
    hipLaunchKernelGGL((tgemv_kernel<G, WAVES, RING, SK, 1, SW_, true, false, false, true>),   \
                       grid, block, la > lb ? la : lb, stream, x0, c0, s0, B, N0, K0, KP0,     \
                       (int64_t)B * K0, (int64_t)B * N0, y0, nullptr, nullptr, 0.f, 0, pr);    \
  } while (0)
  if constexpr (SK / G >= 2) {
    if (sw0) {
      TM_GEMV_PAIR(true);
      return hipGetLastError();
    }
  }
  TM_GEMV_PAIR(false);
#undef TM_GEMV_PAIR
  return hipGetLastError();
}

hipError_t launch_tgemv_pair(const uint16_t* x0, const uint8_t* c0, const uint16_t* s0, int n0,
                             int64_t N0, int64_t K0, float* y0, const uint16_t* x1,
                             const uint8_t* c1, const uint16_t* s1, int n1, int64_t N1,
                             int64_t K1, float* y1, int B, int g, hipStream_t stream) {
  switch (g) {
    case 32:  return launch_pair_g<32>(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, stream);
    case 64:  return launch_pair_g<64>(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, stream);
    case 128: return launch_pair_g<128>(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, stream);
    case 256: return launch_pair_g<256>(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, stream);
    case 512: return launch_pair_g<512>(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, stream);
    default: return hipErrorInvalidValue;
  }
}

static_assert(kTerms == 4 && kGemvSlotK == 512 && kGemvWaves == 4,
              "tgemv_rms_fits (launchers.hpp) assumes this launch shape");

hipError_t launch_tgemv_rms(const float* src, const float* nw, float eps, const uint8_t* codes,
                            const uint16_t* s16, int B, int64_t N, int64_t K, int g, float* y,
                            int accum, hipStream_t stream) {
  return launch_any_g(nullptr, codes, s16, 1, B, N, K, g, y, stream, src, nw, eps, accum);
}

}  // namespace tmk
