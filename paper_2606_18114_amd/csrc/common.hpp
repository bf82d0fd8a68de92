// Shared device helpers for the gfx950 ternary kernels.
//
// Code decode: the packed format keeps, in every 32-bit word of 16 codes,
// element 2i at bits [2i, 2i+2) and element 2i+1 at bits [16+2i, 16+2i+2),
// each as a 2-bit two's complement (00 -> 0, 01 -> +1, 11 -> -1).  Shifting
// the word left by 14 - 2i puts the pair's two codes at bits 14-15 and 30-31;
// masking with 0xC000C000 then leaves, in each 16-bit half, either 0x0000
// (code 0), 0x4000 (bfloat16 +2.0, code +1) or 0xC000 (bfloat16 -2.0, code -1).
// So one shift and one AND turn two codes into two exact bfloat16 operands
// equal to 2*q; the factor 2 is removed in float32 after the contraction.
// The unused pattern 10 decodes to 0x8000 (-0.0) and contributes nothing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tmk {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr uint32_t kPairMask = 0xC000C000u;

// Pair i (elements 2i, 2i+1 of the word) as two bfloat16 values 2*q.
template <int I>
__device__ __forceinline__ uint32_t decode_pair(uint32_t w) {
  static_assert(I >= 0 && I < 8, "pair index");
  return (w << (14 - 2 * I)) & kPairMask;
}

// Eight codes (half H of a word: elements 8H .. 8H+7) as an MFMA operand of
// eight bfloat16 values 2*q, in element order.
template <int H>
__device__ __forceinline__ bf16x8 decode_half(uint32_t w) {
  u32x4 v;
  v.x = decode_pair<4 * H + 0>(w);
  v.y = decode_pair<4 * H + 1>(w);
  v.z = decode_pair<4 * H + 2>(w);
  v.w = decode_pair<4 * H + 3>(w);
  return __builtin_bit_cast(bf16x8, v);
}

// Both halves of two adjacent words (w.x -> a0 (elements 0-7), a1 (8-15);
// w.y -> b0, b1) with 64-bit shifts: shifting the pair (hi = w.y, lo = w.x)
// left by s gives w.x << s in the low dword and w.y << s in the high one (plus
// bits of w.x shifted in below bit s <= 14, which the mask clears), so the 16
// operand dwords cost seven 64-bit shifts and sixteen ANDs instead of 14
// 32-bit shifts and 16 ANDs.  (The shifts are written in assembly: the
// compiler would otherwise fold each masked half back into a 32-bit shift.)
__device__ __forceinline__ u32x2 shl64(u32x2 v, int s) {
  u32x2 r;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(r) : "n"(s), "v"(v));
  return r;
}
__device__ __forceinline__ void decode_words(u32x2 w, bf16x8& a0, bf16x8& a1, bf16x8& b0,
                                             bf16x8& b1) {
  u32x2 r[7];  // r[i] = w << (14 - 2 i), pair i of each word at bits 14-15 / 30-31
  r[0] = shl64(w, 14);
  r[1] = shl64(w, 12);
  r[2] = shl64(w, 10);
  r[3] = shl64(w, 8);
  r[4] = shl64(w, 6);
  r[5] = shl64(w, 4);
  r[6] = shl64(w, 2);
  const u32x4 x0 = {r[0].x & kPairMask, r[1].x & kPairMask, r[2].x & kPairMask, r[3].x & kPairMask};
  const u32x4 x1 = {r[4].x & kPairMask, r[5].x & kPairMask, r[6].x & kPairMask, w.x & kPairMask};
  const u32x4 y0 = {r[0].y & kPairMask, r[1].y & kPairMask, r[2].y & kPairMask, r[3].y & kPairMask};
  const u32x4 y1 = {r[4].y & kPairMask, r[5].y & kPairMask, r[6].y & kPairMask, w.y & kPairMask};
  a0 = __builtin_bit_cast(bf16x8, x0);
  a1 = __builtin_bit_cast(bf16x8, x1);
  b0 = __builtin_bit_cast(bf16x8, y0);
  b1 = __builtin_bit_cast(bf16x8, y1);
}

// Half h (elements 8h .. 8h+7, h chosen at run time) of two words at once
// (w.x -> b0, w.y -> b1) as MFMA operands of eight bfloat16 values 2*q, with
// the half-select shift hs = 8 - 8 h given.  One 64-bit shift moves both
// words, so the two operands cost four 64-bit shifts and eight ANDs instead
// of eight 32-bit shifts and eight ANDs.  Bits of w.x shifted into the high
// word land below bit 14, where the mask clears them.
__device__ __forceinline__ void decode_half_pair_rt(u32x2 w, uint32_t hs, bf16x8& b0,
                                                    bf16x8& b1) {
  u32x2 ws;
  asm("v_lshlrev_b64 %0, %1, %2" : "=v"(ws) : "v"(hs), "v"(w));
  const u32x2 r6 = shl64(ws, 6), r4 = shl64(ws, 4), r2 = shl64(ws, 2);
  const u32x4 x = {r6.x & kPairMask, r4.x & kPairMask, r2.x & kPairMask, ws.x & kPairMask};
  const u32x4 y = {r6.y & kPairMask, r4.y & kPairMask, r2.y & kPairMask, ws.y & kPairMask};
  b0 = __builtin_bit_cast(bf16x8, x);
  b1 = __builtin_bit_cast(bf16x8, y);
}

// Exchange between lanes for all-reduce butterflies, without the LDS
// crossbar where a DPP pattern exists: partner of lane i for step O is
// i ^ 1, i ^ 2 (quad permutes), the mirror lane in its 8 (O = 4) or 16
// (O = 8) lanes, i ^ 16 (ds_swizzle), i ^ 32.  After the steps below O each
// lane's partner holds the sum of a disjoint set of the same size, so the
// mirrors pair up as well as an XOR would, and every lane ends with the same
// sum (two lanes add the same pair in either order).
template <int O>
__device__ __forceinline__ uint32_t lane_xchg(uint32_t v) {
  if constexpr (O == 1)
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
  else if constexpr (O == 2)
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
  else if constexpr (O == 4)
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
  else if constexpr (O == 8)
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);
  else if constexpr (O == 16)
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);
  else
    return (uint32_t)__shfl_xor((int)v, O, 64);
}
template <int O>
__device__ __forceinline__ double lane_xchg_f64(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint64_t lo = lane_xchg<O>((uint32_t)u), hi = lane_xchg<O>((uint32_t)(u >> 32));
  return __longlong_as_double((long long)((hi << 32) | lo));
}
// Sum over aligned groups of L lanes (L a power of two <= 64), in every lane.
template <int L>
__device__ __forceinline__ double group_sum_f64(double v) {
  if constexpr (L >= 2) v += lane_xchg_f64<1>(v);
  if constexpr (L >= 4) v += lane_xchg_f64<2>(v);
  if constexpr (L >= 8) v += lane_xchg_f64<4>(v);
  if constexpr (L >= 16) v += lane_xchg_f64<8>(v);
  if constexpr (L >= 32) v += lane_xchg_f64<16>(v);
  if constexpr (L >= 64) v += lane_xchg_f64<32>(v);
  return v;
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 16-byte global load / store through plain vector types.
__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

// Remap a linear workgroup id so that consecutive ids run on the same XCD.
// The dispatcher hands workgroup i to XCD i % 8; ids that share an XCD share
// its L2, so tiles that reuse the same operand rows should be consecutive
// after the remap.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t bid, uint32_t nblocks) {
  constexpr uint32_t kXcd = 8;
  const uint32_t per = nblocks / kXcd;   // full rounds
  const uint32_t tail = nblocks % kXcd;  // XCDs that get one extra block
  const uint32_t xcd = bid % kXcd;
  const uint32_t local = bid / kXcd;
  // XCD x owns ids [start(x), start(x) + per + (x < tail))
  const uint32_t start = xcd * per + (xcd < tail ? xcd : tail);
  return start + local;
}

}  // namespace tmk
