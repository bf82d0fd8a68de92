// Straight-through backward w.r.t. the input in one float16 pass (paper
// Sec. 3.1):
//   dX[M, K] = dY[M, N] . What[N, K],  What = q * s,
// a contraction over N on the gfx950 matrix cores (v_mfma_f32_32x32x16_f16),
// float32 accumulation.
//
// The scale varies along the contraction, so it has to sit inside the
// operand.  bfloat16 keeps 8 significant bits of it (about 2e-3 relative
// error in dX); the two-pass kernel of tgemm_bwd_dx.hip keeps 16 bits at
// twice the matrix-core work.  Here both operands are float16, which keeps 11
// bits of the scale in a single pass:
//   * dY' = fp16(dY * 2^e[m]) with one power of two per row m, chosen so that
//     the row's largest magnitude lands in [2^14, 2^15): every bfloat16 value
//     within 2^28 of its row maximum converts exactly (8 significant bits fit
//     in 11), smaller ones enter as float16 subnormals or zero;
//   * the weight operand is q * fp16(s * 2^t), one power of two t for the
//     tensor (largest scale in [2^14, 2^15)): each dequantized weight carries
//     a relative error of at most 2^-11;
//   * the products are exact in float32 and the result is
//     dX = acc * 2^-(e[m] + t), applied in the store.
// A prepass (dx_prep_kernel) writes dY', the row exponents and per-wave
// maxima of the scales into a caller-owned workspace; the contraction kernel
// reduces those maxima to t in its prologue.
//
// The contraction kernel is the two-pass kernel with one weight plane: tiles
// of 256 (M) x 256 (K) outputs per workgroup of 4 waves (2 x 2), 128 x 128 per
// wave, 32 weight rows per stage, dY' / codes / scales in a 4-deep LDS ring of
// direct-to-LDS loads issued three stages ahead, the codes decoded one stage
// ahead into a double-buffered float16 plane read back by ds_read_b64_tr_b16,
// 32 MFMAs per wave and stage.  Work split as there: whole tiles round-robin,
// the remainder cut along N and added with float32 atomics into a cleared dX.
// The weight plane is built from the codes with one shift and one AND per two
// codes (the float16 values 2q) and one packed float16 multiply by the scale.
#include "dx_common.hpp"
#include "launchers.hpp"

namespace tmk {

constexpr int kHxTM = 256, kHxTK = 256, kHxBN = 32, kHxRing = 4;
constexpr int kHxY = kHxTM * kHxBN * 2;             // 16 KiB: dY' tile of a stage
constexpr int kHxC = kHxBN * kHxTK / 4;             // 2 KiB: packed codes of a stage
constexpr int kHxS = 1024;                          // scales: <= 32 rows x 8 groups
constexpr int kHxSlot = kHxY + kHxC + kHxS;         // 19 KiB ring slot
constexpr int kHxPlane = kHxBN * kHxTK * 2;         // 16 KiB: one float16 plane
constexpr int kHxRx = 2 * kHxTM * 4;                // row exponents, two items
constexpr int kHxRxBase = 2 * kHxPlane;
constexpr int kHxRingBase = kHxRxBase + kHxRx;
constexpr int kHxLds = kHxRingBase + kHxRing * kHxSlot;  // 110 KiB
constexpr int kHxLoads = 7;                         // direct-to-LDS loads per wave per stage
// At the end of stage s a wave waits until only the dY' loads of stage s + 2
// and all loads of stage s + 3 are in flight: stage s + 1's data and stage
// s + 2's codes and scales (decoded during stage s + 1) have landed.
constexpr int kHxWait = kHxLoads + 4;

constexpr int kScaleParts = kDxScaleParts;
// 16-byte pieces of a dY row each lane of the prepass holds in registers
constexpr int kPrepPieces = 24;

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;

__device__ __forceinline__ f32x16 mfma32h(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, lane_xchg<1>(v));
  v = max(v, lane_xchg<2>(v));
  v = max(v, lane_xchg<4>(v));
  v = max(v, lane_xchg<8>(v));
  v = max(v, lane_xchg<16>(v));
  v = max(v, lane_xchg<32>(v));
  return v;
}

// power of two that puts a magnitude with biased exponent field E (of a
// float with exponent bias 127: bfloat16 or float32; E = 0 for subnormals)
// into [2^14, 2^15); 0 for zero, infinity and NaN
__device__ __forceinline__ int exp_to_2p14(uint32_t E, bool special) {
  return special ? 0 : 141 - (int)E;
}

// two bfloat16 values (one 32-bit word) times 2^e, as two float16 values
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w, int e) {
  const float lo = ldexpf(__uint_as_float(w << 16), e);
  const float hi = ldexpf(__uint_as_float(w & 0xFFFF0000u), e);
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

// Prepass.  Waves 0 .. nparts-1 first take the largest magnitude in one
// slice of the float32 scales (as unsigned bits) into parts[wave].  Then
// every wave converts whole rows of dY: a row is held in registers (when it
// has at most 64 * kPrepPieces pieces of 8 values, else read twice), its
// largest magnitude gives e[m], and the row is written back as float16.
__global__ __launch_bounds__(256) void dx_prep_kernel(
    const uint16_t* __restrict__ dY, const float* __restrict__ scales, int64_t M, int64_t N,
    int64_t nsc, uint16_t* __restrict__ dY16, int32_t* __restrict__ rexp,
    uint32_t* __restrict__ parts, int nparts) {
  const int lane = threadIdx.x & 63;
  const int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nw = (int64_t)gridDim.x * 4;
  if (gw < nparts) {
    const int64_t per = (nsc + nparts - 1) / nparts;
    const int64_t lo = gw * per, hi = lo + per < nsc ? lo + per : nsc;
    const uint32_t* sb = reinterpret_cast<const uint32_t*>(scales);
    uint32_t v = 0;
    for (int64_t i = lo + lane; i < hi; i += 64) v = max(v, sb[i] & 0x7FFFFFFFu);
    v = wave_max_u32(v);
    if (lane == 0) parts[gw] = v;
  }
  const int64_t npc = N / 8;  // 16-byte pieces per row (N % 8 == 0)
  const bool in_regs = npc <= 64 * kPrepPieces;
  for (int64_t m = gw; m < M; m += nw) {
    const u32x4* src = reinterpret_cast<const u32x4*>(dY + m * N);
    u32x4* dst = reinterpret_cast<u32x4*>(dY16 + m * N);
    u32x4 v[kPrepPieces];
    uint32_t mx = 0;
    auto fold = [&](const u32x4& p) {
#pragma unroll
      for (int j = 0; j < 4; ++j) mx = max(mx, max(p[j] & 0x7FFFu, (p[j] >> 16) & 0x7FFFu));
    };
    if (in_regs) {
#pragma unroll
      for (int i = 0; i < kPrepPieces; ++i) {
        const int64_t p = lane + 64 * i;
        v[i] = p < npc ? src[p] : u32x4{0u, 0u, 0u, 0u};
        fold(v[i]);
      }
    } else {
      for (int64_t p = lane; p < npc; p += 64) fold(src[p]);
    }
    mx = wave_max_u32(mx);
    const int e = exp_to_2p14(mx >> 7, mx == 0 || mx >= 0x7F80u);
    auto conv = [&](const u32x4& p) {
      return u32x4{bf16x2_to_f16x2(p[0], e), bf16x2_to_f16x2(p[1], e),
                   bf16x2_to_f16x2(p[2], e), bf16x2_to_f16x2(p[3], e)};
    };
    if (in_regs) {
#pragma unroll
      for (int i = 0; i < kPrepPieces; ++i) {
        const int64_t p = lane + 64 * i;
        if (p < npc) dst[p] = conv(v[i]);
      }
    } else {
      for (int64_t p = lane; p < npc; p += 64) dst[p] = conv(src[p]);
    }
    if (lane == 0) rexp[m] = e;
  }
}

template <int G>
__global__ __launch_bounds__(256) void tgemm_bwd_dx_f16_kernel(
    const uint16_t* __restrict__ dY16, const int32_t* __restrict__ rexp,
    const uint32_t* __restrict__ sparts, int nparts, const uint32_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    float* __restrict__ dX, uint32_t tiles_k, uint32_t ntiles, uint32_t parts) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kHxLds];
  constexpr int kGpt = G < kHxTK ? kHxTK / G : 1;  // scale groups per tile row

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wk = wave & 1;  // 128-row (M) and 128-column (K) halves
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int g16 = lane >> 4;
  const int j16 = lane & 15;
  const uint32_t P = gridDim.x;
  const uint32_t bid = xcd_remap(blockIdx.x, P);
  const uint32_t full = ntiles / P;
  const uint32_t rem = ntiles % P;
  const int nst = (int)((N + kHxBN - 1) / kHxBN);
  const int64_t kw = K / 16;
  const int64_t ng = K / G;
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;

  // the tensor's scale exponent t from the prepass maxima (item 1's exponent
  // buffer serves as scratch; items start after the barrier)
  int tsc;
  {
    uint32_t v = 0;
    for (int i = tid; i < nparts; i += 256) v = max(v, sparts[i]);
    v = wave_max_u32(v);
    uint32_t* red = reinterpret_cast<uint32_t*>(lds + kHxRxBase + kHxTM * 4);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    v = max(max(red[0], red[1]), max(red[2], red[3]));
    tsc = exp_to_2p14(v >> 23, v == 0 || v >= 0x7F800000u);
    __syncthreads();
  }

  const int trow = 8 * (g16 >> 1) + (j16 >> 2);
  const int tcol = 16 * (g16 & 1) + 4 * (j16 & 3);
  uint32_t boff[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) boff[b] = dx_poff(trow, wk * 128 + 32 * b + tcol);
  const int ar = wm * 128 + l32;
  const uint32_t aoff0 = dx_yoff(ar, h), aoff1 = dx_yoff(ar, 2 + h);

  // decode role: weight row dr of the stage, code words 2 dj and 2 dj + 1
  const int dr = tid >> 3, dj = tid & 7;
  const uint32_t hsel = (uint32_t)(dj >> 2);
  const uint32_t dswap = hsel ? 0x02030001u : 0x03020100u;
  const uint32_t dcode = kHxY + dr * 64 + 8 * dj;
  const uint32_t dscale = kHxY + kHxC + 4 * (dr * kGpt + (32 * dj) / G);
  const uint32_t dplane = dx_poff(dr, 32 * dj);

  for (uint32_t item = 0;; ++item) {
    uint32_t tile;
    int s_beg, s_end;
    bool whole;
    if (item < full) {
      tile = item * P + bid;
      s_beg = 0;
      s_end = nst;
      whole = true;
    } else if (item == full && rem != 0 && bid < rem * parts) {
      tile = full * P + bid / parts;
      const uint32_t part = bid % parts;
      const int per = (nst + (int)parts - 1) / (int)parts;
      s_beg = (int)part * per;
      s_end = s_beg + per < nst ? s_beg + per : nst;
      whole = false;
      if (s_beg >= s_end) break;
    } else {
      break;
    }
    const int64_t m0 = (int64_t)(tile / tiles_k) * kHxTM;
    const int64_t k0 = (int64_t)(tile % tiles_k) * kHxTK;
    const int rows = (int)(M - m0 < kHxTM ? M - m0 : kHxTM);
    const uint32_t rx = kHxRxBase + (item & 1u) * (kHxTM * 4);

    uint32_t yrow[4], ycol[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * (4 * wave + i) + (lane >> 2);
      const int u = (lane & 3) ^ ((r >> 1) & 3) ^ ((r >> 3) & 1);
      const int rr = r < rows ? r : rows - 1;
      yrow[i] = (uint32_t)rr * (uint32_t)N * 2u;
      ycol[i] = 8u * (uint32_t)u;
    }
    int crow[2];
    uint32_t cword[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = 64 * (2 * wave + i) + lane;
      crow[i] = idx >> 4;
      const int64_t wd = k0 / 16 + (idx & 15);
      cword[i] = (uint32_t)(wd < kw ? wd : kw - 1);
    }
    int srow;
    uint32_t sgrp;
    {
      int idx = 64 * wave + lane;
      idx = idx < 32 * kGpt ? idx : 32 * kGpt - 1;
      srow = idx / kGpt;
      const int64_t gg = k0 / G + idx % kGpt;
      sgrp = (uint32_t)(gg < ng ? gg : ng - 1);
    }
    const uint8_t* ybase = reinterpret_cast<const uint8_t*>(dY16 + m0 * N);

    struct DmaStage {
      const uint32_t* cb;
      const float* sbp;
      uint32_t ncol, dst;
      int nlast;
    };
    auto dma_begin = [&](int st, int slot) {
      st = st < s_end ? st : s_end - 1;
      const int64_t nb = (int64_t)st * kHxBN;
      DmaStage d;
      d.dst = lds0 + kHxRingBase + slot * kHxSlot;
      d.ncol = (uint32_t)nb;
      d.nlast = (int)(N - 1 - nb);
      d.cb = codes + nb * kw;
      d.sbp = scales + nb * ng;
      return d;
    };
    // the loads of a stage in issue order: codes (2), scales (1), then dY' (4)
    // (pieces i = 4, 5, 6, 0 .. 3), so that a wait can cover a stage's codes
    // without its dY', which is needed one stage later
    auto dma_piece = [&](const DmaStage& d, auto i_tag) {
      constexpr int i = (decltype(i_tag)::value + 4) % kHxLoads;
      if constexpr (i < 4) {
        const uint32_t ncap = (uint32_t)N - 8u;
        uint32_t c = d.ncol + ycol[i];
        c = c < ncap ? c : ncap;
        dx_dma16(ybase, yrow[i] + 2u * c, d.dst + 1024 * (4 * wave + i));
      } else if constexpr (i < 6) {
        const int r = crow[i - 4] < d.nlast ? crow[i - 4] : d.nlast;
        dx_dma4(d.cb, ((uint32_t)r * (uint32_t)kw + cword[i - 4]) * 4u,
                d.dst + kHxY + 256 * (2 * wave + (i - 4)));
      } else {
        const int r = srow < d.nlast ? srow : d.nlast;
        dx_dma4(d.sbp, ((uint32_t)r * (uint32_t)ng + sgrp) * 4u,
                d.dst + kHxY + kHxC + 256 * wave);
      }
    };
    auto dma = [&](int st, int slot) {
      const DmaStage d = dma_begin(st, slot);
      dx_static_for<0, kHxLoads>([&](auto i_tag) { dma_piece(d, i_tag); });
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

    auto frag = [&](const uint8_t* plane, uint32_t off, int t) {
      const dx_s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (dx_lds_s16x4*)(plane + off + 16 * t * 512));
      const dx_s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (dx_lds_s16x4*)(plane + off + (16 * t + 4) * 512));
      const u32x2 l = __builtin_bit_cast(u32x2, x), u = __builtin_bit_cast(u32x2, y);
      return u32x4{l.x, l.y, u.x, u.y};
    };

    // decode inputs of stage st: two code words (rows past N read as 0) and
    // the scale as a float16 pair h = fp16(s * 2^(t - 1))
    struct DecIn {
      u32x2 w;
      float s;
      uint32_t s2;
    };
    auto decode_read = [&](auto slot_tag) {
      constexpr int SLOT = decltype(slot_tag)::value;
      const uint8_t* sb = lds + kHxRingBase + SLOT * kHxSlot;
      DecIn d;
      d.w = *reinterpret_cast<const u32x2*>(sb + dcode);
      d.s = *reinterpret_cast<const float*>(sb + dscale);
      return d;
    };
    auto decode_split = [&](DecIn& d, int st) {
      if ((int64_t)st * kHxBN + dr >= N) d.w = u32x2{0u, 0u};
      d.w.x = __builtin_amdgcn_perm(d.w.x, d.w.x, dswap);
      d.w.y = __builtin_amdgcn_perm(d.w.y, d.w.y, dswap);
      const uint32_t hb = __builtin_bit_cast(uint16_t, (_Float16)ldexpf(d.s, tsc - 1));
      d.s2 = hb | (hb << 16);
    };
    // pair I of both words: w << (14 - 2 I) puts the two codes of each word
    // at bits 14-15 / 30-31 (one 64-bit shift moves both words; bits of
    // word 0 shifted into word 1 land below bit 14), and the mask leaves the
    // float16 values 2q (0x4000 = +2, 0xC000 = -2, as in bfloat16); one
    // packed float16 multiply by h gives q * fp16(s * 2^t) exactly
    auto decode_pair2 = [&](auto i_tag, const DecIn& d, u32x4* v) {
      constexpr int I = decltype(i_tag)::value;
      const u32x2 r = I == 7 ? d.w : shl64(d.w, 14 - 2 * I);
      const f16x2 h = __builtin_bit_cast(f16x2, d.s2);
      v[I / 4][I % 4] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, r.x & kPairMask) * h);
      v[2 + I / 4][I % 4] =
          __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, r.y & kPairMask) * h);
    };
    auto plane_write = [&](uint8_t* qb, int H, int word, const u32x4* v) {
      const uint32_t off = (dplane + 16 * ((uint32_t)H ^ hsel)) ^ (word ? 32u : 0u);
      st16(qb + off, v[2 * word + H]);
    };

    // One stage in ring slot I % kHxRing, plane I % 2: the 32 MFMAs of stage
    // st, one per slot fenced by sched_barrier; the decode of stage st + 1 in
    // slots 1 .. 8 (one pair of both words each), the second 16-row step's
    // operand reads in slots 2 .. 9, the plane writes in slots 10 .. 13, the
    // loads of stage st + 3 in slots 21 .. 27.
    auto stage = [&](auto i_tag, int st) {
      constexpr int I = decltype(i_tag)::value;
      constexpr int SLOT = I & (kHxRing - 1), PL = I & 1;
      constexpr int DSLOT = (I + 1) & (kHxRing - 1), DPL = (I + 1) & 1;
      const uint8_t* yb = lds + kHxRingBase + SLOT * kHxSlot;
      const uint8_t* pb = lds + PL * kHxPlane;
      uint8_t* qb = lds + DPL * kHxPlane;
      DecIn din = decode_read(std::integral_constant<int, DSLOT>{});
      __builtin_amdgcn_sched_barrier(0);
      u32x4 af[2][4], bf[2][4];
      af[0][0] = *reinterpret_cast<const u32x4*>(yb + aoff0);
      bf[0][0] = frag(pb, boff[0], 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 1; b < 4; ++b) bf[0][b] = frag(pb, boff[b], 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int a = 1; a < 4; ++a) af[0][a] = *reinterpret_cast<const u32x4*>(yb + aoff0 + 2048 * a);
      __builtin_amdgcn_sched_barrier(0);
      u32x4 vh[4];
      DmaStage dst;
      dx_static_for<0, 32>([&](auto k_tag) {
        constexpr int k = decltype(k_tag)::value;
        constexpr int t = k / 16, c = (k % 16) / 4, b = k % 4;
        acc[c][b] = mfma32h(af[t][c], bf[t][b], acc[c][b]);
        if constexpr (k == 0) decode_split(din, st + 1);
        if constexpr (k >= 1 && k <= 8) decode_pair2(std::integral_constant<int, k - 1>{}, din, vh);
        if constexpr (k >= 2 && k <= 9) {
          constexpr int x = k - 2;
          if constexpr (x < 4)
            bf[1][x] = frag(pb, boff[x], 1);
          else
            af[1][x - 4] = *reinterpret_cast<const u32x4*>(yb + aoff1 + 2048 * (x - 4));
        }
        // half 0 of both words is complete after slot 4, half 1 after 8
        if constexpr (k == 10 || k == 11) plane_write(qb, 0, k - 10, vh);
        if constexpr (k == 12 || k == 13) plane_write(qb, 1, k - 12, vh);
        if constexpr (k == 20)
          dst = dma_begin(st + kHxRing - 1, (I + kHxRing - 1) & (kHxRing - 1));
        if constexpr (k >= 21 && k < 21 + kHxLoads)
          dma_piece(dst, std::integral_constant<int, k - 21>{});
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    auto decode_all = [&](auto slot_tag, auto plane_tag, int st) {
      constexpr int PL = decltype(plane_tag)::value;
      DecIn din = decode_read(slot_tag);
      decode_split(din, st);
      u32x4 vh[4];
      dx_static_for<0, 8>([&](auto i_tag) { decode_pair2(i_tag, din, vh); });
      uint8_t* qb = lds + PL * kHxPlane;
      plane_write(qb, 0, 0, vh);
      plane_write(qb, 0, 1, vh);
      plane_write(qb, 1, 0, vh);
      plane_write(qb, 1, 1, vh);
    };
    auto mma_only = [&](auto slot_tag, auto plane_tag) {
      constexpr int SLOT = decltype(slot_tag)::value;
      constexpr int PL = decltype(plane_tag)::value;
      const uint8_t* yb = lds + kHxRingBase + SLOT * kHxSlot;
      const uint8_t* pb = lds + PL * kHxPlane;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        u32x4 af[4], bf[4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
          af[a] = *reinterpret_cast<const u32x4*>(yb + (t ? aoff1 : aoff0) + 2048 * a);
#pragma unroll
        for (int b = 0; b < 4; ++b) bf[b] = frag(pb, boff[b], t);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) acc[a][b] = mfma32h(af[a], bf[b], acc[a][b]);
      }
    };

    // prologue: the row exponents of the item (one dword per row, four waves
    // of 64 rows; rows past M re-read row M - 1), then stages s_beg .. s_beg + 2
    {
      const int r = 64 * wave + lane;
      const int rr = r < rows ? r : rows - 1;
      dx_dma4(rexp + m0, (uint32_t)rr * 4u, lds0 + rx + 256 * wave);
    }
#pragma unroll
    for (int p = 0; p < kHxRing - 1; ++p) dma(s_beg + p, p);
    dx_stage_barrier<kHxWait>();
    decode_all(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, s_beg);
    dx_stage_barrier<kHxWait>();

    int st0 = s_beg;
    for (; st0 + kHxRing <= s_end; st0 += kHxRing) {
      dx_static_for<0, kHxRing>([&](auto i_tag) {
        stage(i_tag, st0 + decltype(i_tag)::value);
        dx_stage_barrier<kHxWait>();
      });
    }
    if (st0 < s_end) {
      dx_static_for<0, kHxRing>([&](auto i_tag) {
        constexpr int i = decltype(i_tag)::value;
        const int st = st0 + i;
        if (st < s_end) {
          dma(st + kHxRing - 1, (i + kHxRing - 1) & (kHxRing - 1));
          if (st + 1 < s_end)
            decode_all(std::integral_constant<int, (i + 1) & (kHxRing - 1)>{},
                       std::integral_constant<int, (i + 1) & 1>{}, st + 1);
          mma_only(i_tag, std::integral_constant<int, i & 1>{});
          dx_stage_barrier<kHxWait>();
        }
      });
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();

    // ---- write: lane holds column l32 of each block, rows 8 (i/4) + 4 h +
    // i%4; dX = acc * 2^-(e[m] + t)
    const int32_t* rxv = reinterpret_cast<const int32_t*>(lds + rx);
    const int kleft = (int)(K - k0 - wk * 128 - l32);
    const uint32_t lane_off = (uint32_t)(4 * h) * (uint32_t)K + (uint32_t)l32;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int rowa = wm * 128 + 32 * a;
      const int mleft = rows - rowa - 4 * h;
      float* pa = dX + (m0 + rowa) * K + k0 + wk * 128;
      int ex[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int dm = 8 * (i / 4) + (i % 4);
        const int r = rowa + 4 * h + dm;
        ex[i] = -(rxv[r < kHxTM ? r : kHxTM - 1] + tsc);
      }
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (kleft <= 32 * b) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int dm = 8 * (i / 4) + (i % 4);
          if (dm < mleft) {
            float* q = pa + 32 * b + (uint32_t)dm * (uint32_t)K + lane_off;
            const float v = ldexpf(acc[a][b][i], ex[i]);
            if (whole)
              *q = v;
            else
              atomicAdd(q, v);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

hipError_t launch_tgemm_bwd_dx_f16(const uint16_t* dY, const uint8_t* codes, const float* scales,
                                   int64_t M, int64_t N, int64_t K, int g, float* dX,
                                   void* workspace, hipStream_t stream) {
  auto up = [](int64_t v) { return (v + 255) / 256 * 256; };
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint16_t* dY16 = reinterpret_cast<uint16_t*>(ws);
  int32_t* rexp = reinterpret_cast<int32_t*>(ws + up(M * N * 2));
  uint32_t* sparts = reinterpret_cast<uint32_t*>(ws + up(M * N * 2) + up(M * 4));
  const int cus = current_cu_count();

  // prepass: up to 16 waves per CU, whole rows per wave
  {
    const int64_t waves_cap = (int64_t)cus * 16;
    int64_t waves = M < waves_cap ? M : waves_cap;
    if (waves < kScaleParts) waves = kScaleParts;  // the scale slices need kScaleParts
    const int64_t blocks = (waves + 3) / 4;
    hipLaunchKernelGGL(dx_prep_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dY, scales,
                       M, N, N * (K / g), dY16, rexp, sparts, kScaleParts);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const int64_t tm = (M + kHxTM - 1) / kHxTM, tk = (K + kHxTK - 1) / kHxTK;
  const int64_t ntiles = tm * tk;
  const int64_t P = ntiles < cus ? ntiles : cus;
  const int64_t rem = ntiles % P;
  int64_t parts = rem ? P / rem : 1;
  const int64_t nst = (N + kHxBN - 1) / kHxBN;
  if (parts > nst) parts = nst;
  if (rem) {
    const hipError_t e = launch_zero_tiles_f32(dX, M, K, tk, ntiles - rem, rem, stream);
    if (e != hipSuccess) return e;
  }
  const auto* cw = reinterpret_cast<const uint32_t*>(codes);
  const dim3 grid((unsigned)P), block(256);
  const uint32_t t_k = (uint32_t)tk, nt = (uint32_t)ntiles, pa = (uint32_t)parts;
  const int np = kScaleParts;
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemm_bwd_dx_f16_kernel<32>, grid, block, 0, stream, dY16, rexp, sparts, np, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 64:  hipLaunchKernelGGL(tgemm_bwd_dx_f16_kernel<64>, grid, block, 0, stream, dY16, rexp, sparts, np, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 128: hipLaunchKernelGGL(tgemm_bwd_dx_f16_kernel<128>, grid, block, 0, stream, dY16, rexp, sparts, np, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 256: hipLaunchKernelGGL(tgemm_bwd_dx_f16_kernel<256>, grid, block, 0, stream, dY16, rexp, sparts, np, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 512: hipLaunchKernelGGL(tgemm_bwd_dx_f16_kernel<512>, grid, block, 0, stream, dY16, rexp, sparts, np, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
