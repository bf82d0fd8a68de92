// Straight-through backward w.r.t. the input (paper Sec. 3.1):
//   dX[M, K] = dY[M, N] . What[N, K],  What = s * q,
// a contraction over N on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16),
// float32 accumulation.
//
// The scale varies along the contraction (one per weight row n and group),
// so it cannot be applied after the MFMA as in the forward kernel.  Folding
// it into one bfloat16 operand would cost about 2e-3 relative error; instead
// every dequantized weight is split exactly into two bfloat16 terms
// q*s_hi + q*s_lo, with s_hi = s truncated to bfloat16 and
// s_lo = bf16(s - s_hi) >= 0 (together 16 significant bits of s), and both
// terms run on the matrix cores against the same dY operand and accumulator.
//
// Tile: 256 (M) x 256 (K) outputs per workgroup of 4 waves (2 x 2), 128 x 128
// per wave (4 x 4 MFMA blocks, accumulators in AGPRs); the contraction
// advances 32 weight rows (n) per stage.  Per stage:
//   * dY [256 x 32] bf16, the packed codes [32 x 256] and the stage's scales
//     reach a 4-deep LDS ring by direct-to-LDS loads (global_load_lds) issued
//     three stages ahead.  The 64-byte dY rows have their four 16-byte units
//     XOR-permuted (dx_yoff), so the 16-byte operand reads are free of bank
//     conflicts on the 64-bank LDS;
//   * one stage ahead, all threads decode the codes into the two bfloat16
//     planes q*s_hi and q*s_lo [32 n][256 k] (double-buffered), in natural
//     order with the 32-byte units of each row XOR-permuted (dx_poff);
//   * an MFMA B operand (8 consecutive n of one column k) comes from a plane
//     by two gfx950 transpose reads ds_read_b64_tr_b16: in each group of 16
//     lanes, lane j passes the address of 4 columns of row j / 4 and lane i
//     receives one column of 4 consecutive rows.
//
// Work split (persistent, one workgroup per CU): the T output tiles are dealt
// round-robin, whole, T / P per workgroup; the T % P remaining tiles are each
// cut along the contraction into P / (T % P) parts that are added into dX
// (cleared first) with float32 atomics.
//
// The direct-to-LDS loads are issued from inline assembly, so the compiler
// neither tracks nor waits for them; each wave issues exactly seven per stage
// and counts them itself (vector-memory operations retire in order).
#include "dx_common.hpp"
#include "launchers.hpp"

namespace tmk {

constexpr int kDxTM = 256, kDxTK = 256, kDxBN = 32, kDxRing = 4;
constexpr int kDxY = kDxTM * kDxBN * 2;            // 16 KiB: dY tile of a stage
constexpr int kDxC = kDxBN * kDxTK / 4;            // 2 KiB: packed codes of a stage
constexpr int kDxS = 1024;                         // scales: <= 32 rows x 8 groups
constexpr int kDxSlot = kDxY + kDxC + kDxS;        // 19 KiB ring slot
constexpr int kDxPlane = kDxBN * kDxTK * 2;        // 16 KiB: one bfloat16 plane
constexpr int kDxDec = 2 * kDxPlane;               // hi plane, then lo plane
constexpr int kDxRingBase = 2 * kDxDec;            // planes first, then the ring
constexpr int kDxLds = kDxRingBase + kDxRing * kDxSlot;  // 140 KiB
constexpr int kDxLoads = 7;                        // direct-to-LDS loads per wave per stage

template <int G>
__global__ __launch_bounds__(256) void tgemm_bwd_dx_kernel(
    const uint16_t* __restrict__ dY, const uint32_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    float* __restrict__ dX, uint32_t tiles_k, uint32_t ntiles, uint32_t parts) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kDxLds];
  constexpr int kGpt = G < kDxTK ? kDxTK / G : 1;  // scale groups per tile row

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wk = wave & 1;  // 128-row (M) and 128-column (K) halves
  const int l32 = lane & 31;
  const int h = lane >> 5;
  const int g16 = lane >> 4;                // 16-lane group of the transpose reads
  const int j16 = lane & 15;
  const uint32_t P = gridDim.x;
  const uint32_t bid = xcd_remap(blockIdx.x, P);
  const uint32_t full = ntiles / P;
  const uint32_t rem = ntiles % P;
  const int nst = (int)((N + kDxBN - 1) / kDxBN);
  const int64_t kw = K / 16;                // code words per weight row
  const int64_t ng = K / G;                 // scale groups per weight row
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;

  // transpose-read address of this lane inside a plane: rows trow .. (+16 t,
  // +4 for the second read), the 16 columns of its group
  const int trow = 8 * (g16 >> 1) + (j16 >> 2);
  const int tcol = 16 * (g16 & 1) + 4 * (j16 & 3);
  uint32_t boff[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) boff[b] = dx_poff(trow, wk * 128 + 32 * b + tcol);
  // 16-byte dY operand reads: row ar (+32 a), unit 2 t + h
  const int ar = wm * 128 + l32;
  const uint32_t aoff0 = dx_yoff(ar, h), aoff1 = dx_yoff(ar, 2 + h);

  // decode role: weight row dr of the stage, code words 2 dj and 2 dj + 1
  // (columns 32 dj .. 32 dj + 31, one scale group since G >= 32)
  const int dr = tid >> 3, dj = tid & 7;
  // lanes with dj >= 4 write the two 16-byte halves of each 32-byte unit in
  // the opposite order, so that the 16 lanes of a plane write cover 16
  // distinct 16-byte bank groups; they decode a code word whose byte pairs
  // are swapped (pairs 4-7 first), so both orders use the same registers
  const uint32_t hsel = (uint32_t)(dj >> 2);
  const uint32_t dswap = hsel ? 0x02030001u : 0x03020100u;
  const uint32_t dcode = kDxY + dr * 64 + 8 * dj;
  const uint32_t dscale = kDxY + kDxC + 4 * (dr * kGpt + (32 * dj) / G);
  const uint32_t dplane = dx_poff(dr, 32 * dj);  // word 2 dj + 1 is at dplane ^ 32

  for (uint32_t item = 0;; ++item) {
    // ---- the item: a whole tile, or one contraction range of a remaining tile
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
    const int64_t m0 = (int64_t)(tile / tiles_k) * kDxTM;
    const int64_t k0 = (int64_t)(tile % tiles_k) * kDxTK;
    const int rows = (int)(M - m0 < kDxTM ? M - m0 : kDxTM);

    // ---- loader.  dY: load i of a wave fills LDS rows 16 (4 wave + i) ..
    // +15, lane -> row + lane / 4, physical unit lane % 4 holding logical
    // unit u; rows past M re-read row M - 1 (those outputs are not stored).
    uint32_t yrow[4], ycol[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * (4 * wave + i) + (lane >> 2);
      const int u = (lane & 3) ^ ((r >> 1) & 3) ^ ((r >> 3) & 1);
      const int rr = r < rows ? r : rows - 1;
      yrow[i] = (uint32_t)rr * (uint32_t)N * 2u;
      ycol[i] = 8u * (uint32_t)u;
    }
    // codes: load i fills words 64 (2 wave + i) + lane = [row][word] of the
    // stage; words past the row end re-read its last word (columns past K are
    // not stored)
    int crow[2];
    uint32_t cword[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int idx = 64 * (2 * wave + i) + lane;
      crow[i] = idx >> 4;
      const int64_t wd = k0 / 16 + (idx & 15);
      cword[i] = (uint32_t)(wd < kw ? wd : kw - 1);
    }
    // scales: entry 64 wave + lane = [row][group] of the stage (entries past
    // 32 kGpt re-read the last one into the unused part of the slot)
    int srow;
    uint32_t sgrp;
    {
      int idx = 64 * wave + lane;
      idx = idx < 32 * kGpt ? idx : 32 * kGpt - 1;
      srow = idx / kGpt;
      const int64_t gg = k0 / G + idx % kGpt;
      sgrp = (uint32_t)(gg < ng ? gg : ng - 1);
    }
    const uint8_t* ybase = reinterpret_cast<const uint8_t*>(dY + m0 * N);

    // The loads of one stage, issued in seven pieces: dY rows (pieces 0-3),
    // codes (4-5), scales (6).
    struct DmaStage {
      const uint32_t* cb;
      const float* sbp;
      uint32_t ncol, dst;
      int nlast;
    };
    auto dma_begin = [&](int st, int slot) {
      st = st < s_end ? st : s_end - 1;  // past the range: reload its last stage
      const int64_t nb = (int64_t)st * kDxBN;
      DmaStage d;
      d.dst = lds0 + kDxRingBase + slot * kDxSlot;
      d.ncol = (uint32_t)nb;
      d.nlast = (int)(N - 1 - nb);  // weight rows past N re-read row N - 1
      d.cb = codes + nb * kw;
      d.sbp = scales + nb * ng;
      return d;
    };
    auto dma_piece = [&](const DmaStage& d, auto i_tag) {
      constexpr int i = decltype(i_tag)::value;
      if constexpr (i < 4) {
        // columns past N re-read the last unit (those weight rows decode to 0)
        const uint32_t ncap = (uint32_t)N - 8u;
        uint32_t c = d.ncol + ycol[i];
        c = c < ncap ? c : ncap;
        dx_dma16(ybase, yrow[i] + 2u * c, d.dst + 1024 * (4 * wave + i));
      } else if constexpr (i < 6) {
        const int r = crow[i - 4] < d.nlast ? crow[i - 4] : d.nlast;
        dx_dma4(d.cb, ((uint32_t)r * (uint32_t)kw + cword[i - 4]) * 4u,
                d.dst + kDxY + 256 * (2 * wave + (i - 4)));
      } else {
        const int r = srow < d.nlast ? srow : d.nlast;
        dx_dma4(d.sbp, ((uint32_t)r * (uint32_t)ng + sgrp) * 4u,
                d.dst + kDxY + kDxC + 256 * wave);
      }
    };
    auto dma = [&](int st, int slot) {
      const DmaStage d = dma_begin(st, slot);
      dx_static_for<0, kDxLoads>([&](auto i_tag) { dma_piece(d, i_tag); });
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

    // Decode inputs of stage st from ring slot SLOT: two code words (rows
    // past N read as 0) and the scale split into bfloat16 pairs s_hi, s_lo
    // (s_hi truncated, so s_lo >= 0; s_lo rounded to nearest).  Read and
    // split are separate steps so that the split can wait under the MFMAs.
    struct DecIn {
      u32x2 w;
      float s;
      uint32_t hi2, lo2;
    };
    auto decode_read = [&](auto slot_tag) {
      constexpr int SLOT = decltype(slot_tag)::value;
      const uint8_t* sb = lds + kDxRingBase + SLOT * kDxSlot;
      DecIn d;
      d.w = *reinterpret_cast<const u32x2*>(sb + dcode);
      d.s = *reinterpret_cast<const float*>(sb + dscale);
      return d;
    };
    auto decode_split = [&](DecIn& d, int st) {
      if ((int64_t)st * kDxBN + dr >= N) d.w = u32x2{0u, 0u};
      d.w.x = __builtin_amdgcn_perm(d.w.x, d.w.x, dswap);
      d.w.y = __builtin_amdgcn_perm(d.w.y, d.w.y, dswap);
      const uint32_t sbits = __builtin_bit_cast(uint32_t, d.s) & 0xFFFF0000u;
      const float rest = d.s - __builtin_bit_cast(float, sbits);
      const uint32_t rb = __builtin_bit_cast(uint32_t, rest);
      const uint32_t lo = (rb + 0x7FFFu + ((rb >> 16) & 1u)) >> 16;
      d.hi2 = sbits | (sbits >> 16);
      d.lo2 = lo | (lo << 16);
    };
    auto decode_in = [&](auto slot_tag, int st) {
      DecIn d = decode_read(slot_tag);
      decode_split(d, st);
      return d;
    };
    // Pair I of both words: w << (14 - 2 I) holds the two codes at bits
    // 14-15 / 30-31, w << (15 - 2 I) their low bits at bits 15 / 31; a
    // nonzero code (low bit set) selects the scale, its high bit flips the
    // sign (so negative scales work too).
    // vh / vl: [word 0 elements 0-7, 8-15, word 1 elements 0-7, 8-15]
    auto decode_pair = [&](auto i_tag, const DecIn& d, u32x4* vh, u32x4* vl) {
      constexpr int I = decltype(i_tag)::value;
      const uint32_t sg0 = (d.w.x << (14 - 2 * I)) & 0x80008000u;
      const uint32_t sg1 = (d.w.y << (14 - 2 * I)) & 0x80008000u;
      const uint32_t nz0 = dx_halfmask(d.w.x << (15 - 2 * I));
      const uint32_t nz1 = dx_halfmask(d.w.y << (15 - 2 * I));
      vh[I / 4][I % 4] = (nz0 & d.hi2) ^ sg0;
      vl[I / 4][I % 4] = (nz0 & d.lo2) ^ sg0;
      vh[2 + I / 4][I % 4] = (nz1 & d.hi2) ^ sg1;
      vl[2 + I / 4][I % 4] = (nz1 & d.lo2) ^ sg1;
    };
    // the same for one word (W = 0, 1) of pair I
    auto decode_word_pair = [&](auto i_tag, auto w_tag, const DecIn& d, u32x4* vh, u32x4* vl) {
      constexpr int I = decltype(i_tag)::value;
      constexpr int W = decltype(w_tag)::value;
      const uint32_t w = W ? d.w.y : d.w.x;
      const uint32_t sg = (w << (14 - 2 * I)) & 0x80008000u;
      const uint32_t nz = dx_halfmask(w << (15 - 2 * I));
      vh[2 * W + I / 4][I % 4] = (nz & d.hi2) ^ sg;
      vl[2 * W + I / 4][I % 4] = (nz & d.lo2) ^ sg;
    };
    // plane writes of register half H of both words (elements 8 H .. 8 H + 7,
    // or 8 (1 - H) .. for the lanes that decode swapped words)
    auto decode_out = [&](auto plane_tag, int H, const u32x4* vh, const u32x4* vl) {
      constexpr int PL = decltype(plane_tag)::value;
      uint8_t* pb = lds + PL * kDxDec;
      const uint32_t o = dplane + 16 * ((uint32_t)H ^ hsel);
      st16(pb + o, vh[H]);
      st16(pb + (o ^ 32), vh[2 + H]);
      st16(pb + kDxPlane + o, vl[H]);
      st16(pb + kDxPlane + (o ^ 32), vl[2 + H]);
    };

    // One stage in ring slot I % kDxRing, planes I % 2: run the 64 MFMAs of
    // stage st, decode stage st + 1 into the other plane buffer and issue the
    // loads of stage st + 3.  A single wave issues about one instruction per
    // MFMA-pass group, so the order is fixed by hand, one MFMA per slot fenced
    // by sched_barrier, with the other work spread over the slots: the decode
    // inputs and the first 16-row step's operands are read up front; slot 2
    // splits the scale; the even slots 4 .. 34 each decode one word-pair; the
    // odd slots 5 .. 27 each read one operand of the second step; slots 20 ..
    // 23 and 36 .. 39 write the planes; slots 40 .. 46 issue the loads.
    auto stage = [&](auto i_tag, int st) {
      constexpr int I = decltype(i_tag)::value;
      constexpr int SLOT = I & (kDxRing - 1), PL = I & 1;
      constexpr int DSLOT = (I + 1) & (kDxRing - 1), DPL = (I + 1) & 1;
      const uint8_t* yb = lds + kDxRingBase + SLOT * kDxSlot;
      const uint8_t* pb = lds + PL * kDxDec;
      uint8_t* qb = lds + DPL * kDxDec;
      // reads in the order of first use (LDS reads complete in order)
      // (past the range this decodes a reloaded stage into the idle planes)
      DecIn din = decode_read(std::integral_constant<int, DSLOT>{});
      __builtin_amdgcn_sched_barrier(0);
      u32x4 af[2][4], bh[2][4], bl[2][4];
      af[0][0] = *reinterpret_cast<const u32x4*>(yb + aoff0);
      bh[0][0] = frag(pb, boff[0], 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 1; b < 4; ++b) bh[0][b] = frag(pb, boff[b], 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 0; b < 4; ++b) bl[0][b] = frag(pb + kDxPlane, boff[b], 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int a = 1; a < 4; ++a) af[0][a] = *reinterpret_cast<const u32x4*>(yb + aoff0 + 2048 * a);
      __builtin_amdgcn_sched_barrier(0);
      u32x4 vh[4], vl[4];
      DmaStage dst;
      dx_static_for<0, 64>([&](auto k_tag) {
        constexpr int k = decltype(k_tag)::value;
        constexpr int t = k / 32, c = (k % 32) / 8, j = k % 8, b = j % 4;
        if constexpr (j < 4)
          acc[c][b] = mfma32(as_bf16x8(af[t][c]), as_bf16x8(bh[t][b]), acc[c][b]);
        else
          acc[c][b] = mfma32(as_bf16x8(af[t][c]), as_bf16x8(bl[t][b]), acc[c][b]);
        if constexpr (k == 2) decode_split(din, st + 1);
        if constexpr (k >= 4 && k <= 34 && k % 2 == 0)
          decode_word_pair(std::integral_constant<int, (k - 4) / 4>{},
                           std::integral_constant<int, ((k - 4) / 2) % 2>{}, din, vh, vl);
        if constexpr (k >= 5 && k <= 27 && k % 2 == 1) {
          constexpr int x = (k - 5) / 2;  // 0 .. 11
          if constexpr (x < 4)
            bh[1][x] = frag(pb, boff[x], 1);
          else if constexpr (x < 8)
            bl[1][x - 4] = frag(pb + kDxPlane, boff[x - 4], 1);
          else
            af[1][x - 8] = *reinterpret_cast<const u32x4*>(yb + aoff1 + 2048 * (x - 8));
        }
        if constexpr ((k >= 20 && k < 24) || (k >= 36 && k < 40)) {
          // register half H of word `word` (pairs 0-3 are complete by slot
          // 18, pairs 4-7 by slot 34)
          constexpr int x = k < 24 ? k - 20 : k - 36;
          constexpr int H = k < 24 ? 0 : 1, word = x % 2;
          const uint32_t off = (dplane + 16 * ((uint32_t)H ^ hsel)) ^ (word ? 32u : 0u);
          if constexpr (x < 2)
            st16(qb + off, vh[2 * word + H]);
          else
            st16(qb + kDxPlane + off, vl[2 * word + H]);
        }
        if constexpr (k == 39)
          dst = dma_begin(st + kDxRing - 1, (I + kDxRing - 1) & (kDxRing - 1));
        if constexpr (k >= 40 && k < 40 + kDxLoads)
          dma_piece(dst, std::integral_constant<int, k - 40>{});
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    // decode-only step (prologue) and MFMA-only step (last stages)
    auto decode_all = [&](auto slot_tag, auto plane_tag, int st) {
      const DecIn din = decode_in(slot_tag, st);
      u32x4 vh[4], vl[4];
      dx_static_for<0, 8>([&](auto i_tag) { decode_pair(i_tag, din, vh, vl); });
      decode_out(plane_tag, 0, vh, vl);
      decode_out(plane_tag, 1, vh, vl);
    };
    auto mma_only = [&](auto slot_tag, auto plane_tag) {
      constexpr int SLOT = decltype(slot_tag)::value;
      constexpr int PL = decltype(plane_tag)::value;
      const uint8_t* yb = lds + kDxRingBase + SLOT * kDxSlot;
      const uint8_t* pb = lds + PL * kDxDec;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        u32x4 af[4], bh[4], bl[4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
          af[a] = *reinterpret_cast<const u32x4*>(yb + (t ? aoff1 : aoff0) + 2048 * a);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          bh[b] = frag(pb, boff[b], t);
          bl[b] = frag(pb + kDxPlane, boff[b], t);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            acc[a][b] = mfma32(as_bf16x8(af[a]), as_bf16x8(bh[b]), acc[a][b]);
            acc[a][b] = mfma32(as_bf16x8(af[a]), as_bf16x8(bl[b]), acc[a][b]);
          }
      }
    };

    // prologue: stages s_beg .. s_beg + 2 in flight, s_beg decoded
#pragma unroll
    for (int p = 0; p < kDxRing - 1; ++p) dma(s_beg + p, p);
    dx_stage_barrier<kDxLoads>();
    decode_all(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, s_beg);
    dx_stage_barrier<kDxLoads>();

    // groups of kDxRing stages
    int st0 = s_beg;
    for (; st0 + kDxRing <= s_end; st0 += kDxRing) {
      dx_static_for<0, kDxRing>([&](auto i_tag) {
        stage(i_tag, st0 + decltype(i_tag)::value);
        dx_stage_barrier<kDxLoads>();
      });
    }
    if (st0 < s_end) {  // the last 1 .. kDxRing - 1 stages
      dx_static_for<0, kDxRing>([&](auto i_tag) {
        constexpr int i = decltype(i_tag)::value;
        const int st = st0 + i;
        if (st < s_end) {
          dma(st + kDxRing - 1, (i + kDxRing - 1) & (kDxRing - 1));
          if (st + 1 < s_end)
            decode_all(std::integral_constant<int, (i + 1) & (kDxRing - 1)>{},
                       std::integral_constant<int, (i + 1) & 1>{}, st + 1);
          mma_only(i_tag, std::integral_constant<int, i & 1>{});
          dx_stage_barrier<kDxLoads>();
        }
      });
    }
    // every load of this item has landed before the ring is reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();

    // ---- write: lane holds column l32 of each block, rows 8 (i/4) + 4 h + i%4
    const int kleft = (int)(K - k0 - wk * 128 - l32);  // column valid if > 32 b
    const uint32_t lane_off = (uint32_t)(4 * h) * (uint32_t)K + (uint32_t)l32;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int rowa = wm * 128 + 32 * a;
      const int mleft = rows - rowa - 4 * h;  // rows 8 (i/4) + i%4 valid if below
      float* pa = dX + (m0 + rowa) * K + k0 + wk * 128;  // uniform
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (kleft <= 32 * b) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int dm = 8 * (i / 4) + (i % 4);
          if (dm < mleft) {
            float* q = pa + 32 * b + (uint32_t)dm * (uint32_t)K + lane_off;
            if (whole)
              *q = acc[a][b][i];
            else
              atomicAdd(q, acc[a][b][i]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // one block's values live at a time
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

hipError_t launch_tgemm_bwd_dx(const uint16_t* dY, const uint8_t* codes, const float* scales,
                               int64_t M, int64_t N, int64_t K, int g, float* dX,
                               hipStream_t stream) {
  const int64_t tm = (M + kDxTM - 1) / kDxTM, tk = (K + kDxTK - 1) / kDxTK;
  const int64_t ntiles = tm * tk;
  const int cus = current_cu_count();
  const int64_t P = ntiles < cus ? ntiles : cus;
  const int64_t rem = ntiles % P;
  int64_t parts = rem ? P / rem : 1;
  const int64_t nst = (N + kDxBN - 1) / kDxBN;
  if (parts > nst) parts = nst;
  if (rem) {  // the cut tiles are summed with atomics
    const hipError_t e = launch_zero_tiles_f32(dX, M, K, tk, ntiles - rem, rem, stream);
    if (e != hipSuccess) return e;
  }
  const auto* cw = reinterpret_cast<const uint32_t*>(codes);
  const dim3 grid((unsigned)P), block(256);
  const uint32_t t_k = (uint32_t)tk, nt = (uint32_t)ntiles, pa = (uint32_t)parts;
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemm_bwd_dx_kernel<32>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 64:  hipLaunchKernelGGL(tgemm_bwd_dx_kernel<64>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 128: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<128>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 256: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<256>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    case 512: hipLaunchKernelGGL(tgemm_bwd_dx_kernel<512>, grid, block, 0, stream, dY, cw, scales, M, N, K, dX, t_k, nt, pa); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
