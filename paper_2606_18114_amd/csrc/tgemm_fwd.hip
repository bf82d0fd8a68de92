// Ternary forward GEMM (paper Sec. 3.1): Y[M, N] = X[M, K] . What[N, K]^T,
// What = s * q, on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// Persistent kernel: one workgroup of 8 waves per CU walks 256 x 256 output
// tiles (2 x 4 waves, 128 x 64 outputs per wave).  Consecutive tiles of one
// round go to the same XCD, so its workgroups share the rows of X through
// that XCD's L2.  Tiles left over after the whole rounds (fewer than one
// per workgroup) are cut along K into parts, one per workgroup, which add
// their partial sums into Y with float32 atomics (those rows of Y are
// cleared by a fill kernel first).  Without the cut, a shape with a few
// tiles more than workgroups would take two full rounds; with it the last
// round is spread over all CUs (2048 tokens of in_proj: 27% faster).
//
// Operands reach LDS by direct-to-LDS loads (global_load_lds), with no
// register staging and one barrier per 64-column stage.  The stage stream
// runs straight across tile boundaries, so the next tile's first stages load
// while the current tile finishes and writes Y.
//   * X: a 3-deep ring of 256 x 64 stages, loaded two stages ahead.  The
//     eight 16-byte pieces of row r are stored XOR-permuted by fwd_xswz(r),
//     which keeps the 32-row MFMA operand reads free of bank conflicts.
//   * codes and group scales: a weight row holds only 16 bytes of codes per
//     stage, so loading them per stage would cost one memory request per
//     16 bytes.  When K is a multiple of 256 they are loaded in code stages of
//     four X stages (64 bytes of codes per row, the scales of every group
//     starting in those 256 columns) into a 2-deep ring, one code stage
//     ahead; otherwise per stage into a 3-deep ring, two stages ahead.
//   * Every lane decodes the codes of its own weight row into the MFMA B
//     operand, giving the exact bfloat16 values 2*q; the words of its two
//     rows are decoded together (four 64-bit shifts and eight ANDs per 16
//     codes).
//   * The group scale is applied in float32, not folded into the bfloat16
//     operand (folding would cost about 2e-3 relative error).  Instead of a
//     second set of partial accumulators, each accumulator is kept in units
//     of the current group's scale c: when the next group (scale s) starts,
//     every accumulator block is multiplied by c / s just before its first
//     MFMA of that group and c becomes s, so the matrix cores keep adding
//     exact products into one register set.  At the end Y = c * acc / 2.
//     Groups with s = 0 are masked out of the operand.
//
// Synchronisation: the direct-to-LDS loads are issued from inline assembly,
// so the compiler neither tracks them nor inserts waits of its own for them
// (its LDS-DMA tracking would otherwise wait for every load in flight before
// each LDS read).  Each wave issues a fixed number of them per stage and no
// other vector-memory loads.  At the end of every stage a wave waits until
// only the loads issued after the ones the next stage needs are in flight
// (vector-memory operations retire in order) and its LDS reads are done; the
// barrier then publishes the next stage to all waves and frees the slots read
// in this one.  Y stores issued in between only make that wait stricter.
#include <type_traits>

#include "common.hpp"
#include "launchers.hpp"

namespace tmk {

constexpr int kFwdBM = 256, kFwdBN = 256, kFwdBK = 64;
constexpr int kFwdXRing = 3;
// polls of a cut tile's flag before the second part gives up waiting (the
// first part is already storing when the second starts to wait; this bound
// only keeps every wave's exit certain)
constexpr uint32_t kFwdSpinLimit = 1u << 20;
// fewest cut tiles for which the two parts meet through the tickets
constexpr int64_t kFwdMinTicketTiles = 16;
constexpr int kFwdXStage = kFwdBM * kFwdBK * 2;  // 32 KiB of X per stage

// SS: X stages per code stage (4 when K % 256 == 0, else 1)
template <int G, int SS>
struct FwdCfg {
  static constexpr int kNs = SS == 1 ? 2 : (256 / G > 2 ? 256 / G : 2);  // scales per row
  static constexpr int kCRing = SS == 1 ? 3 : 2;
  static constexpr int kCStage = kFwdBN * 16 * SS;  // code bytes per code stage
  static constexpr int kSStage = kFwdBN * kNs * 4;  // scale bytes per code stage
  static constexpr int kCBase = kFwdXRing * kFwdXStage;
  static constexpr int kSBase = kCBase + kCRing * kCStage;
  static constexpr int kLds = kSBase + kCRing * kSStage;
  static constexpr int kScaleDma = SS == 1 ? 1 : kNs / 2;  // per wave per code stage
  static constexpr int kNc = 2 + kScaleDma;                // code + scale loads per wave
  static constexpr int kUnroll = SS > G / kFwdBK ? SS : G / kFwdBK;  // stages per loop trip
  static_assert(kLds <= 160 * 1024, "LDS budget");
};

// 16-byte piece permutation of X row r inside its stage
__device__ __forceinline__ int fwd_xswz(int r) { return (r & 7) ^ ((r >> 3) & 1); }
// 16-byte chunk permutation of code row r inside a 4-stage code stage
__device__ __forceinline__ int fwd_cswz(int r) {
  return (((r >> 1) ^ (r >> 3)) & 1) | (((r >> 2) & 1) << 1);
}

// Direct-to-LDS loads: lane i of the wave reads 16 (4) bytes at base + voff
// and writes them to LDS byte address lds_base + 16 i (4 i).  base and
// lds_base are wave-uniform.  The instruction takes the LDS base from M0;
// one wait state separates the M0 write from the load.  M0 is a reserved
// register the compiler warns about clobbering; nothing else in this kernel
// uses it.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma_x16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
__device__ __forceinline__ void dma_x4(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

// End of a stage: at most kVm of this wave's loads still in flight, its LDS
// reads complete, then all waves meet.
template <int kVm>
__device__ __forceinline__ void fwd_stage_barrier() {
  __builtin_amdgcn_sched_barrier(0);  // keep each stage's work inside its stage
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kVm) : "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// BF: Y in bfloat16 (each float32 result rounded to nearest even once),
// else float32.  The bfloat16 form never cuts tiles (parts == 1).
template <int G, int SS, bool BF>
__global__ __launch_bounds__(512) void tgemm_fwd_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    void* __restrict__ Yv, uint32_t tiles_n, uint32_t full_rounds, uint32_t extra_units,
    uint32_t parts, uint32_t* __restrict__ tickets) {
  using C = FwdCfg<G, SS>;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[C::kLds];
  __shared__ uint32_t tk_word;  // arrival order of this workgroup at its cut tile

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave >> 2, wn = wave & 3;
  const uint32_t h = (uint32_t)(lane >> 5);  // k half of the MFMA operands
  const int l32 = lane & 31;
  const int nst = (int)(K / kFwdBK);
  const int64_t ng = K / G;
  const int64_t kb = K / 4;  // code bytes per weight row
  const uint32_t bid = xcd_remap(blockIdx.x, gridDim.x);
  const uint32_t nblk = gridDim.x;
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  // in-tile row offsets of the output fit 32 bits (131 rows of N floats)
  const bool small_pitch = N < (int64_t(1) << 22);

  // Work list of this workgroup: full_rounds whole tiles (tile r * nblk + bid
  // in round r) and, for bid < extra_units, one extra unit: part bid % parts
  // of tile full_rounds * nblk + bid / parts, a run of whole trips of its K
  // stages.  With parts > 1 the parts of a tile add into Y with atomics (Y
  // zeroed there beforehand), and odd parts come first: those workgroups
  // then run half a tile out of phase with the others, which spreads the
  // output stores over time instead of all workgroups storing at once.
  // With tickets (two parts per tile, Y not cleared): the part that reaches
  // its epilogue first (word 2t of the tickets, t the cut tile) writes its
  // sums into Y with coherent stores and then raises word 2t + 1; the second
  // waits for that word and adds its sums with atomics.  Two addends give the
  // same bits in either order, and only half the atomics.
  const uint32_t F = full_rounds;
  const bool has_x = bid < extra_units;
  const uint32_t nu = F + (has_x ? 1u : 0u);
  if (nu == 0) return;  // no work: before any load or barrier
  const uint32_t xp = has_x ? bid % parts : 0u;
  const bool x_first = has_x && parts > 1 && (xp & 1u);
  const int trips = nst / C::kUnroll;
  // unit u (units past the end repeat the last one: their loads are never
  // consumed, they only keep the count of loads per stage fixed): tile,
  // first and end stage, and whether it is a part of a tile
  auto unit_of = [&](uint32_t u, uint32_t& tile, int& s0, int& s1, bool& part) {
    u = u < nu ? u : nu - 1;
    const bool extra = has_x && (x_first ? u == 0 : u == F);
    if (extra) {
      tile = F * nblk + bid / parts;
      s0 = (int)(xp * (uint32_t)trips / parts) * C::kUnroll;
      s1 = (int)((xp + 1) * (uint32_t)trips / parts) * C::kUnroll;
      part = parts > 1;
    } else {
      tile = (x_first ? u - 1 : u) * nblk + bid;
      s0 = 0;
      s1 = nst;
      part = false;
    }
  };
  // rows of a tile; rows past M or N are clamped to the last one by the loaders
  auto tile_rows = [&](uint32_t tile, int64_t& m0, int64_t& n0) {
    m0 = (int64_t)(tile / tiles_n) * kFwdBM;
    n0 = (int64_t)(tile % tiles_n) * kFwdBN;
  };

  // ---- X loader: stage xst of unit xu, 4 loads of 1 KiB per wave ----
  uint32_t xu = 0;
  int xst = 0, xend = 0, xslot = 0;
  const uint8_t* xt = nullptr;
  uint32_t xoff[4];
  auto set_xunit = [&](uint32_t u) {
    uint32_t tile;
    bool part;
    int64_t m0, n0;
    unit_of(u, tile, xst, xend, part);
    tile_rows(tile, m0, n0);
    const int mlast = (int)(M - 1 - m0 < 255 ? M - 1 - m0 : 255);
    xt = reinterpret_cast<const uint8_t*>(X + m0 * K);
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // load I = rows 8I .. 8I+7
      const int r = 8 * (wave * 4 + i) + (lane >> 3);
      const int lp = (lane & 7) ^ fwd_xswz(r);  // logical piece this lane fetches
      xoff[i] = (uint32_t)(r < mlast ? r : mlast) * (uint32_t)K * 2u + 16u * lp;
    }
  };
  // kMayWrap: this call may issue the last stage of a unit (known at
  // compile time from the stage's position in the unrolled loop)
  auto dma_x = [&](auto may_wrap) {
    const uint8_t* base = xt + (int64_t)xst * kFwdBK * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      dma_x16(base, xoff[i], lds0 + xslot * kFwdXStage + 1024 * (wave * 4 + i));
    xslot = xslot == kFwdXRing - 1 ? 0 : xslot + 1;
    ++xst;
    if constexpr (decltype(may_wrap)::value) {
      if (xst == xend) set_xunit(++xu);
    }
  };

  // ---- code/scale loader: code stage starting at X stage cst of unit cu ----
  uint32_t cu = 0;
  int cst = 0, cend = 0, cslot = 0;
  const uint8_t *ct = nullptr, *stl = nullptr;
  uint32_t coff[2], soff[C::kScaleDma];
  auto set_cunit = [&](uint32_t u) {
    uint32_t tile;
    bool part;
    int64_t m0, n0;
    unit_of(u, tile, cst, cend, part);
    tile_rows(tile, m0, n0);
    const int nlast = (int)(N - 1 - n0 < 255 ? N - 1 - n0 : 255);
    ct = codes + n0 * kb;
    stl = reinterpret_cast<const uint8_t*>(scales + n0 * ng);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int J = wave * 2 + j;
      if constexpr (SS == 4) {  // load J = rows 16J .. 16J+15, 64 bytes each
        const int r = 16 * J + (lane >> 2);
        const int c = (lane & 3) ^ fwd_cswz(r);  // 16-byte chunk this lane fetches
        coff[j] = (uint32_t)(r < nlast ? r : nlast) * (uint32_t)kb + 16u * c;
      } else {  // load J = rows 16J .. 16J+15, 16 bytes each
        const int r = 16 * J + (lane >> 2);
        coff[j] = (uint32_t)(r < nlast ? r : nlast) * (uint32_t)kb + 4u * (lane & 3);
      }
    }
#pragma unroll
    for (int l = 0; l < C::kScaleDma; ++l) {  // kNs scales per row, kNs lanes per row
      const int L = wave * C::kScaleDma + l;
      const int r = (64 / C::kNs) * L + lane / C::kNs;
      const int q = lane % C::kNs;  // group within the code stage
      const bool real = SS == 4 ? G <= 128 : G == 32;  // otherwise a repeat of group 0
      soff[l] = ((uint32_t)(r < nlast ? r : nlast) * (uint32_t)ng + (real ? q : 0)) * 4u;
    }
  };
  auto dma_c = [&](auto may_wrap) {
    const int64_t k0 = (int64_t)cst * kFwdBK;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t dst = lds0 + C::kCBase + cslot * C::kCStage;
      if constexpr (SS == 4)
        dma_x16(ct + k0 / 4, coff[j], dst + 1024 * (wave * 2 + j));
      else
        dma_x4(ct + k0 / 4, coff[j], dst + 256 * (wave * 2 + j));
    }
#pragma unroll
    for (int l = 0; l < C::kScaleDma; ++l)
      dma_x4(stl + 4 * (k0 / G), soff[l],
             lds0 + C::kSBase + cslot * C::kSStage + 256 * (wave * C::kScaleDma + l));
    cslot = cslot == C::kCRing - 1 ? 0 : cslot + 1;
    cst += SS;
    if constexpr (decltype(may_wrap)::value) {
      if (cst == cend) set_cunit(++cu);
    }
  };

  // prologue: X stages 0 and 1, code stage 0 (and 1 when SS == 1); the
  // waits below count the loads issued after the ones the next stage needs
  const std::true_type wraps;
  set_xunit(0);
  set_cunit(0);
  dma_x(wraps);
  dma_c(wraps);
  dma_x(wraps);
  if constexpr (SS == 1) {
    dma_c(wraps);
    fwd_stage_barrier<4 + C::kNc>();
  } else {
    fwd_stage_barrier<4>();
  }

  const int xsw = fwd_xswz(l32);  // == fwd_xswz(m) for every X row m this lane reads
  const uint32_t hs = 8u - 8u * h;  // shift that moves this lane's code half to the top
  int xs = 0, cs = 0;             // ring slots of the stage being computed

  for (uint32_t u = 0; u < nu; ++u) {
    uint32_t tile;
    int s0, s1;
    bool part;
    int64_t m0, n0;
    unit_of(u, tile, s0, s1, part);
    tile_rows(tile, m0, n0);

    f32x16 acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;
    float cref[2] = {0.f, 0.f};
    uint32_t msk[2] = {0u, 0u};

    // One stage: P = its index inside the code stage, kStart = a group
    // starts at its first column.
    auto stage = [&](auto p_tag, auto start_tag) {
      constexpr int P = decltype(p_tag)::value;
      constexpr bool kStart = decltype(start_tag)::value;
      const uint8_t* xb = lds + xs * kFwdXStage;
      const uint8_t* cb = lds + C::kCBase + cs * C::kCStage;
      const uint8_t* sb = lds + C::kSBase + cs * C::kSStage;
      u32x4 cw[2];
      float sc[2][2];  // [b][q]: scales of the groups starting at step 0, step 2
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int nr = wn * 64 + b * 32 + l32;
        if constexpr (SS == 4) {
          // chunk P of row nr sits at P ^ fwd_cswz(nr) (== fwd_cswz(l32));
          // the opaque copy keeps the compiler from holding one address per P
          uint32_t sw = 16u * fwd_cswz(l32);
          asm volatile("" : "+v"(sw));
          cw[b] = *reinterpret_cast<const u32x4*>(cb + 64 * nr + ((16u * P) ^ sw));
        } else
          cw[b] = *reinterpret_cast<const u32x4*>(cb + 16 * nr);
        if constexpr (kStart) {
          if constexpr (G == 32) {  // groups 2P, 2P + 1 of the code stage
            const u32x2 v = *reinterpret_cast<const u32x2*>(sb + 4 * C::kNs * nr + 8 * P);
            sc[b][0] = __uint_as_float(v.x);
            sc[b][1] = __uint_as_float(v.y);
          } else {  // the group starting at this stage
            constexpr int q = SS == 4 && G <= 128 ? P * kFwdBK / G : 0;
            sc[b][0] = *reinterpret_cast<const float*>(sb + 4 * C::kNs * nr + 4 * q);
            sc[b][1] = sc[b][0];
          }
        }
      }
      auto read_a = [&](int t, bf16x8* ao) {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int m = wm * 128 + a * 32 + l32;
          ao[a] = as_bf16x8(*reinterpret_cast<const u32x4*>(
              xb + 128 * m + 16 * ((2 * t + (int)h) ^ xsw)));
        }
      };
      bf16x8 acur[4];
      read_a(0, acur);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bool start = kStart && (G == 32 ? (t % 2) == 0 : t == 0);
        float r[2] = {1.f, 1.f};
        if (start) {
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const float sv = sc[b][t / 2];
            const bool nz = sv != 0.f;
            msk[b] = nz ? 0xFFFFFFFFu : 0u;
            const float ratio = cref[b] * __builtin_amdgcn_rcpf(nz ? sv : 1.f);
            r[b] = (nz && cref[b] != 0.f) ? ratio : 1.f;
            cref[b] = nz ? sv : cref[b];
          }
        }
        bf16x8 bop[2];
        decode_half_pair_rt(u32x2{cw[0][t] & msk[0], cw[1][t] & msk[1]}, hs, bop[0], bop[1]);
        bf16x8 anext[4];
        if (t < 3) read_a(t + 1, anext);
#pragma unroll
        for (int a = 0; a < 4; ++a) {
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            if (start) acc[a][b] *= r[b];
            acc[a][b] = mfma32(acur[a], bop[b], acc[a][b]);
          }
        }
        if (t < 3) {
#pragma unroll
          for (int a = 0; a < 4; ++a) acur[a] = anext[a];
        }
      }
    };

    // kUnroll stages per trip: a whole number of code stages and of groups
    for (int st = s0; st < s1; st += C::kUnroll) {
      static_for<0, C::kUnroll>([&](auto i_tag) {
        constexpr int i = decltype(i_tag)::value;
        constexpr int P = i % SS;
        constexpr bool kStart = G <= kFwdBK || (i * kFwdBK) % G == 0;
        // units are whole trips, so only these positions move a cursor
        // past the end of a unit: the X cursor (stage st + i + 2
        // issued, st + i + 3 next) and the code cursor (code stage starting
        // at st + i + 4 issued, st + i + 8 next; with SS == 1 like X)
        constexpr int kCAhead = SS == 1 ? 3 : 2 * SS;
        dma_x(std::integral_constant<bool, (i + 3) % C::kUnroll == 0>{});
        if constexpr (P == 0)
          dma_c(std::integral_constant<bool, (i + kCAhead) % C::kUnroll == 0>{});
        stage(std::integral_constant<int, P>{}, std::integral_constant<bool, kStart>{});
        if constexpr (SS == 1 || P < 2)
          fwd_stage_barrier<4 + C::kNc>();
        else
          fwd_stage_barrier<4>();
        xs = xs == kFwdXRing - 1 ? 0 : xs + 1;
        if constexpr (SS == 1)
          cs = xs;
        else if constexpr (P == SS - 1)
          cs ^= 1;
      });
    }

    // epilogue: lane holds column l32 of each block, rows 8*(i/4) + 4*h + i%4.
    // Row offsets inside the tile are compile-time multiples of the row
    // pitch, so a store costs one address add; tiles wholly inside M skip
    // the row test (rows past M only occur in the last row of tiles).  Parts
    // of a tile add their partial sums with float32 atomics.
    {
      const int64_t mrow = m0 + wm * 128;
      constexpr int ES = BF ? 2 : 4;  // bytes per output element
      // two-part cut tile with tickets: which part arrives first
      const bool tk = !BF && part && tickets != nullptr;
      const uint32_t tkt = 2u * (bid / parts);
      bool tk_second = false;
      if (tk) {
        __syncthreads();
        if (threadIdx.x == 0) {
          const uint32_t order = atomicAdd(tickets + tkt, 1u);
          if (order != 0u) {
            // the first part is already in its epilogue: wait (bounded) until
            // its sums have reached memory
            for (uint32_t n = 0; n < kFwdSpinLimit; ++n) {
              if (__hip_atomic_load(tickets + tkt + 1, __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT) != 0u)
                break;
              __builtin_amdgcn_s_sleep(2);
            }
          }
          tk_word = order;
        }
        __syncthreads();
        tk_second = tk_word != 0u;
      }
      uint8_t* ytile = reinterpret_cast<uint8_t*>(Yv) + (mrow * N + n0) * ES;
      const bool full_m = mrow + 128 <= M;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int nl = wn * 64 + b * 32 + l32;  // column in the tile
        if (n0 + nl >= N) continue;
        const float f = 0.5f * cref[b];
        uint8_t* ylane = ytile + ((int64_t)(4 * h) * N + nl) * ES;
        if (!BF && part) {
          int64_t pv = N * 4;
          asm volatile("" : "+v"(pv));
          uint8_t* yp = ylane;
          int64_t row = mrow + 4 * h;
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
#pragma unroll
              for (int i1 = 0; i1 < 4; ++i1) {
                if (row < M) {
                  const float v = f * acc[a][b][4 * i4 + i1];
                  if (tk && !tk_second)  // first of two: write through to memory
                    __hip_atomic_store(reinterpret_cast<float*>(yp), v, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                  else
                    atomicAdd(reinterpret_cast<float*>(yp), v);
                }
                yp += pv;
                ++row;
              }
              yp += 4 * pv;
              row += 4;
            }
        } else if (small_pitch && full_m) {
          // a 32-bit lane offset from the uniform tile base, stepped row by
          // row (rows a*32 + 8*i4 + i1); the empty asm keeps the compiler
          // from precomputing all 64 offsets (which it would spill)
          uint32_t pv = (uint32_t)N * ES;
          asm volatile("" : "+v"(pv));
          const uint32_t pv4 = 4u * pv;
          uint32_t o = (uint32_t)((4 * h) * N + nl) * ES;
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
#pragma unroll
              for (int i1 = 0; i1 < 4; ++i1) {
                if constexpr (BF)
                  *reinterpret_cast<uint16_t*>(ytile + o) =
                      __builtin_bit_cast(uint16_t, (__bf16)(f * acc[a][b][4 * i4 + i1]));
                else
                  __builtin_nontemporal_store(f * acc[a][b][4 * i4 + i1],
                                              reinterpret_cast<float*>(ytile + o));
                o += pv;
              }
              o += pv4;  // rows 8 i4 + 4 .. 8 i4 + 7 belong to the other k half
            }
        } else {
          // rows past M (last row of tiles), or a pitch beyond 32-bit offsets
          int64_t pv = N * ES;
          asm volatile("" : "+v"(pv));
          uint8_t* yp = ylane;
          int64_t row = mrow + 4 * h;
#pragma unroll
          for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int i4 = 0; i4 < 4; ++i4) {
#pragma unroll
              for (int i1 = 0; i1 < 4; ++i1) {
                const float v = f * acc[a][b][4 * i4 + i1];
                if (row < M) {
                  if constexpr (BF)
                    *reinterpret_cast<uint16_t*>(yp) = __builtin_bit_cast(uint16_t, (__bf16)v);
                  else
                    *reinterpret_cast<float*>(yp) = v;
                }
                yp += pv;
                ++row;
              }
              yp += 4 * pv;
              row += 4;
            }
        }
      }
      if (tk && !tk_second) {
        // every wave's coherent stores have completed: raise the tile's flag
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (threadIdx.x == 0)
          __hip_atomic_store(tickets + tkt + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  // loads issued for stages past the end must land before the workgroup's
  // LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

hipError_t launch_tgemm_fwd(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int g, void* Y, bool bf16_out,
                            uint32_t* tickets, hipStream_t stream) {
  const int64_t tm = (M + kFwdBM - 1) / kFwdBM, tn = (N + kFwdBN - 1) / kFwdBN;
  const int64_t ntiles = tm * tn;
  const int cus = current_cu_count();
  const bool wide = K % 256 == 0;  // code stages of four X stages
  // Work split over P = cus persistent workgroups: F whole rounds of tiles,
  // then the R = ntiles mod P remaining tiles cut along K into `parts` runs
  // of whole trips (kUnroll stages), one per workgroup, when that leaves at
  // least two parts per tile; otherwise the remaining tiles go whole to the
  // first R workgroups.
  const int64_t P = cus;
  const int64_t F = ntiles / P, R = ntiles % P;
  const int unroll = (wide ? 4 : 1) > g / kFwdBK ? (wide ? 4 : 1) : g / kFwdBK;
  const int64_t trips = K / kFwdBK / unroll;
  int64_t parts = R > 0 ? P / R : 1;
  if (parts > trips) parts = trips;
  if (parts < 1 || bf16_out) parts = 1;  // bfloat16 results are not summed in parts
  const int64_t extra = R * parts;
  // two parts per cut tile and tickets given: the first part writes, the
  // second adds (Y is not cleared; the tickets are, by a fill kernel).  With
  // few cut tiles the atomics cost little and the second part's wait for the
  // first (which then finishes at about the same time) would show: atomics.
  if (parts != 2 || R < kFwdMinTicketTiles || R > kFwdMaxTicketTiles) tickets = nullptr;
  if (tickets) {
    hipError_t e = launch_fill_zero_f32(reinterpret_cast<float*>(tickets), 2 * R, stream);
    if (e != hipSuccess) return e;
  } else if (parts > 1) {
    // the cut tiles accumulate atomically: clear their rows of Y first (a
    // fill kernel, not a memset node, so the call can be captured)
    const int64_t r0 = F * P / tn * kFwdBM;
    hipError_t e = launch_fill_zero_f32(static_cast<float*>(Y) + r0 * N, (M - r0) * N, stream);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)P), block(512);
  const uint32_t t_n = (uint32_t)tn, fr = (uint32_t)F, xu = (uint32_t)extra,
                 np = (uint32_t)parts;
#define TM_FWD_L(GG, SS_, BF_)                                                                 \
  hipLaunchKernelGGL((tgemm_fwd_kernel<GG, SS_, BF_>), grid, block, 0, stream, X, codes, scales, \
                     M, N, K, Y, t_n, fr, xu, np, tickets)
#define TM_FWD(GG)                                                                             \
  case GG:                                                                                     \
    if (wide) {                                                                                \
      if (bf16_out)                                                                            \
        TM_FWD_L(GG, 4, true);                                                                 \
      else                                                                                     \
        TM_FWD_L(GG, 4, false);                                                                \
    } else {                                                                                   \
      if (bf16_out)                                                                            \
        TM_FWD_L(GG, 1, true);                                                                 \
      else                                                                                     \
        TM_FWD_L(GG, 1, false);                                                                \
    }                                                                                          \
    break;
  switch (g) {
    TM_FWD(32)
    TM_FWD(64)
    TM_FWD(128)
    TM_FWD(256)
    TM_FWD(512)
    default: return hipErrorInvalidValue;
  }
#undef TM_FWD
#undef TM_FWD_L
  return hipGetLastError();
}

}  // namespace tmk
