// Ternary forward GEMM (paper Sec. 3.1): Y[M, N] = X[M, K] . What[N, K]^T,
// What = s * q, on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// Persistent kernel: one workgroup of 8 waves per CU walks 256 x 256 output
// tiles (2 x 4 waves, 128 x 64 outputs per wave).  Consecutive tiles of one
// round go to the same XCD, so its workgroups share the rows of X through
// that XCD's L2.
//
// K advances 64 columns per stage through a 4-deep LDS ring filled by
// direct-to-LDS loads (global_load_lds): no register staging, one barrier per
// stage, loads issued three stages ahead.  The stage stream runs straight
// across tile boundaries, so the next tile's first stages load while the
// current tile finishes and writes Y.
//   * X stage: 256 rows x 128 bytes; the eight 16-byte pieces of row r are
//     stored XOR-permuted by fwd_swz(r), which makes the 32-row MFMA operand reads
//     bank-conflict free.
//   * code stage: 256 weight rows x 16 bytes (64 codes), plus the float32
//     scales of the (at most two) groups that start in the stage, 256 x 2.
//     Every lane decodes
//     the codes of its own weight row into the MFMA B operand, one shift and
//     one AND per two codes, giving the exact bfloat16 values 2*q.
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
// each LDS read).  Each wave issues exactly seven such loads per stage, and
// no other vector-memory loads.  At the end of stage j a wave waits until at
// most the fourteen loads of stages j+2 and j+3 are outstanding (vector-memory
// operations retire in order), i.e. its part of stage j+1 has landed, and
// until its LDS reads are done; the barrier then publishes stage j+1 to all
// waves and frees the slot of stage j for stage j+4.  Y stores issued in
// between only make that wait stricter.
#include <type_traits>

#include "common.hpp"

namespace tmk {

constexpr int kFwdBM = 256, kFwdBN = 256, kFwdBK = 64, kFwdRing = 4;
constexpr int kFwdXStage = kFwdBM * kFwdBK * 2;  // 32 KiB of X per stage
constexpr int kFwdCStage = kFwdBN * kFwdBK / 4;  // 4 KiB of codes per stage
constexpr int kFwdSStage = kFwdBN * 2 * 4;       // 2 KiB of scales per stage
constexpr int kFwdCBase = kFwdRing * kFwdXStage;
constexpr int kFwdSBase = kFwdCBase + kFwdRing * kFwdCStage;
constexpr int kFwdLds = kFwdSBase + kFwdRing * kFwdSStage;  // 152 KiB

// 16-byte piece permutation of X row r inside its stage
__device__ __forceinline__ int fwd_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

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

// end of a stage: this wave's loads of the next stage have landed (at most
// the 14 loads of the two stages after it are in flight) and its LDS reads
// are complete; then all waves meet
__device__ __forceinline__ void fwd_stage_barrier() {
  asm volatile("s_waitcnt vmcnt(14) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int G>
__global__ __launch_bounds__(512) void tgemm_fwd_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ codes,
    const float* __restrict__ scales, int64_t M, int64_t N, int64_t K,
    float* __restrict__ Y, uint32_t tiles_n, uint32_t ntiles) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kFwdLds];

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

  // ---- the seven direct-to-LDS loads of one stage ----
  // Cursor: the stage (ait, ast) whose loads are issued next, its tile's
  // uniform base pointers and this lane's byte offsets inside the tile (rows
  // past M or N are clamped to the last one).  Rounds past the last tile
  // reload the last tile; those loads are never consumed, they only keep the
  // count per stage fixed.
  int ait = 0, ast = 0;
  const uint8_t *xt = nullptr, *ct = nullptr, *stl = nullptr;
  uint32_t xoff[4], coff[2], soff;
  auto set_tile = [&](int it) {
    uint32_t tile = (uint32_t)it * nblk + bid;
    tile = tile < ntiles ? tile : ntiles - 1;
    const int64_t m0 = (int64_t)(tile / tiles_n) * kFwdBM;
    const int64_t n0 = (int64_t)(tile % tiles_n) * kFwdBN;
    const int mlast = (int)(M - 1 - m0 < 255 ? M - 1 - m0 : 255);
    const int nlast = (int)(N - 1 - n0 < 255 ? N - 1 - n0 : 255);
    xt = reinterpret_cast<const uint8_t*>(X + m0 * K);
    ct = codes + n0 * kb;
    stl = reinterpret_cast<const uint8_t*>(scales + n0 * ng);
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // X load I = rows 8I .. 8I+7
      const int r = 8 * (wave * 4 + i) + (lane >> 3);
      const int lp = (lane & 7) ^ fwd_swz(r);  // logical piece this lane fetches
      xoff[i] = (uint32_t)(r < mlast ? r : mlast) * (uint32_t)K * 2u + 16u * lp;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {  // code load J = weight rows 16J .. 16J+15
      const int r = 16 * (wave * 2 + j) + (lane >> 2);
      coff[j] = (uint32_t)(r < nlast ? r : nlast) * (uint32_t)kb + 4u * (lane & 3);
    }
    {  // scales: rows 32w .. 32w+31, groups at columns k0 and k0 + 32
      const int r = 32 * wave + (lane >> 1);
      soff = ((uint32_t)(r < nlast ? r : nlast) * (uint32_t)ng + (G == 32 ? (lane & 1) : 0)) * 4u;
    }
  };
  auto dma = [&](int slot) {
    const int64_t k0 = (int64_t)ast * kFwdBK;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      dma_x16(xt + 2 * k0, xoff[i], lds0 + slot * kFwdXStage + 1024 * (wave * 4 + i));
#pragma unroll
    for (int j = 0; j < 2; ++j)
      dma_x4(ct + k0 / 4, coff[j], lds0 + kFwdCBase + slot * kFwdCStage + 256 * (wave * 2 + j));
    dma_x4(stl + 4 * (k0 / G), soff, lds0 + kFwdSBase + slot * kFwdSStage + 256 * wave);
    if (++ast == nst) {
      ast = 0;
      set_tile(++ait);
    }
  };
  set_tile(0);

  // prologue: stages 0, 1, 2 in flight
#pragma unroll
  for (int p = 0; p < 3; ++p) dma(p);
  fwd_stage_barrier();

  const int xsw = fwd_swz(l32);  // == fwd_swz(m) for every X row m this lane reads
  int s = 0;                     // stage counter, ring slot s % 4

  for (int it = 0;; ++it) {
    const uint32_t tile = (uint32_t)it * nblk + bid;
    if (tile >= ntiles) break;
    const int64_t m0 = (int64_t)(tile / tiles_n) * kFwdBM;
    const int64_t n0 = (int64_t)(tile % tiles_n) * kFwdBN;

    f32x16 acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;
    float cref[2] = {0.f, 0.f};
    uint32_t msk[2] = {0u, 0u};

    // One stage; kGroupStart tells (at compile time) whether a group starts
    // at its first column.
    auto stage = [&](auto group_start_tag, int slot) {
      constexpr bool kGroupStart = decltype(group_start_tag)::value;
      const uint8_t* xb = lds + slot * kFwdXStage;
      u32x4 cw[2];
      float sc[2][2];  // [b][q]: scales of the groups at columns k0, k0 + 32
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int nr = wn * 64 + b * 32 + l32;
        cw[b] = *reinterpret_cast<const u32x4*>(lds + kFwdCBase + slot * kFwdCStage + 16 * nr);
        if (kGroupStart) {
          const u32x2 v =
              *reinterpret_cast<const u32x2*>(lds + kFwdSBase + slot * kFwdSStage + 8 * nr);
          sc[b][0] = __uint_as_float(v.x);
          sc[b][1] = __uint_as_float(v.y);
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
        constexpr int kGS = G < 64 ? G : 64;  // columns between possible starts
        const bool start = kGroupStart && (16 * t) % kGS == 0;
        float r[2] = {1.f, 1.f};
        if (start) {
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            const float sv = sc[b][t / 2];
            const bool nz = sv != 0.f;
            msk[b] = nz ? 0xFFFFFFFFu : 0u;
            const float q = cref[b] * __builtin_amdgcn_rcpf(nz ? sv : 1.f);
            r[b] = (nz && cref[b] != 0.f) ? q : 1.f;
            cref[b] = nz ? sv : cref[b];
          }
        }
        bf16x8 bop[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) bop[b] = decode_half_rt(cw[b][t] & msk[b], h);
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

    // a group spans kPer stages (K % g == 0, so nst is a multiple of kPer);
    // only the first stage of each group rescales
    constexpr int kPer = G > kFwdBK ? G / kFwdBK : 1;
    for (int st = 0; st < nst; st += kPer) {
#pragma unroll
      for (int p = 0; p < kPer; ++p, ++s) {
        dma((s + 3) & (kFwdRing - 1));
        if (p == 0)
          stage(std::true_type{}, s & (kFwdRing - 1));
        else
          stage(std::false_type{}, s & (kFwdRing - 1));
        fwd_stage_barrier();
      }
    }

    // epilogue: lane holds column l32 of each block, rows 8*(i/4) + 4*h + i%4
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int64_t n = n0 + wn * 64 + b * 32 + l32;
      if (n >= N) continue;
      const float f = 0.5f * cref[b];
      const uint32_t voff = (uint32_t)((4 * h * N + n - n0) * 4);
#pragma unroll
      for (int a = 0; a < 4; ++a) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int64_t mu = m0 + wm * 128 + a * 32 + 8 * (i / 4) + (i % 4);  // uniform part
          if (mu + 4 * h < M)
            *reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(Y + mu * N + n0) + voff) =
                f * acc[a][b][i];
        }
      }
    }
  }
  // loads issued for stages past the end must land before the workgroup's
  // LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

hipError_t launch_tgemm_fwd(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int g, float* Y,
                            hipStream_t stream) {
  const int64_t tm = (M + kFwdBM - 1) / kFwdBM, tn = (N + kFwdBN - 1) / kFwdBN;
  const int64_t ntiles = tm * tn;
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        v > 0)
      cus = v;
    else
      cus = 256;
  }
  const int64_t blocks = ntiles < cus ? ntiles : cus;
  const dim3 grid((unsigned)blocks), block(512);
  const uint32_t t_n = (uint32_t)tn, nt = (uint32_t)ntiles;
  switch (g) {
    case 32:  hipLaunchKernelGGL(tgemm_fwd_kernel<32>, grid, block, 0, stream, X, codes, scales, M, N, K, Y, t_n, nt); break;
    case 64:  hipLaunchKernelGGL(tgemm_fwd_kernel<64>, grid, block, 0, stream, X, codes, scales, M, N, K, Y, t_n, nt); break;
    case 128: hipLaunchKernelGGL(tgemm_fwd_kernel<128>, grid, block, 0, stream, X, codes, scales, M, N, K, Y, t_n, nt); break;
    case 256: hipLaunchKernelGGL(tgemm_fwd_kernel<256>, grid, block, 0, stream, X, codes, scales, M, N, K, Y, t_n, nt); break;
    case 512: hipLaunchKernelGGL(tgemm_fwd_kernel<512>, grid, block, 0, stream, X, codes, scales, M, N, K, Y, t_n, nt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tmk
