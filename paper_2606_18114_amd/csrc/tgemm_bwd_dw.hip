// Straight-through backward w.r.t. the latent weight (paper Sec. 3.1,
// identity estimator: the gradient of What passes to W unchanged):
//   dW[N, K] = dY[M, N]^T . X[M, K],
// a plain bfloat16 contraction over the M tokens on the gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16), float32 accumulation.
//
// Both operands arrive token-major, while an MFMA operand lane needs eight
// consecutive tokens of one column.  The tiles are staged in LDS in their
// natural [token][column] order and read with the gfx950 transpose read
// ds_read_b64_tr_b16: in each group of 16 lanes, lane j passes the address of
// 4 columns (col + 4 (j % 4)) of token row j / 4, and lane i receives column
// col + i of 4 consecutive token rows.  Two such reads make one operand.
//
// Tile: 256 (N) x 256 (K) outputs per workgroup of 4 waves (2 x 2), 128 x 128
// per wave (4 x 4 MFMA blocks, accumulators in AGPRs), 32 tokens per stage.
// Stages flow through a 4-deep LDS ring filled by direct-to-LDS loads
// (global_load_lds) three stages ahead; in every token row the 32-byte units
// are XOR-permuted (dw_swz) so that transpose reads are free of bank
// conflicts.
//
// Work split (persistent, one workgroup per CU): the T output tiles are
// dealt round-robin, whole, T / P per workgroup; the T % P remaining tiles
// are each cut along the tokens into P / (T % P) parts that are added into
// dW with float32 atomics (dW is cleared first unless accumulating), so
// every CU does the same work.  Whole tiles are written with plain stores
// (read-add-write when accumulating).
//
// The direct-to-LDS loads are issued from inline assembly, so the compiler
// neither tracks nor waits for them; each wave issues exactly eight per
// stage and counts them itself (vector-memory operations retire in order).
#include <type_traits>

#include "common.hpp"
#include "launchers.hpp"

namespace tmk {

constexpr int kDwTN = 256, kDwTK = 256, kDwBM = 32, kDwRing = 4;
constexpr int kDwOp = kDwBM * 256 * 2;        // 16 KiB per operand per stage
constexpr int kDwSlot = 2 * kDwOp;            // dY tile, then X tile
constexpr int kDwLds = kDwRing * kDwSlot;     // 128 KiB
constexpr int kDwLoads = 8;                   // direct-to-LDS loads per wave per stage

typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__global__ void fill_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i + 3 < n) {
    *reinterpret_cast<f32x4*>(p + i) = f32x4{0.f, 0.f, 0.f, 0.f};
  } else {
    for (int64_t j = i; j < n; ++j) p[j] = 0.f;
  }
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// lane i: 16 bytes at base + voff -> LDS lds_base + 16 i (lds_base wave-uniform)
__device__ __forceinline__ void dw_dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int kVm>
__device__ __forceinline__ void dw_stage_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kVm) : "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int I, int N, typename F>
__device__ __forceinline__ void dw_static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    dw_static_for<I + 1, N>(f);
  }
}

// XOR applied to the 32-byte unit index of token row r: f = (r%4) ^ 2 (r%4)
// is distinct modulo 4 and in its two upper bits over any four consecutive
// rows, so the four rows of a transpose read land in distinct 32-byte bank
// groups, and so do the two column groups (units u, u + 1) read together
__device__ __forceinline__ int dw_swz(int r) { return (r & 3) ^ ((r & 3) << 1); }

// byte offset of (token row r, column c) inside an operand tile, c % 4 == 0
__device__ __forceinline__ uint32_t dw_off(int r, int c) {
  return (uint32_t)(r * 512 + 32 * ((c >> 4) ^ dw_swz(r)) + 2 * (c & 15));
}

__global__ __launch_bounds__(256) void tgemm_bwd_dw_kernel(
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X, int64_t M, int64_t N,
    int64_t K, float* __restrict__ dW, int accumulate, uint32_t tiles_k, uint32_t ntiles,
    uint32_t parts) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kDwLds];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wy = wave >> 1, wx = wave & 1;  // 128-row (N) and 128-column (K) halves
  const int l32 = lane & 31;
  const int g = lane >> 4;                  // 16-lane group of the transpose reads
  const int j16 = lane & 15;
  const uint32_t P = gridDim.x;
  const uint32_t bid = xcd_remap(blockIdx.x, P);
  const uint32_t full = ntiles / P;         // whole tiles per workgroup
  const uint32_t rem = ntiles % P;          // tiles cut into `parts` token ranges
  const int nst = (int)((M + kDwBM - 1) / kDwBM);
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;

  // this lane's transpose-read address inside an operand tile, for token
  // rows k0 .. k0+3 (k0 = 8 (g / 2) + 4 rd) and the 16 columns of its group
  const int trow = 8 * (g >> 1) + (j16 >> 2);
  const int tcol = 16 * (g & 1) + 4 * (j16 & 3);

  for (uint32_t item = 0;; ++item) {
    // ---- the item: a whole tile, or one token range of a remaining tile ----
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
    const int64_t n0 = (int64_t)(tile / tiles_k) * kDwTN;
    const int64_t k0 = (int64_t)(tile % tiles_k) * kDwTK;

    // ---- loader: wave w loads dY rows 8w .. 8w+7 and X rows 8w .. 8w+7 of a
    // stage, 2 rows (1 KiB) per load; lane -> row 2J + lane/32, 16-byte piece
    // lane%32 of the LDS row, holding logical piece lp (unit-permuted)
    uint32_t ycol[4], xcol[4];  // byte offsets of this lane's columns in a row
    const int r_lo = lane >> 5;   // row of load i: 2 (4 wave + i) + r_lo
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 2 * (wave * 4 + i) + r_lo;
      const int p = lane & 31;
      const int lp = 2 * ((p >> 1) ^ dw_swz(r)) + (p & 1);
      int64_t cn = n0 + 8 * lp;
      cn = cn < N ? cn : N - 8;  // past N: re-read the last piece (columns unused)
      int64_t ck = k0 + 8 * lp;
      ck = ck < K ? ck : K - 8;
      ycol[i] = (uint32_t)cn * 2u;
      xcol[i] = (uint32_t)ck * 2u;
    }
    auto dma = [&](int st, int slot) {
      st = st < s_end ? st : s_end - 1;  // past the range: reload its last stage
      const int64_t m0 = (int64_t)st * kDwBM;
      // rows past M re-read row M - 1 (in bounds); those tokens are zeroed in
      // the dY operand below
      const int rows = (int)(M - m0 < kDwBM ? M - m0 : kDwBM);
      const uint8_t* yb = reinterpret_cast<const uint8_t*>(dY + m0 * N);
      const uint8_t* xb = reinterpret_cast<const uint8_t*>(X + m0 * K);
      const uint32_t dst = lds0 + slot * kDwSlot;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int r = 2 * (wave * 4 + i) + r_lo;
        r = r < rows ? r : rows - 1;
        dw_dma16(yb, (uint32_t)(r * N) * 2u + ycol[i], dst + 1024 * (wave * 4 + i));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int r = 2 * (wave * 4 + i) + r_lo;
        r = r < rows ? r : rows - 1;
        dw_dma16(xb, (uint32_t)(r * K) * 2u + xcol[i], dst + kDwOp + 1024 * (wave * 4 + i));
      }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.f;

    // prologue: stages s_beg .. s_beg + 2 in flight
#pragma unroll
    for (int p = 0; p < kDwRing - 1; ++p) dma(s_beg + p, p);
    dw_stage_barrier<2 * kDwLoads>();

    // per-lane byte offsets of the transpose reads of block a (dY) / b (X)
    // inside a stage's operand tile, token rows trow .. (the reads of token
    // group t and half rd add 16 t and 4 rd rows, i.e. constant offsets)
    uint32_t aoff[4], boff[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) aoff[a] = dw_off(trow, wy * 128 + 32 * a + tcol);
#pragma unroll
    for (int b = 0; b < 4; ++b) boff[b] = kDwOp + dw_off(trow, wx * 128 + 32 * b + tcol);

    // One stage in ring slot SLOT (a compile-time constant, so every LDS
    // address below is a register plus an immediate offset).
    auto stage = [&](auto slot_tag, int st) {
      constexpr int SLOT = decltype(slot_tag)::value;
      const uint8_t* sb = lds + SLOT * kDwSlot;
      // tokens of this stage past M contribute nothing (their dY rows are
      // zeroed in the operand); the check is uniform and true at most once
      const int64_t mvalid = M - (int64_t)st * kDwBM;
      auto frag = [&](uint32_t off, int t) {
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(sb + off + 16 * t * 512));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)(sb + off + (16 * t + 4) * 512));
        const u32x2 l = __builtin_bit_cast(u32x2, lo), u = __builtin_bit_cast(u32x2, hi);
        return u32x4{l.x, l.y, u.x, u.y};
      };
#pragma unroll
      for (int t = 0; t < kDwBM / 16; ++t) {
        u32x4 af[4], bf[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) af[a] = frag(aoff[a], t);
#pragma unroll
        for (int b = 0; b < 4; ++b) bf[b] = frag(boff[b], t);
        if (mvalid < kDwBM) {
          // this lane's tokens: 16 t + 8 (g / 2) + e, e = 0 .. 7 (pairs per dword)
          const int base = 16 * t + 8 * (g >> 1);
#pragma unroll
          for (int a = 0; a < 4; ++a) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int m_lo = base + 2 * e;
              const uint32_t keep =
                  (m_lo < mvalid ? 0x0000FFFFu : 0u) | (m_lo + 1 < mvalid ? 0xFFFF0000u : 0u);
              af[a][e] &= keep;
            }
          }
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b)
            acc[a][b] = mfma32(as_bf16x8(af[a]), as_bf16x8(bf[b]), acc[a][b]);
      }
    };

    // groups of kDwRing stages (the stages past s_end only load and wait)
    for (int st0 = s_beg; st0 < s_end; st0 += kDwRing) {
      dw_static_for<0, kDwRing>([&](auto i_tag) {
        constexpr int i = decltype(i_tag)::value;
        const int st = st0 + i;
        dma(st + kDwRing - 1, (i + kDwRing - 1) & (kDwRing - 1));
        if (st < s_end) stage(i_tag, st);
        dw_stage_barrier<2 * kDwLoads>();
      });
    }
    // every load of this item has landed before the ring is reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();

    // ---- write: lane holds column l32 of each block, rows 8 (i/4) + 4 h + i%4
    const int h = lane >> 5;
    const int mode = !whole ? 2 : (accumulate ? 1 : 0);  // atomic add / add / store
    const int kleft = (int)(K - k0 - wx * 128 - l32);      // this lane's column is valid if > 32 b
    const uint32_t lane_off = (uint32_t)(4 * h) * (uint32_t)K + (uint32_t)l32;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int64_t rowa = n0 + wy * 128 + 32 * a;
      const int nleft = (int)(N - rowa) - 4 * h;  // rows 8 (i/4) + i%4 valid if below
      float* pa = dW + rowa * K + k0 + wx * 128;  // uniform
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (kleft <= 32 * b) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int dn = 8 * (i / 4) + (i % 4);
          if (dn < nleft) {
            float* q = pa + 32 * b + (uint32_t)dn * (uint32_t)K + lane_off;
            const float v = acc[a][b][i];
            if (mode == 2)
              atomicAdd(q, v);
            else if (mode == 1)
              *q += v;
            else
              *q = v;
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // one block's values live at a time
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// zeroes tiles t0 .. t0 + count - 1 of a float32 [rows, cols] array dealt in
// 256 x 256 tiles (tile t: row block t / tiles_c, column block t % tiles_c),
// skipping rows and columns past the array: one workgroup of 64 threads per
// tile row (cols % 4 == 0, 16-byte aligned base)
__global__ void zero_tiles_f32(float* __restrict__ out, int64_t rows, int64_t cols,
                               uint32_t tiles_c, uint32_t t0) {
  const uint32_t t = t0 + blockIdx.x / 256u;
  const int64_t r = (int64_t)(t / tiles_c) * 256 + blockIdx.x % 256u;
  const int64_t c = (int64_t)(t % tiles_c) * 256 + 4 * threadIdx.x;
  if (r < rows && c < cols) *reinterpret_cast<f32x4*>(out + r * cols + c) = f32x4{0.f, 0.f, 0.f, 0.f};
}

hipError_t launch_zero_tiles_f32(float* out, int64_t rows, int64_t cols, int64_t tiles_c,
                                 int64_t t0, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_tiles_f32, dim3((unsigned)(count * 256)), dim3(64), 0, stream, out,
                     rows, cols, (uint32_t)tiles_c, (uint32_t)t0);
  return hipGetLastError();
}

hipError_t launch_fill_zero_f32(float* dst, int64_t n, hipStream_t stream) {
  const int64_t threads = (n + 3) / 4;
  hipLaunchKernelGGL(fill_zero_f32, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                     dst, n);
  return hipGetLastError();
}

hipError_t launch_tgemm_bwd_dw(const uint16_t* dY, const uint16_t* X, int64_t M, int64_t N,
                               int64_t K, float* dW, int accumulate, hipStream_t stream) {
  const int64_t tn = (N + kDwTN - 1) / kDwTN, tk = (K + kDwTK - 1) / kDwTK;
  const int64_t ntiles = tn * tk;
  const int cus = current_cu_count();
  const int64_t P = ntiles < cus ? ntiles : cus;
  const int64_t rem = ntiles % P;
  int64_t parts = rem ? P / rem : 1;
  const int64_t nst = (M + kDwBM - 1) / kDwBM;
  if (parts > nst) parts = nst;
  if (rem && !accumulate) {  // the cut tiles (the last rem) are summed with atomics
    const hipError_t e = launch_zero_tiles_f32(dW, N, K, tk, ntiles - rem, rem, stream);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(tgemm_bwd_dw_kernel, dim3((unsigned)P), dim3(256), 0, stream, dY, X, M, N,
                     K, dW, accumulate, (uint32_t)tk, (uint32_t)ntiles, (uint32_t)parts);
  return hipGetLastError();
}

}  // namespace tmk
