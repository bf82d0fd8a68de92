// One decode token per batch row (batch 1 .. 4) through a whole stack of
// ternary Mamba-2 blocks in a single launch (paper Sec. 8: small-batch
// decoding is bound by the weight traffic; Sec. 3.2: the mixer stays in
// FP16).  Per block l, in layer order, for every batch row:
//
// (a block kept in FP16 takes its projections from float16 weights instead)
//   A  zx = in_proj(bf16(rmsnorm(residual) * pre_w[l]))      Z rows, K = d_model
//   B  gated = mixer step per head (conv, FP16 SSM, y * SiLU(z))
//   C  residual += out_proj(bf16(rmsnorm(gated) * norm_w[l]))  d_model rows, K = d_inner
//
// and after the last block x_out = bf16(rmsnorm(residual) * final_w).  The
// first block's residual is the token's embedding.
//
// The grid is one workgroup per CU, and the phases are separated by grid
// barriers: the waves' stores complete, one atomic increment of a counter, a
// spin on the counter (bounded: after 2^16 polls a flag is set and the spin
// ends, and every later wait that sees the flag ends too, so every wave
// always exits soon).  The barriers need every workgroup resident at once.
// A CU holds one of these workgroups (the registers of one wave per SIMD),
// so on a GPU with nothing else running all of them start at once.  The launch
// is an ordinary one: the runtime's cooperative launch gives the same
// placement but spaced the tokens 10 to 120 us apart (it waited for the
// previous kernel to drain before dispatching), against about 3 us here.  If
// other work holds CUs, workgroups start late and the spin covers the wait;
// one that outlasts the spin limit shows in the flag.
// The data that crosses workgroups (zx, the gated values and their sums,
// the residual) is written and read with agent-scope coherent accesses.  Three barriers per block
// replace the three kernel launches per block of the layer-by-layer decode
// (the first is waited for by the heads' workgroups only, the second has
// only those as arrivals).
//
// Ternary rows (phases A and C): one wave per output row at a time; lane l
// takes the 16-column code words l, l + 64, ... of the row.  Each word's
// 16 codes become eight bfloat16 pairs 2q by one shift and one AND per pair,
// which v_dot2_f32_bf16 multiplies by the matching bfloat16 pairs of x
// (exact products, float32 sums); the word's sum is scaled by the group's
// float16 scale, the lanes' sums meet in a butterfly, and 0.5 * sum is the
// output.  The normalized x of the phase is built once per workgroup in LDS
// (every workgroup computes the same sum of squares in the same order) and
// each lane keeps the pairs of its words in registers.  A wave loads the
// code words and scales of its next rows (up to kDsPrefetch words per lane)
// while it waits at the grid barrier that precedes their phase, so their
// memory latency overlaps the wait.
//
// Mixer (phase B): one workgroup per head and batch row (mixer_dev.hpp), the
// head's float16 state loaded during the barrier that precedes the phase; the
// per-head sums of g^2 feed phase C's normalization; the ring position of
// block l (one for all batch rows) moves on in phase C (after every head has
// read it).
//
// Batches of 2 .. 4 rows: every workgroup normalizes each row's residual and
// gate, and a wave decodes each code word once for all rows (the batched
// helpers below).
#include <type_traits>

#include "launchers.hpp"
#include "mixer_dev.hpp"

namespace tmk {

typedef __attribute__((ext_vector_type(2))) __bf16 ds_bf16x2;

constexpr int kDsThreads = 256;
constexpr int kDsWaves = kDsThreads / 64;
constexpr int kDsPrefetch = 24;   // code words per lane held for the next rows
constexpr uint32_t kDsSpinLimit = 1u << 16;   // a barrier takes microseconds
constexpr int kDsCounters = 64;               // barrier counter words (eight per XCD)
constexpr int kDsCounterStride = 32;          // 128 bytes between them
// the three barriers of a block have counter sets of their own; the
// timeout flag follows them
constexpr int kDsSetWords = kDsCounters * kDsCounterStride;

struct DsArgs {
  DecodeStackDesc s;
  const float* emb;
  uint16_t* x_out;
  uint32_t* sync;   // counter sets [256 b + 32 k] (barrier b < 3, word k < 8) and the
                    // timeout flag [6144], all zero at launch
  float* zx;        // [nb, Z]
  float* gated;     // [nb, d_inner]
  float* partial;   // [nb, nheads]
  float* residual;  // [nb, d_model]
  int nb;           // batch rows (1 .. 4)
};

// Every value one workgroup hands to another between barriers is written
// and read with agent-scope coherent accesses (ld_f32 / st_f32 <true>), so a
// barrier only needs each wave's stores to have completed before its
// workgroup arrives; no L2 write-back or invalidation (which cost tens of
// microseconds per barrier when every workgroup issued them).
// The barrier in two halves: ds_arrive (this workgroup's stores have
// completed: one increment of the counter) and ds_wait (spin until every
// workgroup has arrived).  Loads of the next phase's operands go between the
// two, so their memory latency overlaps the wait.
// The arrival counter is spread over kDsCounters words 128 bytes apart
// (workgroup b increments word b % kDsCounters: four workgroups of one XCD
// per word), so the increments of the 256 workgroups do not all queue on one
// address; the first wave of a waiter loads all the words at once, one per
// lane, and adds them across the lanes.
__device__ __forceinline__ void ds_arrive(uint32_t* ctr) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's stores have completed
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(ctr + kDsCounterStride * (blockIdx.x % kDsCounters), 1u);
}
__device__ __forceinline__ void ds_wait(uint32_t* ctr, uint32_t* flag, uint32_t target) {
  static_assert(kDsCounters <= 64, "one counter word per lane");
  if (threadIdx.x < 64) {  // the first wave, every lane active
    const int lane = threadIdx.x;
    uint32_t n = 0;
    for (;;) {
      uint32_t c = lane < kDsCounters
                       ? __hip_atomic_load(ctr + kDsCounterStride * lane, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT)
                       : 0u;
      c += lane_xchg<1>(c);
      c += lane_xchg<2>(c);
      c += lane_xchg<4>(c);
      c += lane_xchg<8>(c);
      c += lane_xchg<16>(c);
      c += lane_xchg<32>(c);
      if (c >= target) break;  // the total, the same in every lane
      __builtin_amdgcn_s_sleep(1);
      ++n;
      if (n == kDsSpinLimit) {  // a workgroup never arrived: give up, report
        if (lane == 0) atomicOr(flag, 1u);
        break;
      }
      // once any workgroup has given up, every later wait ends at once
      if ((n & 255) == 0 &&
          __hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)
        break;
    }
  }
  __syncthreads();
}

__device__ __forceinline__ float ds_wave_sum(float v) {
  v += __uint_as_float(lane_xchg<1>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<2>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<4>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<8>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<16>(__float_as_uint(v)));
  v += __uint_as_float(lane_xchg<32>(__float_as_uint(v)));
  return v;
}

// The four sums a[0 .. 3] of a wave in one butterfly: the lanes swap halves
// of their values across 32 and 16 lanes, then reduce the rest, so that
// lanes 16 b .. 16 b + 15 end with the total of a[b] over the 64 lanes.
__device__ __forceinline__ float ds_wave_sum4(const float (&a)[4]) {
  const int lane = threadIdx.x & 63;
  const bool hi = (lane & 32) != 0;
  float k0 = hi ? a[2] : a[0], k1 = hi ? a[3] : a[1];
  k0 += __uint_as_float(lane_xchg<32>(__float_as_uint(hi ? a[0] : a[2])));
  k1 += __uint_as_float(lane_xchg<32>(__float_as_uint(hi ? a[1] : a[3])));
  const bool mid = (lane & 16) != 0;
  float k = mid ? k1 : k0;
  k += __uint_as_float(lane_xchg<16>(__float_as_uint(mid ? k0 : k1)));
  k += __uint_as_float(lane_xchg<1>(__float_as_uint(k)));
  k += __uint_as_float(lane_xchg<2>(__float_as_uint(k)));
  k += __uint_as_float(lane_xchg<4>(__float_as_uint(k)));
  k += __uint_as_float(lane_xchg<8>(__float_as_uint(k)));
  return k;
}

// two floats as a bfloat16 pair lo | hi << 16, rounded to nearest even
// (one v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t ds_pack_bf16(float lo, float hi) {
  const ds_bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// 16 bytes at byte offset off of a buffer, read coherently at agent scope
// (the sc1 policy: past the per-XCD L2's stale lines)
__device__ __forceinline__ u32x4 ds_ld16_coherent(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16);
}

// x pairs in LDS: xs[i] = bf16(src[2i] r w[2i]) | bf16(src[2i+1] r w[2i+1]) << 16,
// r = 1 / sqrt(sumsq / K + eps), for K <= 1024 NQ.  sumsq: the sum of src^2
// in a fixed order (the same in every workgroup), or, with part != NULL, the
// sum of part[0 .. nparts) (lane j adds j, j + 64; nparts <= 128).  Every
// thread issues all its loads (4 values i = tid + 256 j at 4 i, coherent
// 16-byte loads) at once, so the phase pays one memory latency.
template <int NQ>
__device__ __forceinline__ void ds_norm_x(const float* __restrict__ src,
                                          const float* __restrict__ w, int K, float eps,
                                          const float* part, int nparts, uint32_t* xs,
                                          float* red) {
  const int tid = threadIdx.x, lane = tid & 63;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(src), (short)0, K * 4, 0x00020000);
  // the weights in flight with the values, up to four per thread (more
  // would spill registers; longer rows load them after the sum)
  constexpr bool kEarlyW = NQ <= 4;
  float v[NQ][4];
  u32x4 wv[NQ];
  float pv0 = 0.f, pv1 = 0.f;
  if (part != nullptr) {
    if (lane < nparts) pv0 = ld_f32<true>(part + lane);
    if (lane + 64 < nparts) pv1 = ld_f32<true>(part + lane + 64);
  }
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int i = tid + kDsThreads * j;
    u32x4 b = {0u, 0u, 0u, 0u};
    wv[j] = b;
    if (4 * i < K) {
      b = ds_ld16_coherent(rs, 16u * (uint32_t)i);
      if (kEarlyW) wv[j] = ld16(w + 4 * i);
    }
    v[j][0] = __uint_as_float(b.x);
    v[j][1] = __uint_as_float(b.y);
    v[j][2] = __uint_as_float(b.z);
    v[j][3] = __uint_as_float(b.w);
  }
  float sumsq;
  if (part != nullptr) {
    sumsq = ds_wave_sum(pv0 + pv1);
  } else {
    float sq = 0.f;
#pragma unroll
    for (int j = 0; j < NQ; ++j)
#pragma unroll
      for (int c = 0; c < 4; ++c) sq = __builtin_fmaf(v[j][c], v[j][c], sq);
    sq = ds_wave_sum(sq);
    if (lane == 0) red[tid >> 6] = sq;
    __syncthreads();
    sumsq = (red[0] + red[1]) + (red[2] + red[3]);
  }
  const float r = 1.f / sqrtf(sumsq / (float)K + eps);
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int i = tid + kDsThreads * j;
    if (4 * i < K) {
      if (!kEarlyW) wv[j] = ld16(w + 4 * i);
      xs[2 * i] = ds_pack_bf16(v[j][0] * r * __uint_as_float(wv[j].x),
                               v[j][1] * r * __uint_as_float(wv[j].y));
      xs[2 * i + 1] = ds_pack_bf16(v[j][2] * r * __uint_as_float(wv[j].z),
                                   v[j][3] * r * __uint_as_float(wv[j].w));
    }
  }
  __syncthreads();
}

// The code words and scales of a wave's rows r0 + wave, + kDsWaves, ... (at
// most kDsPrefetch / T of them), loaded ahead of their phase.
struct DsRows {
  uint32_t cw[kDsPrefetch];
  uint16_t sc[kDsPrefetch];
  float base[kDsPrefetch];  // the value each row's output is added to (or 0)
  int first, count;  // rows first, first + kDsWaves, ... (count of them)
};

// T = code words per lane and row (K <= 1024 T); a wave holds up to
// kDsPrefetch / T rows at a time
// base (NULL: none): the values the rows' outputs are added to, read with
// coherent loads along with the codes
// With NB > 1 batch rows, lane 16 b (b < nb) holds batch row b's base
// (base + b * ldb), the lane that writes that row's output.
template <int G, int T, int NB = 1>
__device__ __forceinline__ void ds_rows_load(DsRows& p, const uint8_t* __restrict__ codes,
                                             const uint16_t* __restrict__ s16, int K, int first,
                                             int end, const float* base, int ldb = 0,
                                             int nb = 1) {
  constexpr int kRows = kDsPrefetch / T;
  const int lane = threadIdx.x & 63;
  const int nw = K / 16;
  int count = (end - first + kDsWaves - 1) / kDsWaves;
  count = count < 0 ? 0 : (count > kRows ? kRows : count);
  p.first = first;
  p.count = count;
#pragma unroll
  for (int i = 0; i < kRows * T; ++i) {
    const int j = i / T, t = i % T, w = lane + 64 * t;
    p.cw[i] = 0u;
    p.sc[i] = 0;
    if (j < count && w < nw) {
      const int64_t r = first + (int64_t)j * kDsWaves;
      p.cw[i] = reinterpret_cast<const uint32_t*>(codes + r * (K / 4))[w];
      p.sc[i] = s16[r * (K / G) + (16 * w) / G];
    }
  }
  if constexpr (NB == 1) {
#pragma unroll
    for (int j = 0; j < kRows; ++j)
      p.base[j] = base != nullptr && j < count ? ld_f32<true>(base + first + j * kDsWaves) : 0.f;
  } else {
    const int bl = lane >> 4;
    const bool mine = base != nullptr && (lane & 15) == 0 && bl < nb;
#pragma unroll
    for (int j = 0; j < kRows; ++j)
      p.base[j] = mine && j < count
                      ? ld_f32<true>(base + (int64_t)bl * ldb + first + j * kDsWaves)
                      : 0.f;
  }
}

// out(r, base + y) for the rows held in p: y = sum_k x[k] q[r, k] s16[r, k / G].
// With at most two words per lane the rows go in groups of up to nine, all
// their dependency chains interleaved; with more, in pairs.  Each chain is
// split into even and odd pairs.
template <int G, int T>
__device__ __forceinline__ float ds_row_sum(const DsRows& p, const uint32_t (&xr)[T][8],
                                            int j) {
  float aj = 0.f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const uint32_t cw = p.cw[j * T + t];
    float e = 0.f, o = 0.f;
#pragma unroll
    for (int q = 0; q < 8; q += 2) {
      const uint32_t p0 = (cw << (14 - 2 * q)) & kPairMask;
      const uint32_t p1 = (cw << (12 - 2 * q)) & kPairMask;
      e = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(ds_bf16x2, p0),
                                          __builtin_bit_cast(ds_bf16x2, xr[t][q]), e, false);
      o = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(ds_bf16x2, p1),
                                          __builtin_bit_cast(ds_bf16x2, xr[t][q + 1]), o, false);
    }
    aj = __builtin_fmaf(e + o, h2f(p.sc[j * T + t]), aj);
  }
  return aj;
}

template <int G, int T, typename Out>
__device__ __forceinline__ void ds_rows_compute(const DsRows& p, const uint32_t (&xr)[T][8],
                                                Out out) {
  constexpr int kRows = kDsPrefetch / T;
  // groups of up to nine rows (a wave's share of in_proj at d_model 2048),
  // so the slots past the rows held are not computed
  constexpr int kStep = T <= 2 ? (kRows < 9 ? kRows : 9) : 2;
  const int lane = threadIdx.x & 63, rl = lane >> 4;
#pragma unroll
  for (int j0 = 0; j0 < kRows; j0 += kStep) {
    if (j0 < p.count) {
      float acc[kStep];
#pragma unroll
      for (int jj = 0; jj < kStep; ++jj)
        acc[jj] = ds_row_sum<G, T>(p, xr, j0 + jj < kRows ? j0 + jj : j0);
      // the rows' sums meet four at a time; lane 16 i writes row jq + i
#pragma unroll
      for (int jq = 0; jq < kStep; jq += 4) {
        float a4[4], b4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          a4[i] = jq + i < kStep ? acc[jq + i] : 0.f;
          b4[i] = jq + i < kStep && j0 + jq + i < kRows ? p.base[j0 + jq + i] : 0.f;
        }
        const float v = ds_wave_sum4(a4);
        const float bv = rl == 0 ? b4[0] : (rl == 1 ? b4[1] : (rl == 2 ? b4[2] : b4[3]));
        const int j = j0 + jq + rl;
        if ((lane & 15) == 0 && jq + rl < kStep && j < p.count)
          out(p.first + j * kDsWaves, bv + 0.5f * v);
      }
    }
  }
}

// Rows r0 + wave, + kDsWaves, ... (< r1) of a float16 matrix W [rows, K] (a
// block kept in FP16): out(r, base[r] + sum_k x[k] W[r, k]), base NULL: 0.
// A wave takes up to four rows at a time (8 / T, so 64 registers hold their
// pieces), their 16-byte pieces (the columns of the lane's x pairs) loaded
// together; each float16 weight times the float32 value of its bfloat16 x is
// exact, summed in float32 in a fixed order.
template <int T, typename Out>
__device__ __forceinline__ void ds_dense_rows(const uint16_t* __restrict__ W, int K, int r0,
                                              int r1, const uint32_t (&xr)[T][8],
                                              const float* base, Out out) {
  constexpr int kR = T >= 8 ? 1 : (T >= 4 ? 2 : 4);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = K / 16;
  for (int r = r0 + wave; r < r1; r += kR * kDsWaves) {
    u32x4 wv[kR][T][2];
    float bv[kR];
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const int ri = r + i * kDsWaves;
      const int rr = ri < r1 ? ri : r;  // past the range: row r again (not used)
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int w = lane + 64 * t;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          wv[i][t][h] = u32x4{0u, 0u, 0u, 0u};
          if (w < nw) wv[i][t][h] = ld16(W + (int64_t)rr * K + 16 * w + 8 * h);
        }
      }
      bv[i] = base != nullptr && ri < r1 ? ld_f32<true>(base + ri) : 0.f;
    }
    float acc[kR];
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      float e = 0.f, o = 0.f;
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t wq[4] = {wv[i][t][h].x, wv[i][t][h].y, wv[i][t][h].z, wv[i][t][h].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t xp = xr[t][4 * h + q];
            e = __builtin_fmaf(h2f((uint16_t)(wq[q] & 0xFFFFu)), __uint_as_float(xp << 16), e);
            o = __builtin_fmaf(h2f((uint16_t)(wq[q] >> 16)), __uint_as_float(xp & 0xFFFF0000u), o);
          }
        }
      acc[i] = ds_wave_sum(e + o);
    }
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < kR; ++i)
        if (r + i * kDsWaves < r1) out(r + i * kDsWaves, bv[i] + acc[i]);
    }
  }
}

// index of block l among the blocks kept in FP16, or -1 (ternary)
__device__ __forceinline__ int ds_kept(const DecodeStackDesc& s, int l) {
  for (int i = 0; i < s.n_kept; ++i)
    if (s.kept[i] == l) return i;
  return -1;
}

// this lane's x pairs (words lane, lane + 64, ...; zero past the row)
template <int T>
__device__ __forceinline__ void ds_x_regs(const uint32_t* xs, int K, uint32_t (&xr)[T][8]) {
  const int lane = threadIdx.x & 63;
  const int nw = K / 16;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int w = lane + 64 * t;
    u32x4 a = {0u, 0u, 0u, 0u}, b = {0u, 0u, 0u, 0u};
    if (w < nw) {
      a = *reinterpret_cast<const u32x4*>(xs + 8 * w);
      b = *reinterpret_cast<const u32x4*>(xs + 8 * w + 4);
    }
    xr[t][0] = a.x; xr[t][1] = a.y; xr[t][2] = a.z; xr[t][3] = a.w;
    xr[t][4] = b.x; xr[t][5] = b.y; xr[t][6] = b.z; xr[t][7] = b.w;
  }
}

// all rows [.., r1) of the wave: the prefetched first ones, then the rest
template <int G, int T, typename Out>
__device__ __forceinline__ void ds_rows_all(DsRows& p, const uint8_t* codes, const uint16_t* s16,
                                            int K, int r1, const uint32_t (&xr)[T][8],
                                            const float* base, Out out) {
  for (;;) {
    ds_rows_compute<G, T>(p, xr, out);
    const int next = p.first + p.count * kDsWaves;
    if (p.count == 0 || next >= r1) break;
    ds_rows_load<G, T>(p, codes, s16, K, next, r1, base);
  }
}

// ---- batches of nb = 2 .. 4 tokens (NB = 4 slots)
//
// The x pairs of batch row b sit in LDS at xs + b * xstride.  A wave takes
// one ternary row at a time as above, but decodes each code word once for
// all batch rows: the eight pairs 2q of a word go through v_dot2_f32_bf16
// against each row's x pairs (read from LDS per word column, once per group
// of rows), and each (row, batch row) keeps its own float32 sum, in the same
// order as the batch-1 form.  Slots b >= nb see zero x.

// this lane's x pairs of word column w for every batch row (zero past the
// row and for b >= nb)
template <int NB>
__device__ __forceinline__ void ds_x_col(const uint32_t* xs, int xstride, int w, int nw, int nb,
                                         uint32_t (&xv)[NB][8]) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    u32x4 lo = {0u, 0u, 0u, 0u}, hi = {0u, 0u, 0u, 0u};
    if (w < nw && b < nb) {
      lo = *reinterpret_cast<const u32x4*>(xs + b * xstride + 8 * w);
      hi = *reinterpret_cast<const u32x4*>(xs + b * xstride + 8 * w + 4);
    }
    xv[b][0] = lo.x; xv[b][1] = lo.y; xv[b][2] = lo.z; xv[b][3] = lo.w;
    xv[b][4] = hi.x; xv[b][5] = hi.y; xv[b][6] = hi.z; xv[b][7] = hi.w;
  }
}

// Rows of every batch row: x = bf16(src[b] r_b w) for b < nb, r_b from the
// sum of squares of src row b (rows K apart), or of part[b * nparts ..
// + nparts); the same order per row as ds_norm_x.  Rows go in chunks of
// kC (all at once up to 16 values per thread, their loads issued together).
template <int NQ, int NB>
__device__ __forceinline__ void ds_norm_xb(const float* __restrict__ src,
                                           const float* __restrict__ w, int K, float eps,
                                           const float* part, int nparts, int nb, uint32_t* xs,
                                           int xstride, float* red) {
  constexpr int kC = NQ * NB <= 16 ? NB : (16 / NQ > 0 ? 16 / NQ : 1);
  const int tid = threadIdx.x, lane = tid & 63;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(src), (short)0, nb * K * 4, 0x00020000);
  u32x4 wv[NQ];  // the weights, in flight with the first chunk's values
#pragma unroll
  for (int j = 0; j < NQ; ++j) {
    const int i = tid + kDsThreads * j;
    wv[j] = u32x4{0u, 0u, 0u, 0u};
    if (4 * i < K) wv[j] = ld16(w + 4 * i);
  }
#pragma unroll
  for (int b0 = 0; b0 < NB; b0 += kC) {
    if (b0 >= nb) break;
    float v[kC][NQ][4];
    float pv[kC][2];
#pragma unroll
    for (int c = 0; c < kC; ++c) {
      const int b = b0 + c;
      pv[c][0] = pv[c][1] = 0.f;
      if (part != nullptr && b < nb) {
        if (lane < nparts) pv[c][0] = ld_f32<true>(part + b * nparts + lane);
        if (lane + 64 < nparts) pv[c][1] = ld_f32<true>(part + b * nparts + lane + 64);
      }
#pragma unroll
      for (int j = 0; j < NQ; ++j) {
        const int i = tid + kDsThreads * j;
        u32x4 q = {0u, 0u, 0u, 0u};
        if (b < nb && 4 * i < K)
          q = ds_ld16_coherent(rs, 4u * (uint32_t)(b * K) + 16u * (uint32_t)i);
        v[c][j][0] = __uint_as_float(q.x);
        v[c][j][1] = __uint_as_float(q.y);
        v[c][j][2] = __uint_as_float(q.z);
        v[c][j][3] = __uint_as_float(q.w);
      }
    }
    float sumsq[kC];
    if (part != nullptr) {
#pragma unroll
      for (int c = 0; c < kC; ++c) sumsq[c] = ds_wave_sum(pv[c][0] + pv[c][1]);
    } else {
#pragma unroll
      for (int c = 0; c < kC; ++c) {
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < NQ; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) sq = __builtin_fmaf(v[c][j][e], v[c][j][e], sq);
        sq = ds_wave_sum(sq);
        if (lane == 0) red[(b0 + c) * kDsWaves + (tid >> 6)] = sq;
      }
      __syncthreads();
#pragma unroll
      for (int c = 0; c < kC; ++c) {
        const float* rb = red + (b0 + c) * kDsWaves;
        sumsq[c] = (rb[0] + rb[1]) + (rb[2] + rb[3]);
      }
    }
#pragma unroll
    for (int c = 0; c < kC; ++c) {
      const int b = b0 + c;
      if (b >= nb) break;
      const float r = 1.f / sqrtf(sumsq[c] / (float)K + eps);
      uint32_t* xb = xs + b * xstride;
#pragma unroll
      for (int j = 0; j < NQ; ++j) {
        const int i = tid + kDsThreads * j;
        if (4 * i < K) {
          xb[2 * i] = ds_pack_bf16(v[c][j][0] * r * __uint_as_float(wv[j].x),
                                   v[c][j][1] * r * __uint_as_float(wv[j].y));
          xb[2 * i + 1] = ds_pack_bf16(v[c][j][2] * r * __uint_as_float(wv[j].z),
                                       v[c][j][3] * r * __uint_as_float(wv[j].w));
        }
      }
    }
  }
  __syncthreads();
}

// out(r, b, base + 0.5 sum) for the rows held in p and every batch row b <
// nb, called by lane 16 b
template <int G, int T, int NB, typename Out>
__device__ __forceinline__ void ds_rows_compute_b(const DsRows& p, const uint32_t* xs,
                                                  int xstride, int K, int nb, Out out) {
  static_assert(NB == 4, "batch slots of the four-way butterfly");
  constexpr int kRows = kDsPrefetch / T;
  constexpr int kStep = kRows < 9 ? kRows : 9;
  const int lane = threadIdx.x & 63;
  const int nw = K / 16, bl = lane >> 4;
  const bool writer = (lane & 15) == 0 && bl < nb;
#pragma unroll
  for (int j0 = 0; j0 < kRows; j0 += kStep) {
    if (j0 < p.count) {
      float acc[kStep][NB];
#pragma unroll
      for (int jj = 0; jj < kStep; ++jj)
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[jj][b] = 0.f;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        // one word column's x at a time (hoisting them all would take
        // 32 T registers)
        if (T > 2) __builtin_amdgcn_sched_barrier(0);
        uint32_t xv[NB][8];
        ds_x_col<NB>(xs, xstride, lane + 64 * t, nw, nb, xv);
#pragma unroll
        for (int jj = 0; jj < kStep; ++jj) {
          const int j = j0 + jj;
          if (j >= kRows) break;
          const uint32_t cw = p.cw[j * T + t];
          const float sc = h2f(p.sc[j * T + t]);
          uint32_t pr[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) pr[q] = (cw << (14 - 2 * q)) & kPairMask;
#pragma unroll
          for (int b = 0; b < NB; ++b) {
            float e = 0.f, o = 0.f;
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
              e = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(ds_bf16x2, pr[q]),
                                                  __builtin_bit_cast(ds_bf16x2, xv[b][q]), e,
                                                  false);
              o = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(ds_bf16x2, pr[q + 1]),
                                                  __builtin_bit_cast(ds_bf16x2, xv[b][q + 1]),
                                                  o, false);
            }
            acc[jj][b] = __builtin_fmaf(e + o, sc, acc[jj][b]);
          }
        }
      }
#pragma unroll
      for (int jj = 0; jj < kStep; ++jj) {
        const int j = j0 + jj;
        if (j >= kRows || j >= p.count) break;
        const float v = ds_wave_sum4(acc[jj]);
        if (writer) out(p.first + j * kDsWaves, bl, p.base[j] + 0.5f * v);
      }
    }
  }
}

template <int G, int T, int NB, typename Out>
__device__ __forceinline__ void ds_rows_all_b(DsRows& p, const uint8_t* codes,
                                              const uint16_t* s16, int K, int r1,
                                              const uint32_t* xs, int xstride, int nb,
                                              const float* base, int ldb, Out out) {
  for (;;) {
    ds_rows_compute_b<G, T, NB>(p, xs, xstride, K, nb, out);
    const int next = p.first + p.count * kDsWaves;
    if (p.count == 0 || next >= r1) break;
    ds_rows_load<G, T, NB>(p, codes, s16, K, next, r1, base, ldb, nb);
  }
}

// ds_dense_rows for every batch row b < nb: out(r, b, base[b * ldb + r] +
// sum_k x_b[k] W[r, k]), called by lane 16 b; each float16 weight is
// converted once for all batch rows
template <int T, int NB, typename Out>
__device__ __forceinline__ void ds_dense_rows_b(const uint16_t* __restrict__ W, int K, int r0,
                                                int r1, const uint32_t* xs, int xstride, int nb,
                                                const float* base, int ldb, Out out) {
  static_assert(NB == 4, "batch slots of the four-way butterfly");
  constexpr int kR = T >= 4 ? 1 : 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = K / 16, bl = lane >> 4;
  const bool writer = (lane & 15) == 0 && bl < nb;
  for (int r = r0 + wave; r < r1; r += kR * kDsWaves) {
    u32x4 wv[kR][T][2];
    float bv[kR];
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const int ri = r + i * kDsWaves;
      const int rr = ri < r1 ? ri : r;  // past the range: row r again (not used)
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const int w = lane + 64 * t;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          wv[i][t][h] = u32x4{0u, 0u, 0u, 0u};
          if (w < nw) wv[i][t][h] = ld16(W + (int64_t)rr * K + 16 * w + 8 * h);
        }
      }
      bv[i] = base != nullptr && writer && ri < r1 ? ld_f32<true>(base + (int64_t)bl * ldb + ri)
                                                   : 0.f;
    }
    float e[kR][NB], o[kR][NB];
#pragma unroll
    for (int i = 0; i < kR; ++i)
#pragma unroll
      for (int b = 0; b < NB; ++b) e[i][b] = o[i][b] = 0.f;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      if (T > 2) __builtin_amdgcn_sched_barrier(0);
      uint32_t xv[NB][8];
      ds_x_col<NB>(xs, xstride, lane + 64 * t, nw, nb, xv);
#pragma unroll
      for (int i = 0; i < kR; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t wq[4] = {wv[i][t][h].x, wv[i][t][h].y, wv[i][t][h].z, wv[i][t][h].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float w0 = h2f((uint16_t)(wq[q] & 0xFFFFu)), w1 = h2f((uint16_t)(wq[q] >> 16));
#pragma unroll
            for (int b = 0; b < NB; ++b) {
              const uint32_t xp = xv[b][4 * h + q];
              e[i][b] = __builtin_fmaf(w0, __uint_as_float(xp << 16), e[i][b]);
              o[i][b] = __builtin_fmaf(w1, __uint_as_float(xp & 0xFFFF0000u), o[i][b]);
            }
          }
        }
    }
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const float a4[4] = {e[i][0] + o[i][0], e[i][1] + o[i][1], e[i][2] + o[i][2],
                           e[i][3] + o[i][3]};
      const float v = ds_wave_sum4(a4);
      if (writer && r + i * kDsWaves < r1) out(r + i * kDsWaves, bl, bv[i] + v);
    }
  }
}

// TA, TC: code words per lane of an in_proj row (d_model <= 1024 TA) and of
// an out_proj row (d_inner <= 1024 TC); NB: 1, or 4 batch slots (nb = 2 .. 4
// rows, the mixer's workgroups then one per (head, batch row))
template <int G, int TA, int TC, int NB>
__global__ __launch_bounds__(kDsThreads) void decode_stack_kernel(DsArgs a) {
  const DecodeStackDesc& s = a.s;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int P = (int)gridDim.x, bid = (int)blockIdx.x;
  const int D = s.d_model, H = s.nheads, DI = H * kMxP;
  const int Z = 2 * DI + 2 * kMxN + H;
  const int conv_dim = DI + 2 * kMxN;
  const int nb = NB == 1 ? 1 : a.nb;
  const int heads = H * nb;  // the mixer's workgroups
  constexpr int kXs = (TA > TC ? TA : TC) * 64 * 8;  // x pair words of one batch row
  __shared__ __attribute__((aligned(16))) uint32_t xs[NB * kXs];
  __shared__ float red[NB * kDsWaves];

  const int za = (Z + P - 1) / P, zr0 = bid * za < Z ? bid * za : Z;
  const int zr1 = zr0 + za < Z ? zr0 + za : Z;
  const int ca = (D + P - 1) / P, cr0 = bid * ca < D ? bid * ca : D;
  const int cr1 = cr0 + ca < D ? cr0 + ca : D;
  uint32_t* bar_a = a.sync;                    // in_proj rows done (all workgroups)
  uint32_t* bar_b = a.sync + kDsSetWords;      // mixer done (the heads' workgroups)
  uint32_t* bar_c = a.sync + 2 * kDsSetWords;  // residual done (all workgroups)
  uint32_t* flag = a.sync + 3 * kDsSetWords;
  // this workgroup's head and batch row in the mixer phase
  const int hh = bid % H, hb = bid < heads ? bid / H : 0;
  DsRows rows;
  u32x4 sv[4];

  // block 0's in_proj rows
  int kd = ds_kept(s, 0);
  if (kd < 0) ds_rows_load<G, TA, NB>(rows, s.in_codes, s.in_s16, D, zr0 + wave, zr1, nullptr);
  for (int l = 0; l < s.n_layers; ++l) {
    const uint8_t* inc = s.in_codes + (int64_t)l * Z * (D / 4);
    const uint16_t* ins = s.in_s16 + (int64_t)l * Z * (D / G);
    const uint8_t* outc = s.out_codes + (int64_t)l * D * (DI / 4);
    const uint16_t* outs = s.out_s16 + (int64_t)l * D * (DI / G);
    const float* src = l == 0 ? a.emb : a.residual;

    // ---- A: in_proj of the normalized residual
    if constexpr (NB == 1) {
      ds_norm_x<TA>(src, s.pre_w + (int64_t)l * D, D, s.eps, nullptr, 0, xs, red);
      uint32_t xr[TA][8];
      ds_x_regs<TA>(xs, D, xr);
      auto put = [&](int r, float y) { st_f32<true>(a.zx + r, y); };
      if (kd < 0)
        ds_rows_all<G, TA>(rows, inc, ins, D, zr1, xr, nullptr, put);
      else
        ds_dense_rows<TA>(s.in_w16 + (int64_t)kd * Z * D, D, zr0, zr1, xr, nullptr, put);
    } else {
      ds_norm_xb<TA, NB>(src, s.pre_w + (int64_t)l * D, D, s.eps, nullptr, 0, nb, xs, kXs, red);
      auto put = [&](int r, int b, float y) { st_f32<true>(a.zx + (int64_t)b * Z + r, y); };
      if (kd < 0)
        ds_rows_all_b<G, TA, NB>(rows, inc, ins, D, zr1, xs, kXs, nb, nullptr, 0, put);
      else
        ds_dense_rows_b<TA, NB>(s.in_w16 + (int64_t)kd * Z * D, D, zr0, zr1, xs, kXs, nb,
                                nullptr, 0, put);
    }
    // the mixer's state, and this workgroup's out_proj rows, during the barrier
    // (only the heads' workgroups wait for every in_proj row; the others go
    // on to wait for the heads)
    ds_arrive(bar_a);
    uint16_t* ssm_h = s.ssm_state + (((int64_t)l * nb + hb) * H + hh) * kMxP * kMxN;
    if (bid < heads) mixer_state_load(ssm_h, tid, sv);
    if (kd < 0) ds_rows_load<G, TC, NB>(rows, outc, outs, DI, cr0 + wave, cr1, src, D, nb);

    // ---- B: mixer step, one workgroup per head and batch row
    if (bid < heads) {
      ds_wait(bar_a, flag, (uint32_t)(l + 1) * (uint32_t)P);
      const int pos = s.conv_pos[l] & 3;
      mixer_head_step<true>(a.zx + (int64_t)hb * Z, hh, H,
                            s.conv_state + ((int64_t)l * nb + hb) * conv_dim * 4, ssm_h, sv,
                            [&]() { return pos; }, s.conv_w + (int64_t)l * conv_dim * 4,
                            s.conv_b + (int64_t)l * conv_dim, s.dt_bias + (int64_t)l * H,
                            s.A_log + (int64_t)l * H, s.D + (int64_t)l * H,
                            a.gated + (int64_t)hb * DI, a.partial + hb * H + hh);
      ds_arrive(bar_b);
    }
    ds_wait(bar_b, flag, (uint32_t)(l + 1) * (uint32_t)heads);

    // ---- C: out_proj of the normalized gate, added into the residual
    // (the heads' sums of g^2 give the norm, in the same order everywhere)
    if constexpr (NB == 1) {
      ds_norm_x<TC>(a.gated, s.norm_w + (int64_t)l * DI, DI, s.eps, a.partial, H, xs, red);
      uint32_t xr[TC][8];
      ds_x_regs<TC>(xs, DI, xr);
      auto put = [&](int r, float y) { st_f32<true>(a.residual + r, y); };
      if (kd < 0)
        ds_rows_all<G, TC>(rows, outc, outs, DI, cr1, xr, src, put);
      else
        ds_dense_rows<TC>(s.out_w16 + (int64_t)kd * D * DI, DI, cr0, cr1, xr, src, put);
    } else {
      ds_norm_xb<TC, NB>(a.gated, s.norm_w + (int64_t)l * DI, DI, s.eps, a.partial, H, nb, xs,
                         kXs, red);
      auto put = [&](int r, int b, float y) { st_f32<true>(a.residual + (int64_t)b * D + r, y); };
      if (kd < 0)
        ds_rows_all_b<G, TC, NB>(rows, outc, outs, DI, cr1, xs, kXs, nb, src, D, put);
      else
        ds_dense_rows_b<TC, NB>(s.out_w16 + (int64_t)kd * D * DI, DI, cr0, cr1, xs, kXs, nb, src,
                                D, put);
    }
    if (bid == 0 && tid == 0) s.conv_pos[l] = (s.conv_pos[l] + 1) & 3;
    // the next block's in_proj rows during the barrier
    ds_arrive(bar_c);
    kd = l + 1 < s.n_layers ? ds_kept(s, l + 1) : -1;
    if (l + 1 < s.n_layers && kd < 0)
      ds_rows_load<G, TA, NB>(rows, inc + (int64_t)Z * (D / 4), ins + (int64_t)Z * (D / G), D,
                              zr0 + wave, zr1, nullptr);
    ds_wait(bar_c, flag, (uint32_t)(l + 1) * (uint32_t)P);
  }
  // final norm of the residual (workgroup 0)
  if (bid == 0) {
    const float* fin = s.n_layers > 0 ? a.residual : a.emb;
    if constexpr (NB == 1)
      ds_norm_x<TA>(fin, s.final_w, D, s.eps, nullptr, 0, xs, red);
    else
      ds_norm_xb<TA, NB>(fin, s.final_w, D, s.eps, nullptr, 0, nb, xs, kXs, red);
    uint32_t* xo = reinterpret_cast<uint32_t*>(a.x_out);
    for (int b = 0; b < nb; ++b)
      for (int i = tid; i < D / 2; i += kDsThreads) xo[b * (D / 2) + i] = xs[b * kXs + i];
  }
}

// the instantiation for group size g, (TA, TC) rounded up to a supported
// pair and batch (1, or 2 .. 4 with TA <= 2 and TC <= 4), or NULL
static const void* decode_stack_fn(int g, int ta, int tc, int nb) {
  auto pick = [&](auto gt, auto bt) -> const void* {
    constexpr int G = decltype(gt)::value, NB = decltype(bt)::value;
    if (ta <= 1 && tc <= 1) return reinterpret_cast<const void*>(&decode_stack_kernel<G, 1, 1, NB>);
    if (ta <= 1 && tc <= 2) return reinterpret_cast<const void*>(&decode_stack_kernel<G, 1, 2, NB>);
    if (ta <= 2 && tc <= 4) return reinterpret_cast<const void*>(&decode_stack_kernel<G, 2, 4, NB>);
    // (batches: rows up to d_model 2048 and d_inner 4096, where the
    // registers hold every value without spilling)
    if constexpr (NB == 1)
      if (ta <= 4 && tc <= 8)
        return reinterpret_cast<const void*>(&decode_stack_kernel<G, 4, 8, 1>);
    return nullptr;
  };
  auto by_batch = [&](auto gt) -> const void* {
    if (nb == 1) return pick(gt, std::integral_constant<int, 1>{});
    if (nb <= 4) return pick(gt, std::integral_constant<int, 4>{});
    return nullptr;
  };
  switch (g) {
    case 64:  return by_batch(std::integral_constant<int, 64>{});
    case 128: return by_batch(std::integral_constant<int, 128>{});
    case 256: return by_batch(std::integral_constant<int, 256>{});
    default: return nullptr;
  }
}

hipError_t launch_decode_stack(const DecodeStackDesc& s, const float* emb, uint16_t* x_out,
                               void* workspace, hipStream_t stream) {
  auto up = [](int64_t v) { return (v + 255) / 256 * 256; };
  const int64_t nb = s.batch;
  const int64_t DI = (int64_t)s.nheads * kMxP, Z = 2 * DI + 2 * kMxN + s.nheads;
  if (nb < 1 || nb > kDecodeStackMaxBatch) return hipErrorInvalidValue;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  DsArgs a;
  a.s = s;
  a.emb = emb;
  a.x_out = x_out;
  a.nb = (int)nb;
  const int64_t hd = kDecodeStackSyncBytes;
  const int64_t o_gated = hd + up(nb * Z * 4), o_part = o_gated + up(nb * DI * 4);
  a.sync = reinterpret_cast<uint32_t*>(ws);
  a.zx = reinterpret_cast<float*>(ws + hd);
  a.gated = reinterpret_cast<float*>(ws + o_gated);
  a.partial = reinterpret_cast<float*>(ws + o_part);
  a.residual = reinterpret_cast<float*>(ws + o_part + up(nb * s.nheads * 4));
  static_assert(4 * (3 * kDsSetWords + 1) <= kDecodeStackSyncBytes,
                "barrier words fit the workspace header");
  // the barrier counter and the timeout flag start at zero (a fill kernel,
  // so the call stays capturable)
  hipError_t e = launch_fill_zero_f32(reinterpret_cast<float*>(ws), 3 * kDsSetWords + 1, stream);
  if (e != hipSuccess) return e;
  const int cus = current_cu_count();
  const int ta = (s.d_model / 16 + 63) / 64, tc = (s.nheads * kMxP / 16 + 63) / 64;
  const void* fn = decode_stack_fn(s.g, ta, tc, (int)nb);
  if (fn == nullptr) return hipErrorInvalidValue;
  int per_cu = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kDsThreads, 0)) !=
      hipSuccess)
    return e;
  // every workgroup must fit at once (one per CU), one per head and batch row
  if (per_cu < 1 || cus < s.nheads * nb) return hipErrorInvalidValue;
  void* args[] = {&a};
  return hipLaunchKernel(fn, dim3((unsigned)cus), dim3(kDsThreads), args, 0, stream);
}

}  // namespace tmk
