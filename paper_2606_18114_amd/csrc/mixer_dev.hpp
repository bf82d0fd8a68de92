// The per-head Mamba-2 mixer decode step (the part of a decoding layer the
// paper keeps in FP16, Sec. 3.2), as device functions shared by the mixer
// kernels (mixer.hip) and the whole-stack decode kernel (decode_stack.hip).
//
// One workgroup of kMxThreads threads per (head, batch row):
//   * causal depthwise convolution step (d_conv = 4) over the head's 64 x
//     channels and the 2 x d_state B/C channels shared by all heads, SiLU;
//   * dt' = softplus(dt + dt_bias), decay a = exp(-dt' exp(A_log));
//   * state[p, n] <- a state[p, n] + dt' x[p] B[n]  (float16 state, float32
//     arithmetic, rounded once to float16 when stored);
//   * y[p] = sum_n state[p, n] C[n] + D x[p];  g = y * SiLU(z).
// Thread t owns channel p = t / 4 and states n = 32 (t % 4) .. + 31.
//
// Convolution state: a ring of 4 float16 slots per channel; the window of a
// step, oldest first, is slots (pos + 1 .. pos + 3) % 4 and the new input,
// which then overwrites slot pos (the oldest).  Every head reads the B/C
// channels' window, so no workgroup may shift it in place while others still
// read: the ring writes only the slot nobody reads (head 0 writes the shared
// B/C channels), and the caller moves the position on after every head of
// the step is done.
#pragma once

#include "common.hpp"

namespace tmk {

constexpr int kMxP = 64;    // headdim
constexpr int kMxN = 128;   // d_state
constexpr int kMxThreads = 256;

__device__ __forceinline__ float mx_silu(float v) { return v / (1.f + expf(-v)); }
__device__ __forceinline__ float mx_softplus(float v) { return v > 20.f ? v : log1pf(expf(v)); }

// float32 accesses to data other workgroups of the same launch write or read
// between grid barriers (COH): agent-scope coherent loads and stores, which
// bypass the per-XCD L2's stale lines and write through it, so no L2
// write-back or invalidation is needed at the barriers; plain otherwise
template <bool COH>
__device__ __forceinline__ float ld_f32(const float* p) {
  if constexpr (COH)
    return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    return *p;
}
template <bool COH>
__device__ __forceinline__ void st_f32(float* p, float v) {
  if constexpr (COH)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

__device__ __forceinline__ float h2f(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ uint16_t f2h(float f) {  // round to nearest even
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// The 64 bytes of the head's float16 state [64][128] (ssm_h) thread tid
// owns: channel tid / 4, states 32 (tid % 4) .. + 31.
__device__ __forceinline__ void mixer_state_load(const uint16_t* ssm_h, int tid,
                                                 u32x4 (&sv)[4]) {
  const uint16_t* sp = ssm_h + (tid >> 2) * kMxN + 32 * (tid & 3);
#pragma unroll
  for (int k = 0; k < 4; ++k) sv[k] = ld16(sp + 8 * k);
}

// One head's step.  row: the head's batch row of zxbcdt (z | xBC | dt);
// conv_b: that batch row's ring [conv_dim][4]; ssm_h: the head's state,
// whose thread slice sv was loaded by mixer_state_load; pos_of(): the ring
// position, called once the ring words have been loaded; gated_b: that batch
// row's gated output [d_inner]; part: if not NULL, receives the head's sum of
// g^2 (every channel counted once).  COH: row, gated_b and part are shared
// with other workgroups of the launch (coherent accesses, see ld_f32).
template <bool COH = false, typename PosFn>
__device__ __forceinline__ void mixer_head_step(
    const float* __restrict__ row, int h, int nheads, uint16_t* __restrict__ conv_b,
    uint16_t* __restrict__ ssm_h, const u32x4 (&sv)[4], PosFn pos_of,
    const float* __restrict__ conv_w, const float* __restrict__ conv_bias,
    const float* __restrict__ dt_bias, const float* __restrict__ A_log,
    const float* __restrict__ Dp, float* __restrict__ gated_b, float* __restrict__ part) {
  const int tid = threadIdx.x;
  const int d_inner = nheads * kMxP;
  __shared__ float u[kMxP + 2 * kMxN];  // x of the head, then B, then C (after SiLU)
  __shared__ float wsum[kMxThreads / 64];
  const int p = tid >> 2, q = tid & 3;

  // convolution: local channel i < 64 is x channel 64 h + i, then the B/C
  // channels d_inner + (i - 64); a thread takes at most two channels
  constexpr int kMxCh = (kMxP + 2 * kMxN + kMxThreads - 1) / kMxThreads;
  uint32_t ring[kMxCh][2];
  float xin[kMxCh], cw[kMxCh][4], cb[kMxCh];
  // the head's dt and this thread's z, loaded with the conv inputs, and every
  // parameter of the step, so the step pays one memory latency
  const float dt_raw = ld_f32<COH>(row + 2 * d_inner + 2 * kMxN + h);
  const float zp = ld_f32<COH>(row + h * kMxP + p);
  const float dtb = dt_bias[h], alog = A_log[h], dskip = Dp[h];
#pragma unroll
  for (int t = 0; t < kMxCh; ++t) {
    const int i = tid + t * kMxThreads;
    if (i >= kMxP + 2 * kMxN) break;
    const int c = i < kMxP ? h * kMxP + i : d_inner + (i - kMxP);
    const u32x2 r2 = *reinterpret_cast<const u32x2*>(conv_b + (int64_t)c * 4);
    ring[t][0] = r2.x;
    ring[t][1] = r2.y;
    xin[t] = ld_f32<COH>(row + d_inner + c);
#pragma unroll
    for (int j = 0; j < 4; ++j) cw[t][j] = conv_w[(int64_t)c * 4 + j];
    cb[t] = conv_bias[c];
  }
  const int pos = pos_of();
#pragma unroll
  for (int t = 0; t < kMxCh; ++t) {
    const int i = tid + t * kMxThreads;
    if (i >= kMxP + 2 * kMxN) break;
    const int c = i < kMxP ? h * kMxP + i : d_inner + (i - kMxP);
    auto slot = [&](int k) {  // float16 of ring slot k (0 .. 3)
      const uint32_t wd = ring[t][k >> 1];
      return h2f((uint16_t)((k & 1) ? wd >> 16 : wd & 0xFFFFu));
    };
    float acc = cb[t];
#pragma unroll
    for (int j = 0; j < 3; ++j) acc = __builtin_fmaf(slot((pos + 1 + j) & 3), cw[t][j], acc);
    acc = __builtin_fmaf(xin[t], cw[t][3], acc);
    u[i] = mx_silu(acc);
    // the slot nobody reads; the shared B/C channels are written by head 0
    if (i < kMxP || h == 0) conv_b[(int64_t)c * 4 + pos] = f2h(xin[t]);
  }
  __syncthreads();

  const float dtp = mx_softplus(dt_raw + dtb);
  const float a = expf(-dtp * expf(alog));
  const float xp = u[p];
  const float dx = dtp * xp;
  uint16_t* sp = ssm_h + p * kMxN + 32 * q;
  float y = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t wv[4] = {sv[k].x, sv[k].y, sv[k].z, sv[k].w};
    uint32_t o[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int n0 = 32 * q + 8 * k + 2 * t;
      const float s0 = __builtin_fmaf(a, h2f((uint16_t)(wv[t] & 0xFFFFu)), dx * u[kMxP + n0]);
      const float s1 = __builtin_fmaf(a, h2f((uint16_t)(wv[t] >> 16)), dx * u[kMxP + n0 + 1]);
      y = __builtin_fmaf(s0, u[kMxP + kMxN + n0], y);
      y = __builtin_fmaf(s1, u[kMxP + kMxN + n0 + 1], y);
      o[t] = (uint32_t)f2h(s0) | ((uint32_t)f2h(s1) << 16);
    }
    st16(sp + 8 * k, u32x4{o[0], o[1], o[2], o[3]});
  }
  // the four threads of a channel (lanes 4p' .. 4p' + 3 of the wave)
  y += __uint_as_float(lane_xchg<1>(__float_as_uint(y)));
  y += __uint_as_float(lane_xchg<2>(__float_as_uint(y)));
  y = __builtin_fmaf(dskip, xp, y);
  const float g = y * mx_silu(zp);
  if (q == 0) st_f32<COH>(gated_b + h * kMxP + p, g);
  if (part == nullptr) return;
  // sum of g^2 over the head's 64 channels: each channel counted once (q = 0)
  float sq = q == 0 ? g * g : 0.f;
  sq += __uint_as_float(lane_xchg<1>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<2>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<4>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<8>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<16>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<32>(__float_as_uint(sq)));
  if ((tid & 63) == 0) wsum[tid >> 6] = sq;
  __syncthreads();
  if (tid == 0) st_f32<COH>(part, (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]));
}

}  // namespace tmk
