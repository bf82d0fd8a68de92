// One Mamba-2 mixer decode step between in_proj and out_proj: the part of a
// decoding layer the paper keeps in FP16 (Sec. 3.2; batch-1 decode, Sec. 8).
//
// Kernel 1, one workgroup per (head, batch row): the per-head step of
// mixer_dev.hpp (convolution step, float16 SSM update, gated output g =
// y * SiLU(z)); g (float32) and the head's sum of g^2 go to the workspace.
// The head's SSM state is loaded at the start, so its memory latency
// overlaps the convolution.
// (The fused decode runs kernel 1 alone and normalizes g in out_proj.)
// Kernel 2, one workgroup per batch row: the gated RMSNorm over all d_inner
// channels, out = bf16(g / sqrt(mean(g^2) + eps) * w), the bfloat16 input
// of out_proj (the per-head partial sums meet in a wave butterfly); and the
// convolution ring position advances, after every workgroup of kernel 1 is
// done.
#include <atomic>

#include "launchers.hpp"
#include "mixer_dev.hpp"

namespace tmk {

// grid (nheads, B); layout: zxbcdt [B, Z] with Z = 2 d_inner + 2 N + nheads,
// conv [B, conv_dim, 4] float16 ring, ssm [B, nheads, P, N] float16,
// gated [B, d_inner] and partial [B, nheads] float32.
// GATE (the fused decode's form): no partial sums (the fused out_proj takes
// its own), and the ring position advances here: every workgroup reads the
// position word by adding 4 to it (one atomic, issued first, whose result
// holds the position in its low two bits and the number of workgroups that
// came before in the rest), and the last one to arrive stores the next
// position with a zero count at its end.  No workgroup reads the word after
// the last one has.  The ring slots of a channel are loaded all four at
// once, before the position is known, and picked afterwards.
template <bool GATE>
__global__ __launch_bounds__(kMxThreads) void mixer_ssm_kernel(
    const float* __restrict__ zxbcdt, int nheads, uint16_t* __restrict__ conv,
    int* __restrict__ conv_pos, uint16_t* __restrict__ ssm,
    const float* __restrict__ conv_w, const float* __restrict__ conv_b,
    const float* __restrict__ dt_bias, const float* __restrict__ A_log,
    const float* __restrict__ Dp, float* __restrict__ gated, float* __restrict__ partial) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x;
  const int d_inner = nheads * kMxP;
  const int conv_dim = d_inner + 2 * kMxN;
  const int64_t Z = (int64_t)2 * d_inner + 2 * kMxN + nheads;
  __shared__ int pos_word;
  if (GATE && tid == 0) pos_word = atomicAdd(conv_pos, 4);
  uint16_t* ssm_h = ssm + ((int64_t)b * nheads + h) * kMxP * kMxN;
  u32x4 sv[4];
  mixer_state_load(ssm_h, tid, sv);
  auto pos_of = [&]() {
    if constexpr (GATE) {
      __syncthreads();  // the position word has arrived in LDS
      return pos_word & 3;
    } else {
      return conv_pos[0] & 3;
    }
  };
  mixer_head_step(zxbcdt + (int64_t)b * Z, h, nheads, conv + (int64_t)b * conv_dim * 4, ssm_h,
                  sv, pos_of, conv_w, conv_b, dt_bias, A_log, Dp, gated + (int64_t)b * d_inner,
                  GATE ? nullptr : partial + (int64_t)b * nheads + h);
  if constexpr (GATE) {
    if (tid == 0 && (pos_word >> 2) == (int)(gridDim.x * gridDim.y) - 1)
      atomicExch(conv_pos, (pos_word + 1) & 3);  // every other workgroup has read it
  }
}

// grid (B); out[b, i] = bf16(g[b, i] / sqrt(sum_h partial[b, h] / d_inner + eps) * w[i])
__global__ __launch_bounds__(kMxThreads) void mixer_norm_kernel(
    const float* __restrict__ gated, const float* __restrict__ partial, int nheads,
    const float* __restrict__ norm_w, float eps, uint16_t* __restrict__ out,
    int* __restrict__ conv_pos) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int d_inner = nheads * kMxP;
  __shared__ float wsum[kMxThreads / 64];
  float s2 = 0.f;
  for (int h = tid; h < nheads; h += kMxThreads) s2 += partial[(int64_t)b * nheads + h];
  s2 += __uint_as_float(lane_xchg<1>(__float_as_uint(s2)));
  s2 += __uint_as_float(lane_xchg<2>(__float_as_uint(s2)));
  s2 += __uint_as_float(lane_xchg<4>(__float_as_uint(s2)));
  s2 += __uint_as_float(lane_xchg<8>(__float_as_uint(s2)));
  s2 += __uint_as_float(lane_xchg<16>(__float_as_uint(s2)));
  s2 += __uint_as_float(lane_xchg<32>(__float_as_uint(s2)));
  if ((tid & 63) == 0) wsum[tid >> 6] = s2;
  __syncthreads();
  const float r = 1.f / sqrtf(((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) / (float)d_inner + eps);
  for (int i = tid; i < d_inner; i += kMxThreads) {
    const float v = gated[(int64_t)b * d_inner + i] * r * norm_w[i];
    const uint32_t bits = __float_as_uint(v);
    out[(int64_t)b * d_inner + i] = (uint16_t)((bits + 0x7FFFu + ((bits >> 16) & 1u)) >> 16);
  }
  if (b == 0 && tid == 0) conv_pos[0] = (conv_pos[0] + 1) & 3;
}

// grid (B): residual[b] += y[b] (y may be null), then
// x[b, i] = bf16(residual[b, i] / sqrt(mean(residual[b]^2) + eps) * w[i])
__global__ __launch_bounds__(kMxThreads) void residual_rmsnorm_kernel(
    float* __restrict__ residual, const float* __restrict__ y, int64_t D,
    const float* __restrict__ w, float eps, uint16_t* __restrict__ x) {
  constexpr int kReg = 16;  // values kept in registers per thread (D <= 4096)
  const int b = blockIdx.x;
  float* r = residual + (int64_t)b * D;
  const float* yy = y ? y + (int64_t)b * D : nullptr;
  __shared__ float wsum[kMxThreads / 64];
  float v[kReg];
  float sq = 0.f;
#pragma unroll
  for (int j = 0; j < kReg; ++j) {
    const int64_t i = threadIdx.x + (int64_t)j * kMxThreads;
    v[j] = i < D ? r[i] + (yy ? yy[i] : 0.f) : 0.f;
  }
#pragma unroll
  for (int j = 0; j < kReg; ++j) {
    const int64_t i = threadIdx.x + (int64_t)j * kMxThreads;
    if (yy && i < D) r[i] = v[j];
    sq = __builtin_fmaf(v[j], v[j], sq);
  }
  for (int64_t i = threadIdx.x + (int64_t)kReg * kMxThreads; i < D; i += kMxThreads) {
    float t = r[i];
    if (yy) {
      t += yy[i];
      r[i] = t;
    }
    sq = __builtin_fmaf(t, t, sq);
  }
  sq += __uint_as_float(lane_xchg<1>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<2>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<4>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<8>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<16>(__float_as_uint(sq)));
  sq += __uint_as_float(lane_xchg<32>(__float_as_uint(sq)));
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = sq;
  __syncthreads();
  const float scale = 1.f / sqrtf(((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) / (float)D + eps);
  auto put = [&](int64_t i, float t) {
    const uint32_t bits = __float_as_uint(t * scale * w[i]);
    x[(int64_t)b * D + i] = (uint16_t)((bits + 0x7FFFu + ((bits >> 16) & 1u)) >> 16);
  };
#pragma unroll
  for (int j = 0; j < kReg; ++j) {
    const int64_t i = threadIdx.x + (int64_t)j * kMxThreads;
    if (i < D) put(i, v[j]);
  }
  for (int64_t i = threadIdx.x + (int64_t)kReg * kMxThreads; i < D; i += kMxThreads) put(i, r[i]);
}

hipError_t launch_residual_rmsnorm(float* residual, const float* y, int B, int64_t D,
                                   const float* w, float eps, uint16_t* x, hipStream_t stream) {
  hipLaunchKernelGGL(residual_rmsnorm_kernel, dim3((unsigned)B), dim3(kMxThreads), 0, stream,
                     residual, y, D, w, eps, x);
  return hipGetLastError();
}

hipError_t launch_mixer_step(const float* zxbcdt, int B, int nheads, uint16_t* conv_state,
                             int* conv_pos, uint16_t* ssm_state, const float* conv_w,
                             const float* conv_b, const float* dt_bias, const float* A_log,
                             const float* D, const float* norm_w, float eps, float* workspace,
                             uint16_t* out, hipStream_t stream) {
  float* gated = workspace;
  float* partial = workspace + (int64_t)B * nheads * kMxP;
  hipLaunchKernelGGL(mixer_ssm_kernel<false>, dim3((unsigned)nheads, (unsigned)B),
                     dim3(kMxThreads), 0, stream, zxbcdt, nheads, conv_state, conv_pos,
                     ssm_state, conv_w, conv_b, dt_bias, A_log, D, gated, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mixer_norm_kernel, dim3((unsigned)B), dim3(kMxThreads), 0, stream, gated,
                     partial, nheads, norm_w, eps, out, conv_pos);
  return hipGetLastError();
}

hipError_t launch_mixer_gate(const float* zxbcdt, int B, int nheads, uint16_t* conv_state,
                             int* conv_pos, uint16_t* ssm_state, const float* conv_w,
                             const float* conv_b, const float* dt_bias, const float* A_log,
                             const float* D, float* gated, hipStream_t stream) {
  hipLaunchKernelGGL(mixer_ssm_kernel<true>, dim3((unsigned)nheads, (unsigned)B),
                     dim3(kMxThreads), 0, stream, zxbcdt, nheads, conv_state, conv_pos,
                     ssm_state, conv_w, conv_b, dt_bias, A_log, D, gated, nullptr);
  return hipGetLastError();
}

// Allocation-free variant: the workspace is a file-scope device array (one
// copy per GPU, kept until the process ends).  Host code never passes the
// array's name to a kernel: its device address is looked up once per device
// with hipGetSymbolAddress (with that device current) and cached.
constexpr int64_t kMixerScratchFloats = 16 * (8192 + 128);  // B * (d_inner + nheads) <= this
static __device__ __align__(256) float scratch[kMixerScratchFloats];

int64_t mixer_scratch_floats() { return kMixerScratchFloats; }

hipError_t launch_mixer_step_noalloc(const float* zxbcdt, int B, int nheads,
                                     uint16_t* conv_state, int* conv_pos, uint16_t* ssm_state,
                                     const float* conv_w, const float* conv_b,
                                     const float* dt_bias, const float* A_log, const float* D,
                                     const float* norm_w, float eps, uint16_t* out,
                                     hipStream_t stream) {
  if ((int64_t)B * (nheads * kMxP + nheads) > kMixerScratchFloats) return hipErrorInvalidValue;
  constexpr int kMaxDev = 64;
  static std::atomic<float*> ptrs[kMaxDev];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  float* ws = ptrs[dev].load(std::memory_order_acquire);
  if (ws == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    ws = static_cast<float*>(p);
    ptrs[dev].store(ws, std::memory_order_release);
  }
  return launch_mixer_step(zxbcdt, B, nheads, conv_state, conv_pos, ssm_state, conv_w, conv_b,
                           dt_bias, A_log, D, norm_w, eps, ws, out, stream);
}

}  // namespace tmk
