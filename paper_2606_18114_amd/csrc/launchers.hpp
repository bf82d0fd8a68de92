// Host-side launchers implemented in the kernel translation units.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include <atomic>

namespace tmk {

// Compute units of the current device (the persistent grids are sized by
// it), cached per device; safe to call from several host threads.
inline int current_cu_count() {
  constexpr int kMaxDev = 64;
  static std::atomic<int> cache[kMaxDev];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < kMaxDev) {
    const int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
    v = 256;
  if (dev < kMaxDev) cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

hipError_t launch_ternarize_pack(const float* W, int64_t N, int64_t K, int g, float eps,
                                 const float* row_mult, const float* tau_in, uint8_t* codes,
                                 float* scales,
                                 uint16_t* scales_f16, uint64_t* zero_count,
                                 hipStream_t stream);
// out[n, j] = sum over group j of row n of q * dW (float64 sums, float32 out)
hipError_t launch_group_code_dot(const uint8_t* codes, const float* dW, int64_t N, int64_t K,
                                 int g, float* out, hipStream_t stream);
// ds[n, j] = sum over group j of dWhat * (q - m w s/d^2), dw = dWhat m s/d
// (d = fl32(s + eps), m the float32 clip mask); dw may be NULL or dWhat
hipError_t launch_scale_ste_grad(const float* W, const uint8_t* codes, const float* scale,
                                 const float* dWhat, int64_t N, int64_t K, int g, float eps,
                                 float* ds, float* dw, hipStream_t stream);
// Y: float32 [M, N], or bfloat16 bits [M, N] when bf16_out.  tickets:
// NULL, or 2 * kFwdMaxTicketTiles words of caller memory through which the
// two parts of each cut tile meet (then Y is not cleared first)
constexpr int kFwdMaxTicketTiles = 1024;
hipError_t launch_tgemm_fwd(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int g, void* Y, bool bf16_out,
                            uint32_t* tickets, hipStream_t stream);
hipError_t launch_tgemm_bwd_dx(const uint16_t* dY, const uint8_t* codes, const float* scales,
                               int64_t M, int64_t N, int64_t K, int g, float* dX,
                               hipStream_t stream);
// the one-pass float16 form: a prepass writes fp16(dY * 2^e[m]), the row
// exponents and the scale maxima into workspace (dx_f16_workspace_bytes)
// (the scale maxima come from kDxScaleParts waves of the prepass)
constexpr int kDxScaleParts = 256;
inline int64_t dx_f16_workspace_bytes(int64_t M, int64_t N) {
  auto up = [](int64_t v) { return (v + 255) / 256 * 256; };
  return up(M * N * 2) + up(M * 4) + kDxScaleParts * 4;
}
hipError_t launch_tgemm_bwd_dx_f16(const uint16_t* dY, const uint8_t* codes, const float* scales,
                                   int64_t M, int64_t N, int64_t K, int g, float* dX,
                                   void* workspace, hipStream_t stream);
hipError_t launch_tgemm_bwd_dw(const uint16_t* dY, const uint16_t* X, int64_t M, int64_t N,
                               int64_t K, float* dW, int accumulate, hipStream_t stream);
// dst[0 .. n) = 0 (float32), by a plain fill kernel
hipError_t launch_fill_zero_f32(float* dst, int64_t n, hipStream_t stream);
// zeroes tiles t0 .. t0 + count - 1 of a float32 [rows, cols] array dealt in
// 256 x 256 tiles, tiles_c per row of tiles (cols % 4 == 0, 16-byte aligned)
hipError_t launch_zero_tiles_f32(float* out, int64_t rows, int64_t cols, int64_t tiles_c,
                                 int64_t t0, int64_t count, hipStream_t stream);
hipError_t launch_tgemv(const uint16_t* x, const uint8_t* codes, const uint16_t* s16, int count,
                        int B, int64_t N, int64_t K, int g, float* y, hipStream_t stream);
// batches of 9 .. 16 rows at g >= 64 on the bfloat16 matrix cores (the batch
// rows as the MFMA's A rows); same arguments and results as launch_tgemv
bool tgemv_b16_takes(int B, int g);
hipError_t launch_tgemv_b16(const uint16_t* x, const uint8_t* codes, const uint16_t* s16,
                            int count, int B, int64_t N, int64_t K, int g, float* y,
                            hipStream_t stream);
// two strided stacks of matrices (e.g. a decode token's in_proj and out_proj
// layers) in one launch; same g and B, everything else per stack
hipError_t launch_tgemv_pair(const uint16_t* x0, const uint8_t* c0, const uint16_t* s0, int n0,
                             int64_t N0, int64_t K0, float* y0, const uint16_t* x1,
                             const uint8_t* c1, const uint16_t* s1, int n1, int64_t N1,
                             int64_t K1, float* y1, int B, int g, hipStream_t stream);
// Fused decode projection: x = bf16(src / sqrt(mean(src^2) + eps) * nw) per
// batch row, y = (or +=, accum) x times the ternary matrix.  Shapes the
// kernel stages in one part (tgemv_rms_fits) only.
// (4 A rows per batch item and group, 512-column slots; 8 waves once K has
// eight slots, else 4; at most two 16-column pieces per thread)
inline bool tgemv_rms_fits(int B, int64_t K, int g) {
  const int H = g < 128 ? 128 / g : 1;
  const int64_t pieces = (K + 127) / 128 * 8;
  const int waves = (K + 511) / 512 >= 8 ? 8 : 4;
  return 4 * B * H <= 16 && B * pieces <= 2 * 64 * waves;
}
hipError_t launch_tgemv_rms(const float* src, const float* nw, float eps, const uint8_t* codes,
                            const uint16_t* s16, int B, int64_t N, int64_t K, int g, float* y,
                            int accum, hipStream_t stream);
// y[c, b, n] = sum_k x[c, b, k] * W16[c, n, k] (dense float16 weights)
hipError_t launch_dgemv(const uint16_t* x, const uint16_t* W16, int count, int B, int64_t N,
                        int64_t K, float* y, hipStream_t stream);
// the fused form of launch_tgemv_rms for one dense float16 matrix
hipError_t launch_dgemv_rms(const float* src, const float* nw, float eps, const uint16_t* W16,
                            int B, int64_t N, int64_t K, float* y, int accum,
                            hipStream_t stream);

// one Mamba-2 mixer decode step (headdim 64, d_state 128): conv ring step,
// float16 SSM update, gated RMSNorm -> bfloat16 out; workspace holds
// B * (d_inner + nheads) floats
hipError_t launch_mixer_step(const float* zxbcdt, int B, int nheads, uint16_t* conv_state,
                             int* conv_pos, uint16_t* ssm_state, const float* conv_w,
                             const float* conv_b, const float* dt_bias, const float* A_log,
                             const float* D, const float* norm_w, float eps, float* workspace,
                             uint16_t* out, hipStream_t stream);

// the same with the workspace in a file-scope device array of
// mixer_scratch_floats() floats (hipErrorInvalidValue when it does not fit)
int64_t mixer_scratch_floats();
hipError_t launch_mixer_step_noalloc(const float* zxbcdt, int B, int nheads,
                                     uint16_t* conv_state, int* conv_pos, uint16_t* ssm_state,
                                     const float* conv_w, const float* conv_b,
                                     const float* dt_bias, const float* A_log, const float* D,
                                     const float* norm_w, float eps, uint16_t* out,
                                     hipStream_t stream);
// the step up to the gated output g = y * SiLU(z) (float32 [B, d_inner], not
// normalized: the fused out_proj normalizes it), one launch; the conv ring
// position advances when the last workgroup is done
hipError_t launch_mixer_gate(const float* zxbcdt, int B, int nheads, uint16_t* conv_state,
                             int* conv_pos, uint16_t* ssm_state, const float* conv_w,
                             const float* conv_b, const float* dt_bias, const float* A_log,
                             const float* D, float* gated, hipStream_t stream);

// One decode token per batch row (batch 1 .. 4) through a stack of ternary
// Mamba-2 blocks in one launch with grid barriers (headdim 64, d_state 128,
// d_conv 4); arrays per block are stacked along a leading layer dimension.
constexpr int kDecodeStackMaxKept = 64;
constexpr int kDecodeStackMaxBatch = 4;
struct DecodeStackDesc {
  int n_layers, d_model, nheads, g, batch;
  float eps;
  const uint8_t* in_codes;    // [L, Z, d_model / 4], Z = 2 d_inner + 256 + nheads
  const uint16_t* in_s16;     // [L, Z, d_model / g]
  const uint8_t* out_codes;   // [L, d_model, d_inner / 4]
  const uint16_t* out_s16;    // [L, d_model, d_inner / g]
  const float* pre_w;         // [L, d_model]
  const float* conv_w;        // [L, conv_dim, 4], conv_dim = d_inner + 256
  const float* conv_b;        // [L, conv_dim]
  const float* dt_bias;       // [L, nheads]
  const float* A_log;         // [L, nheads]
  const float* D;             // [L, nheads]
  const float* norm_w;        // [L, d_inner]
  const float* final_w;       // [d_model]
  uint16_t* conv_state;       // [L, batch, conv_dim, 4] float16 ring
  int* conv_pos;              // [L] (one position for every batch row)
  uint16_t* ssm_state;        // [L, batch, nheads, 64, 128] float16
  // blocks kept in FP16: their indices (ascending), and their projections
  // (those blocks' entries of the code arenas are not read)
  int n_kept;
  int kept[kDecodeStackMaxKept];
  const uint16_t* in_w16;     // [n_kept, Z, d_model] float16
  const uint16_t* out_w16;    // [n_kept, d_model, d_inner] float16
};
// [barrier words and timeout flag: kDecodeStackSyncBytes] zx [batch, Z]
// gated [batch, d_inner] partial [batch, nheads] residual [batch, d_model],
// each piece 256-byte aligned
constexpr int kDecodeStackSyncBytes = 32768;
inline int64_t decode_stack_workspace_bytes(int d_model, int nheads, int batch) {
  auto up = [](int64_t v) { return (v + 255) / 256 * 256; };
  const int64_t b = batch, di = 64 * (int64_t)nheads, z = 2 * di + 256 + nheads;
  return kDecodeStackSyncBytes + up(b * z * 4) + up(b * di * 4) + up(b * nheads * 4) +
         up(b * d_model * 4);
}
hipError_t launch_decode_stack(const DecodeStackDesc& s, const float* emb, uint16_t* x_out,
                               void* workspace, hipStream_t stream);

// residual += y (y may be null); x = bf16(rmsnorm(residual) * w), B rows of D
hipError_t launch_residual_rmsnorm(float* residual, const float* y, int B, int64_t D,
                                   const float* w, float eps, uint16_t* x, hipStream_t stream);

}  // namespace tmk
