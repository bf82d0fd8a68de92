/*
 * tmamba.h — C ABI of the grouped-absmean ternary (W1.58A16) linear layer
 * for AMD MI355X (gfx950).
 *
 * The operation (paper: "Ternary Mamba: Grouped Quantization-Aware Training
 * of W1.58A16 State Space Models", Sec. 3.1, TernaryLinear Module):
 *   - the latent weight W [N, K] (out x in) is split into groups of g
 *     consecutive input-dimension elements of one output row;
 *   - group scale s[n, j] = mean_i |W[n, j*g + i]|, recomputed on every call
 *     (not a learned parameter);
 *   - code q[n, k] = round(clip(W[n, k] / (s + eps), -1, 1)) in {-1, 0, +1},
 *     round-half-to-even;
 *   - dequantized weight What[n, k] = s[n, k/g] * q[n, k];
 *   - forward Y = X . What^T; the straight-through estimator passes the
 *     gradient through the quantizer unchanged, so dX = dY . What and
 *     dW = dY^T . X.
 * Deployment storage is 2-bit codes plus per-group scales (Sec. 8).
 *
 * Conventions for every call
 *   - Every array pointer is DEVICE memory, allocated and owned by the caller.
 *     The library allocates and frees nothing, keeps no mutable global state
 *     beyond a per-device cache of the CU count, and is safe to call from
 *     several host threads.
 *   - Any clearing a call needs is done by a fill kernel on `stream`, never a
 *     memset node, so the calls can be captured into a HIP graph.
 *   - Arrays are dense, row-major, with the shapes given per call.  bfloat16
 *     data is passed as uint16_t bit patterns.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the default
 *     stream) and the call returns without synchronizing.  Device faults, if
 *     any, surface at the caller's next synchronization.
 *   - All arguments are checked on the host before anything is enqueued.
 *     On any error nothing is enqueued and a status code is returned: no
 *     exceptions cross the ABI, nothing aborts, nothing is printed.
 *   - Outputs must not overlap inputs or each other (TM_EINVAL).
 *   - Group sizes: g in {32, 64, 128, 256, 512}; K % g == 0 and K % 64 == 0.
 *
 * Packed code format (one row = K/4 bytes = K/16 little-endian uint32 words;
 * word w holds elements k = 16*w + e, e = 0..15):
 *   element e = 2*i   at bits [2*i,      2*i + 2)
 *   element e = 2*i+1 at bits [16 + 2*i, 16 + 2*i + 2)
 *   2-bit value = two's complement of the code: 00 -> 0, 01 -> +1, 11 -> -1.
 *   10 is never written; the kernels read it as 0.
 */
#ifndef TMAMBA_H
#define TMAMBA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TM_OK = 0,
  TM_EINVAL = 1,   /* null required pointer, overlapping arrays, bad eps/flag */
  TM_ESHAPE = 2,   /* a size < 1, K % g, K % 64, g not allowed, B/count range */
  TM_EALIGN = 3,   /* a pointer below its required alignment */
  TM_EHIP = 4,     /* the HIP runtime rejected a launch */
  TM_ENOTIMPL = 5  /* reserved */
} tm_status;

typedef struct ihipStream_t* tm_stream; /* the same type as hipStream_t */

#define TM_ABI_VERSION 15

/* ABI version of the loaded library (TM_ABI_VERSION it was built with). */
int tm_abi_version(void);

/* Human-readable name of a status code (static storage; never NULL). */
const char* tm_status_str(tm_status s);

/*
 * tm_ternarize_pack — Sec. 3.1 (group scale, ternary code) and Sec. 8 (packed
 * 2-bit storage), plus the zero-code count behind the zero ratio of Sec. 3.1
 * and Table 1.  One pass over W.
 *
 *   W           float32 [N, K]            in   (16-byte aligned, finite)
 *   N, K, g     K % g == 0, K % 64 == 0
 *   eps         float32, finite, >= 0; added to the scale before the
 *               division only (eps = 0 is the paper's formula)
 *   codes       uint8 [N, K/4]            out  (16-byte aligned)
 *   scales      float32 [N, K/g]          out  (4-byte aligned): the group
 *               mean, accumulated in float64 and rounded once to float32
 *   scales_f16  uint16 [N, K/g] or NULL   out  float16 bits, RNE of `scales`
 *   zero_count  uint64 [1] or NULL        out  number of zero codes; set on
 *               the stream (zeroed, then accumulated)
 * The code decision is the float32 one: q = 0 exactly when the float32
 * quotient |W| / fl32(s + eps) rounds to at most 1/2.
 */
tm_status tm_ternarize_pack(const float* W, int64_t N, int64_t K, int32_t g,
                            float eps, uint8_t* codes, float* scales,
                            uint16_t* scales_f16, uint64_t* zero_count,
                            tm_stream stream);

/*
 * tm_tgemm_fwd — Sec. 3.1 forward: Y = X . What^T with What = q * s.
 *
 *   X       bf16 [M, K]      in   (16-byte aligned)
 *   codes   uint8 [N, K/4]   in   packed codes (16-byte aligned)
 *   scales  float32 [N, K/g] in   (4-byte aligned)
 *   Y       float32 [M, N]   out  (16-byte aligned)
 *   K <= 2^22 and N <= 2^26 (TM_ESHAPE otherwise).
 * Products are exact (bf16 times {-1,0,1}) and accumulated in float32 on the
 * matrix cores; the group scale is applied in float32 per group.  Groups
 * whose scale is 0 contribute 0 whatever their codes.  Precondition (met by
 * any weights that are not extreme): within a row n, the largest nonzero
 * scale divided by the smallest, times sum_k |X[m, k]|, stays below 1e38.
 * Tiles of 256 x 256 outputs are spread over one workgroup per CU; when the
 * tile count is not a multiple of the CU count, the tiles left over are cut
 * along K and their parts add into Y with float32 atomics (those rows of Y
 * are cleared first).  Their elements may then differ in the last bits from
 * one call to the next (two parts add exactly in either order).
 */
tm_status tm_tgemm_fwd(const uint16_t* X, const uint8_t* codes,
                       const float* scales, int64_t M, int64_t N, int64_t K,
                       int32_t g, float* Y, tm_stream stream);

/*
 * tm_tgemm_fwd_ws — tm_tgemm_fwd with a small workspace through which the two
 * parts of each cut tile meet (Sec. 3.1, the same product): when the
 * tiles left over are cut in two along K, the part that finishes first
 * writes its sums into Y and the second adds its own to them, so Y needs no
 * clearing, the parts issue half the atomics, and repeated calls give
 * identical bits (two addends).  Tiles cut into more parts, and launches
 * with fewer than 16 cut tiles, add with atomics as in tm_tgemm_fwd.
 *   workspace        device memory owned by the caller, at least
 *                    tm_tgemm_fwd_workspace() bytes, 4-byte aligned,
 *                    overlapping no other argument; its contents are
 *                    scratch (cleared by the call, nothing kept after it)
 *   workspace_bytes  its size (TM_ESHAPE if too small)
 *   every other argument, limit and status as for tm_tgemm_fwd.
 * The second part of a cut tile waits (bounded) for the first, which is
 * already running when the wait starts.  Calls that share a workspace must
 * not run concurrently.
 */
tm_status tm_tgemm_fwd_ws(const uint16_t* X, const uint8_t* codes,
                          const float* scales, int64_t M, int64_t N, int64_t K,
                          int32_t g, float* Y, void* workspace,
                          int64_t workspace_bytes, tm_stream stream);

/* Workspace bytes of tm_tgemm_fwd_ws (independent of the shape). */
int64_t tm_tgemm_fwd_workspace(void);

/*
 * tm_tgemm_fwd_bf16 — tm_tgemm_fwd with the output in bfloat16: each float32
 * result is rounded to nearest even once (relative error <= 2^-9 per
 * element), as a bfloat16 model stores a linear layer's output; the gradient
 * arriving for it is then bfloat16 too, so the backward calls read it
 * without a cast.  Tiles are never cut along K here, so repeated calls give
 * identical bits.
 *   Y  bfloat16 bits [M, N]  out  (16-byte aligned)
 *   every other argument, limit and status as for tm_tgemm_fwd.
 */
tm_status tm_tgemm_fwd_bf16(const uint16_t* X, const uint8_t* codes,
                            const float* scales, int64_t M, int64_t N, int64_t K,
                            int32_t g, uint16_t* Y, tm_stream stream);

/*
 * tm_tgemm_bwd_dx — Sec. 3.1 straight-through backward w.r.t. the input:
 * dX = dY . What (contraction over N).
 *
 *   dY      bf16 [M, N]      in   (16-byte aligned; N % 8 == 0)
 *   codes   uint8 [N, K/4]   in   the codes of the forward call
 *   scales  float32 [N, K/g] in   the scales of the forward call
 *   dX      float32 [M, K]   out  (16-byte aligned)
 *   N <= 2^22 and K <= 2^26 (TM_ESHAPE otherwise)
 * The scale varies along the contraction, so each dequantized weight is
 * split into two bfloat16 terms (hi + lo) whose sum carries 16 bits of the
 * float32 scale; both terms run on the matrix cores.  When there are more
 * 256 x 256 output tiles than compute units and their count is not a
 * multiple of it, some tiles are split along N and reduced with float32
 * atomic adds, so the last bits of dX then depend on the summation order.
 */
tm_status tm_tgemm_bwd_dx(const uint16_t* dY, const uint8_t* codes,
                          const float* scales, int64_t M, int64_t N, int64_t K,
                          int32_t g, float* dX, tm_stream stream);

/*
 * tm_tgemm_bwd_dx_f16 — the same product (Sec. 3.1, straight-through
 * backward w.r.t. the input) in one float16 pass on the matrix cores.
 *
 *   dY, codes, scales, dX   as for tm_tgemm_bwd_dx (same limits, N % 8 == 0)
 *   workspace               device memory owned by the caller, at least
 *                           tm_tgemm_bwd_dx_f16_workspace(M, N) bytes,
 *                           256-byte aligned, overlapping no other argument;
 *                           its contents are scratch (nothing need be set
 *                           before the call, nothing is kept after it)
 *   workspace_bytes         its size (TM_ESHAPE if too small)
 * A prepass writes fp16(dY * 2^e[m]) into the workspace, with one power of
 * two per row of dY that puts the row's largest magnitude in [2^14, 2^15)
 * (every value within 2^28 of it converts exactly); the weight operand is
 * q * fp16(s * 2^t) with one power of two for the tensor (largest |s| in
 * [2^14, 2^15)); products are exact in float32, accumulated in float32, and
 * scaled back by 2^-(e[m] + t) in the store.  Each dequantized weight so
 * carries a relative error of at most 2^-11, which bounds every output by
 * 2^-11 * sum_n |dY[m, n] q[n, k] s| plus float32 accumulation (about 2e-4
 * relative Frobenius error on Gaussian weights).  Scales may have either
 * sign; dY must be finite.  Cut tiles and atomics as for tm_tgemm_bwd_dx.
 * Calls that share a workspace must not run concurrently.
 */
tm_status tm_tgemm_bwd_dx_f16(const uint16_t* dY, const uint8_t* codes,
                              const float* scales, int64_t M, int64_t N,
                              int64_t K, int32_t g, float* dX, void* workspace,
                              int64_t workspace_bytes, tm_stream stream);

/* Workspace bytes tm_tgemm_bwd_dx_f16 needs for an M x N dY (-1 if M or N
 * is below 1 or the size overflows). */
int64_t tm_tgemm_bwd_dx_f16_workspace(int64_t M, int64_t N);

/*
 * tm_tgemm_bwd_dw_ste — Sec. 3.1 straight-through backward w.r.t. the latent
 * weight (identity estimator: no clip mask, no gradient through the scale):
 * dW = dY^T . X (contraction over the M tokens).
 *
 *   dY          bf16 [M, N]    in   (16-byte aligned; N % 8 == 0)
 *   X           bf16 [M, K]    in   (16-byte aligned)
 *   dW          float32 [N, K] out  (16-byte aligned)
 *   accumulate  0: dW = dY^T X;  1: dW += dY^T X
 *   N, K <= 2^26 (TM_ESHAPE otherwise)
 * The token dimension is split across workgroups and reduced with float32
 * atomic adds, so the last bits of dW depend on the summation order.
 */
tm_status tm_tgemm_bwd_dw_ste(const uint16_t* dY, const uint16_t* X,
                              int64_t M, int64_t N, int64_t K, float* dW,
                              int32_t accumulate, tm_stream stream);

/*
 * tm_tgemv — decode-time product with packed weights (Sec. 8: batch-1
 * decoding is bound by weight traffic), strided-batched over `count`
 * same-shape matrices (e.g. the 48 in_proj layers):
 *   y[c, b, n] = sum_k x[c, b, k] * q_c[n, k] * s16_c[n, k/g]
 *
 *   x           bf16 [count, B, K]       in   (16-byte aligned)
 *   codes       uint8 [count, N, K/4]    in   (16-byte aligned)
 *   scales_f16  uint16 [count, N, K/g]   in   float16 bits (2-byte aligned)
 *   count       1 .. 65535;  B  1 .. 16;  N * K / 4 <= 2^31 (bytes per matrix)
 *   y           float32 [count, B, N]    out  (16-byte aligned)
 * Each 32-column block of a row of x is split into FP8 terms whose
 * power-of-two scales are taken from the block itself (two magnitude
 * classes of two terms each), so every element within 2^16 of its block's
 * largest magnitude is represented exactly, and smaller ones err by less
 * than 2^-19 of that maximum; an outlier affects only its own block.  The
 * matrix cores add the exact products at float32-like precision and the
 * float16 scale is applied in float32 per group.  x must be finite.
 * Results are deterministic for a given shape and count.  A launch with few
 * row blocks (fewer than two per CU, e.g. count = 1) splits K across the
 * waves of a workgroup and adds the parts in a fixed order, so its last bits
 * can differ from the same matrix inside a larger launch.
 * Batches of 9 .. 16 rows at g >= 64 take the bfloat16 matrix cores instead:
 * the bfloat16 x times the exact 2q of the codes (exact products, float32
 * sums), the float16 scale applied in float32 per group, one workgroup per
 * matrix and 16-row block with the K range split over its waves in a fixed
 * order (deterministic); tm_tgemv_pair then launches each stack on its own.
 */
tm_status tm_tgemv(const uint16_t* x, const uint8_t* codes,
                   const uint16_t* scales_f16, int32_t count, int32_t B,
                   int64_t N, int64_t K, int32_t g, float* y, tm_stream stream);

/*
 * tm_tgemv_pair — the decode product of tm_tgemv (Sec. 8, batch-1 decoding
 * bound by weight traffic) over two strided stacks in one launch, e.g. all
 * in_proj layers and all out_proj layers of a decode token:
 *   y0[c, b, n] = sum_k x0[c, b, k] * q0_c[n, k] * s0_c[n, k/g]  (c < count0)
 *   y1[c, b, n] = sum_k x1[c, b, k] * q1_c[n, k] * s1_c[n, k/g]  (c < count1)
 * Each stack's arguments, layout, alignment and limits are those of
 * tm_tgemv; the stacks share B and g.  Neither output may overlap the other
 * or any input.  The workgroups of both stacks form one grid (those of the
 * stack with the longer rows first), so the GPU does not drain between the
 * stacks.  Shapes
 * whose staging differs between the stacks run as two launches instead.
 * Results are deterministic and equal tm_tgemv's on the same stack bit for
 * bit, except where tm_tgemv splits K for a stack of few row blocks (fewer
 * than two per CU): there the last bits can differ.
 */
tm_status tm_tgemv_pair(const uint16_t* x0, const uint8_t* codes0,
                        const uint16_t* scales0, int32_t count0, int64_t N0,
                        int64_t K0, float* y0, const uint16_t* x1,
                        const uint8_t* codes1, const uint16_t* scales1,
                        int32_t count1, int64_t N1, int64_t K1, float* y1,
                        int32_t B, int32_t g, tm_stream stream);

/*
 * tm_dgemv — decode-time product of a layer kept in FP16 (Sec. 7,
 * layer-selective quantization: the first and last blocks are not
 * ternarized), strided-batched like tm_tgemv:
 *   y[c, b, n] = sum_k x[c, b, k] * W16[c, n, k]
 *
 *   x      bf16 [count, B, K]     in   (16-byte aligned)
 *   W16    float16 bits [count, N, K]  in   (16-byte aligned)
 *   count  1 .. 65535;  B  1 .. 8;  K % 64 == 0 and B * K <= 16384
 *   y      float32 [count, B, N]  out  (4-byte aligned)
 * Each product of a float16 weight and the float32 value of a bfloat16
 * activation is exact; they are summed with float32 fused multiply-adds and
 * a float32 butterfly across lanes, in a fixed order (deterministic).
 */
tm_status tm_dgemv(const uint16_t* x, const uint16_t* W16, int32_t count, int32_t B, int64_t N,
                   int64_t K, float* y, tm_stream stream);

/*
 * tm_residual_rmsnorm — the Mamba-2 block wrapper around the mixer in
 * decode: the residual stream takes the previous layer's out_proj output,
 * and the pre-norm gives the next layer's in_proj input:
 *   residual[b] += y[b]   (skipped when y is NULL);
 *   x[b, i] = bf16(residual[b, i] / sqrt(mean_i(residual[b, i]^2) + eps) * w[i]).
 *   residual  float32 [B, D]  in/out;  y  float32 [B, D] in or NULL
 *   w         float32 [D];  eps float32, finite, >= 0
 *   x         bfloat16 bits [B, D]  out
 *   B 1 .. 65535;  arrays must not overlap
 */
tm_status tm_residual_rmsnorm(float* residual, const float* y, int32_t B, int64_t D,
                              const float* w, float eps, uint16_t* x, tm_stream stream);

/*
 * tm_mixer_step — one Mamba-2 mixer decode step between in_proj and
 * out_proj, the part of a decoding layer kept in FP16 (Sec. 3.2: the
 * convolution, SSM parameters and state are not ternarized; Sec. 8:
 * batch-1 decode).  Per token b, with d_inner = nheads * 64, d_state = 128,
 * conv_dim = d_inner + 2 d_state and zxbcdt[b] = [z | xBC | dt] (in_proj's
 * output, widths d_inner | conv_dim | nheads):
 *   u = SiLU(conv step of xBC: window = the 3 previous inputs and xBC,
 *            u[c] = conv_b[c] + sum_t window[t] conv_w[c, t]);
 *   x, B, C = u[:d_inner], u[d_inner:d_inner+128], u[d_inner+128:];
 *   dt' = softplus(dt + dt_bias[h]);  a = exp(-dt' exp(A_log[h]));
 *   S[h,p,n] <- a S[h,p,n] + dt' x[h,p] B[n];  y = S C + D[h] x;
 *   g = y * SiLU(z);  out[b] = bf16(g / sqrt(mean(g^2) + eps) * norm_w).
 *
 *   zxbcdt      float32 [B, 2 d_inner + 2 d_state + nheads]   in
 *   B 1 .. 65535;  nheads 1 .. 4096;  headdim == 64;  d_state == 128
 *   conv_state  float16 [B, conv_dim, 4]   in/out (8-byte aligned): a ring
 *               of the last 4 inputs per channel; slot (pos + j) % 4 holds
 *               the j-th oldest, j = 0 .. 3 (pos = 0: slots in time order)
 *   conv_pos    int32 [1]   in/out: pos, advanced by one (mod 4) per call
 *   ssm_state   float16 [B, nheads, 64, 128]  in/out (16-byte aligned);
 *               updated in float32 and rounded once to float16
 *   conv_w      float32 [conv_dim, 4] (oldest tap first);  conv_b [conv_dim]
 *   dt_bias, A_log, D  float32 [nheads];  norm_w  float32 [d_inner]
 *   eps         float32, finite, >= 0
 *   workspace   float32 [B * (d_inner + nheads)]  scratch owned by the caller
 *               (4-byte aligned): the gated values and per-head sums of
 *               squares between the two launches
 *   out         bfloat16 bits [B, d_inner]  out: out_proj's input
 * Two launches on `stream`: the step (a workgroup per head and token), then
 * the normalization (a workgroup per token), which also advances conv_pos.
 * The state arrays, conv_pos, workspace and out must not overlap each other
 * or the inputs; calls that share state or workspace must not run
 * concurrently.
 */
tm_status tm_mixer_step(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                        int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                        uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                        const float* dt_bias, const float* A_log, const float* D,
                        const float* norm_w, float eps, float* workspace, uint16_t* out,
                        tm_stream stream);

/*
 * tm_mixer_step_noalloc — tm_mixer_step for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses
 * that forbid hipMalloc): the same computation and kernels, with the
 * workspace taken from a file-scope device array of the library instead of
 * an argument.  That array holds B * (d_inner + nheads) <= 16 * (8192 + 128)
 * floats (larger calls return TM_ESHAPE); each GPU the library runs on has
 * its own copy, kept until the process ends, whose address is looked up
 * once per device on the first call.  The call allocates nothing.  Every
 * call on a GPU shares that GPU's array: calls on one GPU that overlap in
 * time (different streams, host threads) race on it and must be serialized
 * by the caller.  All other arguments, checks and results as tm_mixer_step.
 */
tm_status tm_mixer_step_noalloc(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                                int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                                uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                                const float* dt_bias, const float* A_log, const float* D,
                                const float* norm_w, float eps, uint16_t* out,
                                tm_stream stream);

/*
 * The fused decode block (Sec. 8, batch-1 decode: a token streams each
 * layer's weights once; Sec. 3.2: the state update between the projections
 * stays FP16).  A Mamba-2 block in layer order runs three launches:
 *   zx  = tm_tgemv_rms(residual, w_pre)           pre-norm + in_proj
 *   g   = tm_mixer_gate(zx, states)               conv + SSM step + gate
 *   residual += tm_tgemv_rms(g, norm_w, acc = 1)  gated norm + out_proj
 * (tm_dgemv_rms for a layer kept in FP16).  The normalizations are folded
 * into the products' activation staging: every workgroup normalizes the
 * whole source row itself, so no launch exists only to normalize.
 *
 * tm_tgemv_rms — one packed matrix applied to normalized float32 rows:
 *   x[b, k] = bf16(src[b, k] / sqrt(mean_k(src[b, k]^2) + eps) * norm_w[k]);
 *   y[b, n] = sum_k x[b, k] q[n, k] s16[n, k/g]   (accumulate 0), or
 *   y[b, n] += that sum                           (accumulate 1).
 *   src         float32 [B, K]   in   (16-byte aligned)
 *   norm_w      float32 [K]      in   (16-byte aligned)
 *   eps         float32, finite, >= 0
 *   codes, scales_f16, g   as tm_tgemv with count = 1
 *   B  1 .. 16 with 4 B (128 / g if g < 128, else 1) <= 16 and
 *      B * ceil(K / 128) * 8 <= 512 (1024 when K > 3584): the shapes whose
 *      rows one workgroup stages at once (TM_ESHAPE otherwise)
 *   y           float32 [B, N]   out or in/out (16-byte aligned)
 * x is split and multiplied as in tm_tgemv.  The row sums of squares are
 * taken in a fixed order (deterministic results).  y must not overlap the
 * inputs.
 */
tm_status tm_tgemv_rms(const float* src, const float* norm_w, float eps, const uint8_t* codes,
                       const uint16_t* scales_f16, int32_t B, int64_t N, int64_t K, int32_t g,
                       float* y, int32_t accumulate, tm_stream stream);

/*
 * tm_dgemv_rms — tm_tgemv_rms for one matrix kept in FP16 (Sec. 7):
 * x as there, y[b, n] (+)= sum_k x[b, k] W16[n, k], summed as tm_dgemv.
 *   src float32 [B, K], norm_w float32 [K] (16-byte aligned); W16 as tm_dgemv
 *   B 1 .. 8;  K % 64 == 0 and B * K <= 16384;  y float32 [B, N] (4-byte aligned)
 */
tm_status tm_dgemv_rms(const float* src, const float* norm_w, float eps, const uint16_t* W16,
                       int32_t B, int64_t N, int64_t K, float* y, int32_t accumulate,
                       tm_stream stream);

/*
 * tm_mixer_gate — tm_mixer_step up to the gated values, in one launch:
 *   gated[b] = g = y * SiLU(z)   (float32 [B, d_inner], not normalized)
 * with the same convolution, state update and arguments as tm_mixer_step
 * (no norm_w, eps or workspace).  The convolution ring position advances
 * inside the launch: conv_pos[0] & 3 is the position; every workgroup adds
 * 4 once it has read it and the last one stores the next position, so
 * between calls conv_pos[0] holds just the position, as for tm_mixer_step
 * (either call continues the other's ring).  gated must not overlap the
 * other arrays.
 */
tm_status tm_mixer_gate(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                        int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                        uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                        const float* dt_bias, const float* A_log, const float* D, float* gated,
                        tm_stream stream);

/*
 * A stack of ternary Mamba-2 blocks for whole-stack decoding (Sec. 8:
 * small-batch decoding, bound by the weight traffic; Sec. 3.2: the mixer
 * and its states stay in FP16).  Every array is device memory, stacked along
 * a leading layer dimension L = n_layers; d_inner = 64 nheads, d_state 128,
 * d_conv 4, Z = 2 d_inner + 256 + nheads, conv_dim = d_inner + 256.
 *   n_layers >= 1; d_model and d_inner multiples of g and of 64, at most 4096
 *   and 8192 (the workgroup's x pairs); g in {64, 128, 256}; 1 <= nheads <= the
 *   device's CU count; eps: RMSNorm epsilon (finite, >= 0)
 *   batch      1 .. 4 tokens decoded together (one per batch row); above 1,
 *              d_model <= 2048, d_inner <= 4096 and nheads * batch <= the
 *              device's CU count
 *   in_codes   uint8 [L, Z, d_model/4]        in_scales  fp16 [L, Z, d_model/g]
 *   out_codes  uint8 [L, d_model, d_inner/4]  out_scales fp16 [L, d_model, d_inner/g]
 *   pre_w      float32 [L, d_model]   the block's pre-norm weight
 *   conv_w     float32 [L, conv_dim, 4], conv_b float32 [L, conv_dim]
 *   dt_bias, A_log, D  float32 [L, nheads]
 *   norm_w     float32 [L, d_inner]   the gated RMSNorm's weight
 *   final_w    float32 [d_model]      the final norm's weight
 *   conv_state fp16 [L, batch, conv_dim, 4] (8-byte aligned), conv_pos int32
 *              [L] (one ring position for every batch row),
 *   ssm_state  fp16 [L, batch, nheads, 64, 128] (16-byte aligned): the decode
 *              state, in and out, as for tm_mixer_step with B = batch
 * Codes, pre_w, norm_w and final_w 16-byte aligned, scales 2-byte, the other
 * float arrays 4-byte.
 * Blocks kept in FP16 (Sec. 7, layer-selective quantization), optional:
 *   n_kept     0 .. 64 (0: every block ternary; the fields below unused)
 *   kept       HOST array int32 [n_kept]: the kept blocks' indices, strictly
 *              ascending, each < n_layers (read during the call)
 *   in_w16     float16 [n_kept, Z, d_model], out_w16 float16 [n_kept,
 *              d_model, d_inner]: their projections, in the order of kept
 *              (16-byte aligned); the code and scale arenas keep their
 *              [n_layers, ...] shape, the kept blocks' entries unread
 */
typedef struct {
  int32_t n_layers, d_model, nheads, g;
  float eps;
  const uint8_t* in_codes;
  const uint16_t* in_scales;
  const uint8_t* out_codes;
  const uint16_t* out_scales;
  const float* pre_w;
  const float* conv_w;
  const float* conv_b;
  const float* dt_bias;
  const float* A_log;
  const float* D;
  const float* norm_w;
  const float* final_w;
  uint16_t* conv_state;
  int32_t* conv_pos;
  uint16_t* ssm_state;
  int32_t n_kept;
  const int32_t* kept;
  const uint16_t* in_w16;
  const uint16_t* out_w16;
  int32_t batch;
} tm_mamba2_stack;

/*
 * tm_mamba2_decode_token — one decode token per batch row through every
 * block of the stack in a single launch: per block, in layer order,
 *   zx        = in_proj(bf16(rmsnorm(residual) * pre_w))        (tm_tgemv_rms)
 *   g         = conv + FP16 SSM step + y * SiLU(z)               (tm_mixer_gate)
 *   residual += out_proj(bf16(rmsnorm(g) * norm_w))             (tm_tgemv_rms)
 * with residual = emb for the first block, then
 *   x_out = bf16(rmsnorm(residual) * final_w).
 * A block kept in FP16 takes its two projections from in_w16 / out_w16
 * (tm_dgemv_rms: each float16 weight times the float32 value of the
 * bfloat16 x, float32 sums).
 *   stack      host pointer to the description above (read during the call)
 *   emb        float32 [batch, d_model] in (16-byte aligned);  x_out  bf16
 *              [batch, d_model] out (4-byte aligned: stored in pairs)
 *   workspace  device scratch of tm_mamba2_decode_workspace(d_model, nheads,
 *              batch) bytes, 256-byte aligned, owned by the caller; nothing need be
 *              set before the call.  Its uint32 word 6144 is nonzero after a
 *              call whose grid barrier gave up waiting; the outputs and
 *              states of such a call are not valid.
 * One workgroup per CU; the blocks' phases are separated by grid barriers
 * (three per block) instead of kernel launches, so every workgroup must be
 * resident at once: on an otherwise idle GPU each CU takes one and they all
 * start together; other kernels running at the same time (other streams or
 * processes) can delay some, and a barrier waits for them for tens of
 * milliseconds before it gives up and sets the flag above.  The mixer step
 * takes one workgroup per head and batch row.
 * The ternary products take the bfloat16 x against the codes (exact
 * products, float32 sums, float16 group scale in float32), so they agree
 * with tm_tgemv_rms to float32 rounding; the normalizations sum in a
 * different order, which can move an x element by one bfloat16 step.
 * Calls sharing the state arrays or the workspace must not overlap in time.
 */
tm_status tm_mamba2_decode_token(const tm_mamba2_stack* stack, const float* emb,
                                 uint16_t* x_out, void* workspace, int64_t workspace_bytes,
                                 tm_stream stream);

/* Workspace bytes of tm_mamba2_decode_token (-1 for sizes out of range). */
int64_t tm_mamba2_decode_workspace(int32_t d_model, int32_t nheads, int32_t batch);

/*
 * Scale-parameterization variants (paper appendix, Decoupled Quantization
 * Ablations; Sec. 4, Zero-Ratio Collapse).
 *
 * tm_ternarize_pack_thresh — tm_ternarize_pack with a per-row rounding
 * threshold: row n's codes divide by fl32(fl32(row_mult[n] * s) + eps)
 * instead of fl32(s + eps).  The stored scales are still the group absmean
 * s, which keeps scaling the codes.  This is the appendix's asymmetric gate
 * thresholds: 0.8 x absmean on in_proj rows 0-4095, 1 elsewhere.
 *   row_mult   float32 [N] or NULL (NULL: every multiplier 1, the same as
 *              tm_ternarize_pack); 4-byte aligned, device memory.  Each
 *              value must be finite and > 0; other values give unspecified
 *              codes (they are not checked: the array is on the device).
 *   every other argument as for tm_ternarize_pack.
 */
tm_status tm_ternarize_pack_thresh(const float* W, int64_t N, int64_t K, int32_t g,
                                   float eps, const float* row_mult, uint8_t* codes,
                                   float* scales, uint16_t* scales_f16,
                                   uint64_t* zero_count, tm_stream stream);

/*
 * tm_ternarize_codes — the codes of a2/a3 against caller-given per-group
 * thresholds instead of the absmean:
 *   q[n, k] = RoundClip(W[n, k] / fl32(tau[n, k/g] + eps), -1, 1),
 * packed and counted as by tm_ternarize_pack.  This is the forward of the
 * learnable-scale layer of Sec. 4 (tau = the learned s_g, which also scales
 * the codes) and of a fixed threshold tau_g chosen by the caller.
 *   W     float32 [N, K]    in   (16-byte aligned)
 *   tau   float32 [N, K/g]  in   (4-byte aligned); each value finite and
 *         > 0, else the codes are unspecified (device data is not checked)
 *   codes uint8 [N, K/4]    out  (16-byte aligned)
 *   zero_count uint64 [1]   out, or NULL (8-byte aligned); zeroed on-stream
 *   No scales are written.  Status codes and ownership as tm_ternarize_pack.
 */
tm_status tm_ternarize_codes(const float* W, int64_t N, int64_t K, int32_t g, float eps,
                             const float* tau, uint8_t* codes, uint64_t* zero_count,
                             tm_stream stream);

/*
 * tm_group_code_dot — gradient of a per-group magnitude that multiplies the
 * codes:
 *   out[n, j] = sum_{i < g} q[n, j*g + i] * dW[n, j*g + i].
 * With What = alpha_g * q (decoupled quantization: the absmean only decides
 * the codes) this is d alpha_g.  For a learnable scale (Sec. 4) it is the
 * gradient through the magnitude; the hard forward rounding passes nothing
 * back through the threshold.  dW is the gradient with respect to the
 * dequantized weights, i.e. the output of tm_tgemm_bwd_dw_ste.
 *   codes  uint8 [N, K/4]   in   (16-byte aligned), packed as above
 *   dW     float32 [N, K]   in   (16-byte aligned)
 *   out    float32 [N, K/g] out  (4-byte aligned); sums taken in float64,
 *          rounded once
 */
tm_status tm_group_code_dot(const uint8_t* codes, const float* dW, int64_t N, int64_t K,
                            int32_t g, float* out, tm_stream stream);

/*
 * tm_scale_ste_grad — gradients of a learnable scale (Sec. 4: s_g an
 * nn.Parameter) and of the latent weights when only the rounding is
 * straight-through (Sec. 3.1's estimator applied to round, clip keeping its
 * derivative), i.e. what a layer computing s * ste(round(clip(w / (s + eps))))
 * receives:
 *   ds[n, j] = sum_{i < g} dWhat[n, i'] * (q[n, i'] - m[n, i'] * s * w / d^2),
 *   dW[n, k] = dWhat[n, k] * m[n, k] * s / d,         i' = j*g + i,
 * with d = fl32(s[n, k/g] + eps) and m = 1 where the float32 quotient
 * |W| / d is at most 1 (the clip's closed range), else 0.  Unlike
 * tm_group_code_dot (magnitude path only), the threshold term feeds back
 * into s, and the weights' gradient is clip-masked.
 *   W       float32 [N, K]    in   latent weights (16-byte aligned)
 *   codes   uint8 [N, K/4]    in   the codes of the forward call, i.e.
 *                                  tm_ternarize_codes against tau = s
 *   scale   float32 [N, K/g]  in   the learned s (4-byte aligned); each value
 *                                  finite and > 0 (not checked: device data)
 *   dWhat   float32 [N, K]    in   gradient w.r.t. the dequantized weights
 *                                  (tm_tgemm_bwd_dw_ste's output)
 *   eps     float32, finite, >= 0
 *   ds      float32 [N, K/g]  out  terms and sums in float64, rounded once
 *   dW      float32 [N, K]    out  or NULL (not written); may be dWhat
 *                                  itself (in place), no other overlap
 */
tm_status tm_scale_ste_grad(const float* W, const uint8_t* codes, const float* scale,
                            const float* dWhat, int64_t N, int64_t K, int32_t g, float eps,
                            float* ds, float* dW, tm_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* TMAMBA_H */
