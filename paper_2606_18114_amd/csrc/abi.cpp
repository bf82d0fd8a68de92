// C ABI of the ternary linear library: argument checks, then one launcher.
// Every check runs on the host before any HIP call, so a rejected call
// enqueues nothing (and can be exercised on a machine without a GPU).
#include <cmath>
#include <cstdint>

#include "../../include/tmamba.h"
#include "launchers.hpp"

namespace {

struct Span {
  uintptr_t lo = 0, hi = 0;  // [lo, hi)
};

bool bytes_of(int64_t a, int64_t b, int64_t elem, int64_t* out) {
  int64_t t;
  if (a < 0 || b < 0) return false;
  if (__builtin_mul_overflow(a, b, &t)) return false;
  if (__builtin_mul_overflow(t, elem, &t)) return false;
  if (t > (int64_t(1) << 46)) return false;  // 64 TiB: far beyond any device
  *out = t;
  return true;
}

Span span(const void* p, int64_t bytes) {
  Span s;
  s.lo = reinterpret_cast<uintptr_t>(p);
  s.hi = s.lo + static_cast<uintptr_t>(bytes);
  return s;
}

bool overlap(Span a, Span b) {
  if (a.lo == 0 || b.lo == 0 || a.hi == a.lo || b.hi == b.lo) return false;
  return a.lo < b.hi && b.lo < a.hi;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool group_ok(int32_t g) { return g == 32 || g == 64 || g == 128 || g == 256 || g == 512; }

tm_status shape_kg(int64_t K, int32_t g) {
  if (!group_ok(g)) return TM_ESHAPE;
  if (K < 1 || K % g != 0 || K % 64 != 0) return TM_ESHAPE;
  return TM_OK;
}

tm_status hip_status(hipError_t e) { return e == hipSuccess ? TM_OK : TM_EHIP; }

hipStream_t to_hip(tm_stream s) { return reinterpret_cast<hipStream_t>(s); }

constexpr int64_t kMaxGridBlocks = (int64_t(1) << 31) - 1;

// Y holds es-byte elements: 4 (float32) or 2 (bfloat16 bits)
// workspace NULL: the calls without one (cut tiles add with atomics)
tm_status tgemm_fwd_checked(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int32_t g, void* Y, int es,
                            void* workspace, int64_t workspace_bytes, tm_stream stream) {
  if (!X || !codes || !scales || !Y) return TM_EINVAL;
  if (M < 1 || N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t xb, cb, sb, yb;
  if (!bytes_of(M, K, 2, &xb) || !bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K / g, 4, &sb) ||
      !bytes_of(M, N, es, &yb))
    return TM_ESHAPE;
  if (((M + 255) / 256) * ((N + 255) / 256) > kMaxGridBlocks) return TM_ESHAPE;
  if (K > (int64_t(1) << 22) || N > (int64_t(1) << 26)) return TM_ESHAPE;  // 32-bit tile offsets
  if (!aligned(X, 16) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(Y, 16))
    return TM_EALIGN;
  const Span y = span(Y, yb);
  if (overlap(y, span(X, xb)) || overlap(y, span(codes, cb)) || overlap(y, span(scales, sb)))
    return TM_EINVAL;
  if (workspace) {
    if (workspace_bytes < tm_tgemm_fwd_workspace()) return TM_ESHAPE;
    if (!aligned(workspace, 4)) return TM_EALIGN;
    const Span w = span(workspace, tm_tgemm_fwd_workspace());
    if (overlap(w, y) || overlap(w, span(X, xb)) || overlap(w, span(codes, cb)) ||
        overlap(w, span(scales, sb)))
      return TM_EINVAL;
  }
  return hip_status(tmk::launch_tgemm_fwd(X, codes, scales, M, N, K, g, Y, es == 2,
                                          static_cast<uint32_t*>(workspace), to_hip(stream)));
}

// argument checks of both dX calls; workspace NULL: the two-pass call,
// which takes none
tm_status bwd_dx_checked(const uint16_t* dY, const uint8_t* codes, const float* scales,
                         int64_t M, int64_t N, int64_t K, int32_t g, float* dX,
                         const void* workspace, int64_t workspace_bytes) {
  if (!dY || !codes || !scales || !dX) return TM_EINVAL;
  if (M < 1 || N < 1 || N % 8 != 0) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  if (N > (int64_t(1) << 22) || K > (int64_t(1) << 26)) return TM_ESHAPE;
  int64_t yb, cb, sb, xb;
  if (!bytes_of(M, N, 2, &yb) || !bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K / g, 4, &sb) ||
      !bytes_of(M, K, 4, &xb))
    return TM_ESHAPE;
  if (((M + 255) / 256) * ((K + 255) / 256) > kMaxGridBlocks) return TM_ESHAPE;
  if (!aligned(dY, 16) || !aligned(codes, 16) || !aligned(scales, 4) || !aligned(dX, 16))
    return TM_EALIGN;
  const Span o = span(dX, xb);
  if (overlap(o, span(dY, yb)) || overlap(o, span(codes, cb)) || overlap(o, span(scales, sb)))
    return TM_EINVAL;
  if (workspace) {
    const int64_t need = tmk::dx_f16_workspace_bytes(M, N);
    if (workspace_bytes < need) return TM_ESHAPE;
    if (!aligned(workspace, 256)) return TM_EALIGN;
    const Span w = span(workspace, need);
    if (overlap(w, o) || overlap(w, span(dY, yb)) || overlap(w, span(codes, cb)) ||
        overlap(w, span(scales, sb)))
      return TM_EINVAL;
  }
  return TM_OK;
}

// batches of 9 .. 16 rows at g >= 64 go to the bfloat16 matrix-core form
// (one workgroup per matrix and 16-row block)
bool tgemv_on_bf16_mfma(int32_t count, int32_t B, int64_t N, int32_t g) {
  return tmk::tgemv_b16_takes(B, g) && (int64_t)count * ((N + 15) / 16) <= 0x7FFFFFFF;
}

// argument checks of one strided stack of tm_tgemv; out / ins: the spans of
// y and of x, codes, scales
tm_status tgemv_checked(const uint16_t* x, const uint8_t* codes, const uint16_t* scales_f16,
                        int32_t count, int32_t B, int64_t N, int64_t K, int32_t g, float* y,
                        Span* out, Span* ins) {
  if (!x || !codes || !scales_f16 || !y) return TM_EINVAL;
  if (count < 1 || count > 65535 || B < 1 || B > 16 || N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t cbm, sbm, xb, cb, sb, yb, ybm;
  if (!bytes_of(N, K / 4, 1, &cbm) || !bytes_of(N, K / g, 2, &sbm) ||
      !bytes_of((int64_t)count * B, K, 2, &xb) || !bytes_of(count, cbm, 1, &cb) ||
      !bytes_of(count, sbm, 1, &sb) || !bytes_of((int64_t)B, N, 4, &ybm) ||
      !bytes_of(count, ybm, 1, &yb))
    return TM_ESHAPE;
  if ((N + 63) / 64 > kMaxGridBlocks) return TM_ESHAPE;
  if (cbm > (int64_t(1) << 31)) return TM_ESHAPE;  // 32-bit offsets inside one matrix
  if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(scales_f16, 2) || !aligned(y, 16))
    return TM_EALIGN;
  *out = span(y, yb);
  ins[0] = span(x, xb);
  ins[1] = span(codes, cb);
  ins[2] = span(scales_f16, sb);
  if (overlap(*out, ins[0]) || overlap(*out, ins[1]) || overlap(*out, ins[2])) return TM_EINVAL;
  return TM_OK;
}

// argument checks of the mixer step; workspace NULL: the library's own
// scratch array (no overlap check needed: no caller array can overlap it)
// gate_only: the gated float32 output of tm_mixer_gate in place of the
// normalized bfloat16 one (no norm_w, eps or workspace)
tm_status mixer_checked(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                        int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                        uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                        const float* dt_bias, const float* A_log, const float* D,
                        const float* norm_w, float eps, float* workspace, const void* out,
                        bool gate_only = false) {
  if (!zxbcdt || !conv_state || !conv_pos || !ssm_state || !conv_w || !conv_b || !dt_bias ||
      !A_log || !D || (!gate_only && !norm_w) || !out)
    return TM_EINVAL;
  if (!gate_only && (!(eps >= 0.0f) || !std::isfinite(eps))) return TM_EINVAL;
  if (B < 1 || B > 65535 || nheads < 1 || nheads > 4096 || headdim != 64 || d_state != 128)
    return TM_ESHAPE;
  const int64_t di = (int64_t)nheads * headdim, cd = di + 2 * (int64_t)d_state;
  const int64_t zw = 2 * di + 2 * (int64_t)d_state + nheads;
  int64_t zb, cb, sb, wb, ob;
  if (!bytes_of(B, zw, 4, &zb) || !bytes_of((int64_t)B * cd, 4, 2, &cb) ||
      !bytes_of((int64_t)B * nheads * headdim, d_state, 2, &sb) ||
      !bytes_of(B, di + nheads, 4, &wb) || !bytes_of(B, di, gate_only ? 4 : 2, &ob))
    return TM_ESHAPE;
  if (!aligned(zxbcdt, 4) || !aligned(conv_state, 8) || !aligned(conv_pos, 4) ||
      !aligned(ssm_state, 16) || !aligned(conv_w, 4) || !aligned(conv_b, 4) ||
      !aligned(dt_bias, 4) || !aligned(A_log, 4) || !aligned(D, 4) || !aligned(norm_w, 4) ||
      !aligned(workspace, 4) || !aligned(out, gate_only ? 4 : 2))
    return TM_EALIGN;
  const Span outs[5] = {span(conv_state, cb), span(conv_pos, 4), span(ssm_state, sb),
                        span(workspace, workspace ? wb : 0), span(out, ob)};
  const Span ins[7] = {span(zxbcdt, zb), span(conv_w, cd * 16), span(conv_b, cd * 4),
                       span(dt_bias, (int64_t)nheads * 4), span(A_log, (int64_t)nheads * 4),
                       span(D, (int64_t)nheads * 4), span(norm_w, norm_w ? di * 4 : 0)};
  for (int i = 0; i < 5; ++i) {
    for (int j = i + 1; j < 5; ++j)
      if (overlap(outs[i], outs[j])) return TM_EINVAL;
    for (const Span& in : ins)
      if (overlap(outs[i], in)) return TM_EINVAL;
  }
  return TM_OK;
}

}  // namespace

extern "C" {

int tm_abi_version(void) { return TM_ABI_VERSION; }

const char* tm_status_str(tm_status s) {
  switch (s) {
    case TM_OK: return "TM_OK";
    case TM_EINVAL: return "TM_EINVAL: null pointer, overlapping arrays or bad scalar argument";
    case TM_ESHAPE: return "TM_ESHAPE: unsupported sizes (size < 1, K % g, K % 64, g, B or count)";
    case TM_EALIGN: return "TM_EALIGN: pointer below its required alignment";
    case TM_EHIP: return "TM_EHIP: the HIP runtime rejected a launch";
    case TM_ENOTIMPL: return "TM_ENOTIMPL: not implemented";
  }
  return "unknown tm_status";
}

tm_status tm_ternarize_pack(const float* W, int64_t N, int64_t K, int32_t g, float eps,
                            uint8_t* codes, float* scales, uint16_t* scales_f16,
                            uint64_t* zero_count, tm_stream stream) {
  return tm_ternarize_pack_thresh(W, N, K, g, eps, nullptr, codes, scales, scales_f16,
                                  zero_count, stream);
}

tm_status tm_ternarize_pack_thresh(const float* W, int64_t N, int64_t K, int32_t g, float eps,
                                   const float* row_mult, uint8_t* codes, float* scales,
                                   uint16_t* scales_f16, uint64_t* zero_count,
                                   tm_stream stream) {
  if (!W || !codes || !scales) return TM_EINVAL;
  if (!std::isfinite(eps) || eps < 0.f) return TM_EINVAL;
  if (N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t wb, cb, sb, hb;
  if (!bytes_of(N, K, 4, &wb) || !bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K / g, 4, &sb) ||
      !bytes_of(N, K / g, 2, &hb))
    return TM_ESHAPE;
  if ((N * (K / 16) + 255) / 256 > kMaxGridBlocks) return TM_ESHAPE;
  if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scales, 4) ||
      !aligned(scales_f16, 2) || !aligned(zero_count, 8) || !aligned(row_mult, 4))
    return TM_EALIGN;
  const Span in = span(W, wb), c = span(codes, cb), s = span(scales, sb),
             h = span(scales_f16, scales_f16 ? hb : 0), z = span(zero_count, zero_count ? 8 : 0),
             m = span(row_mult, row_mult ? N * 4 : 0);
  const Span outs[4] = {c, s, h, z};
  for (int i = 0; i < 4; ++i) {
    if (overlap(in, outs[i]) || overlap(m, outs[i])) return TM_EINVAL;
    for (int j = i + 1; j < 4; ++j)
      if (overlap(outs[i], outs[j])) return TM_EINVAL;
  }
  return hip_status(tmk::launch_ternarize_pack(W, N, K, g, eps, row_mult, nullptr, codes,
                                              scales, scales_f16, zero_count, to_hip(stream)));
}

tm_status tm_ternarize_codes(const float* W, int64_t N, int64_t K, int32_t g, float eps,
                             const float* tau, uint8_t* codes, uint64_t* zero_count,
                             tm_stream stream) {
  if (!W || !tau || !codes) return TM_EINVAL;
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return TM_EINVAL;
  if (N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t wb, cb, tb;
  if (!bytes_of(N, K, 4, &wb) || !bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K / g, 4, &tb))
    return TM_ESHAPE;
  if ((N * (K / 16) + 255) / 256 > kMaxGridBlocks) return TM_ESHAPE;
  if (!aligned(W, 16) || !aligned(tau, 4) || !aligned(codes, 16) || !aligned(zero_count, 8))
    return TM_EALIGN;
  const Span c = span(codes, cb), z = span(zero_count, zero_count ? 8 : 0);
  const Span ins[2] = {span(W, wb), span(tau, tb)};
  for (const Span& in : ins)
    if (overlap(in, c) || overlap(in, z)) return TM_EINVAL;
  if (overlap(c, z)) return TM_EINVAL;
  return hip_status(tmk::launch_ternarize_pack(W, N, K, g, eps, nullptr, tau, codes, nullptr,
                                              nullptr, zero_count, to_hip(stream)));
}

tm_status tm_group_code_dot(const uint8_t* codes, const float* dW, int64_t N, int64_t K,
                            int32_t g, float* out, tm_stream stream) {
  if (!codes || !dW || !out) return TM_EINVAL;
  if (N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t cb, wb, ob;
  if (!bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K, 4, &wb) || !bytes_of(N, K / g, 4, &ob))
    return TM_ESHAPE;
  if (!aligned(codes, 16) || !aligned(dW, 16) || !aligned(out, 4)) return TM_EALIGN;
  const Span o = span(out, ob);
  if (overlap(o, span(codes, cb)) || overlap(o, span(dW, wb))) return TM_EINVAL;
  return hip_status(tmk::launch_group_code_dot(codes, dW, N, K, g, out, to_hip(stream)));
}


tm_status tm_scale_ste_grad(const float* W, const uint8_t* codes, const float* scale,
                            const float* dWhat, int64_t N, int64_t K, int32_t g, float eps,
                            float* ds, float* dW, tm_stream stream) {
  if (!W || !codes || !scale || !dWhat || !ds) return TM_EINVAL;
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return TM_EINVAL;
  if (N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  int64_t wb, cb, sb;
  if (!bytes_of(N, K, 4, &wb) || !bytes_of(N, K / 4, 1, &cb) || !bytes_of(N, K / g, 4, &sb))
    return TM_ESHAPE;
  if (!aligned(W, 16) || !aligned(codes, 16) || !aligned(scale, 4) || !aligned(dWhat, 16) ||
      !aligned(ds, 4) || !aligned(dW, 16))
    return TM_EALIGN;
  const Span o = span(ds, sb), w = span(dW, dW ? wb : 0), g_in = span(dWhat, wb);
  const Span ins[3] = {span(W, wb), span(codes, cb), span(scale, sb)};
  for (const Span& in : ins)
    if (overlap(in, o) || overlap(in, w)) return TM_EINVAL;
  if (overlap(o, g_in) || overlap(o, w)) return TM_EINVAL;
  // dW may be dWhat itself (in place), but no other overlap of the two
  if (dW && static_cast<const void*>(dW) != static_cast<const void*>(dWhat) && overlap(w, g_in))
    return TM_EINVAL;
  return hip_status(tmk::launch_scale_ste_grad(W, codes, scale, dWhat, N, K, g, eps, ds, dW,
                                               to_hip(stream)));
}

tm_status tm_tgemm_fwd(const uint16_t* X, const uint8_t* codes, const float* scales, int64_t M,
                       int64_t N, int64_t K, int32_t g, float* Y, tm_stream stream) {
  return tgemm_fwd_checked(X, codes, scales, M, N, K, g, Y, 4, nullptr, 0, stream);
}

int64_t tm_tgemm_fwd_workspace(void) { return 8 * (int64_t)tmk::kFwdMaxTicketTiles; }

tm_status tm_tgemm_fwd_ws(const uint16_t* X, const uint8_t* codes, const float* scales,
                          int64_t M, int64_t N, int64_t K, int32_t g, float* Y, void* workspace,
                          int64_t workspace_bytes, tm_stream stream) {
  if (!workspace) return TM_EINVAL;
  return tgemm_fwd_checked(X, codes, scales, M, N, K, g, Y, 4, workspace, workspace_bytes,
                           stream);
}

tm_status tm_tgemm_fwd_bf16(const uint16_t* X, const uint8_t* codes, const float* scales,
                            int64_t M, int64_t N, int64_t K, int32_t g, uint16_t* Y,
                            tm_stream stream) {
  return tgemm_fwd_checked(X, codes, scales, M, N, K, g, Y, 2, nullptr, 0, stream);
}

tm_status tm_tgemm_bwd_dx(const uint16_t* dY, const uint8_t* codes, const float* scales,
                          int64_t M, int64_t N, int64_t K, int32_t g, float* dX,
                          tm_stream stream) {
  if (tm_status st = bwd_dx_checked(dY, codes, scales, M, N, K, g, dX, nullptr, 0)) return st;
  return hip_status(tmk::launch_tgemm_bwd_dx(dY, codes, scales, M, N, K, g, dX, to_hip(stream)));
}

int64_t tm_tgemm_bwd_dx_f16_workspace(int64_t M, int64_t N) {
  int64_t yb;
  if (M < 1 || N < 1 || !bytes_of(M, N, 2, &yb)) return -1;
  return tmk::dx_f16_workspace_bytes(M, N);
}

tm_status tm_tgemm_bwd_dx_f16(const uint16_t* dY, const uint8_t* codes, const float* scales,
                              int64_t M, int64_t N, int64_t K, int32_t g, float* dX,
                              void* workspace, int64_t workspace_bytes, tm_stream stream) {
  if (!workspace) return TM_EINVAL;
  if (tm_status st = bwd_dx_checked(dY, codes, scales, M, N, K, g, dX, workspace,
                                    workspace_bytes))
    return st;
  return hip_status(tmk::launch_tgemm_bwd_dx_f16(dY, codes, scales, M, N, K, g, dX, workspace,
                                                 to_hip(stream)));
}

tm_status tm_tgemm_bwd_dw_ste(const uint16_t* dY, const uint16_t* X, int64_t M, int64_t N,
                              int64_t K, float* dW, int32_t accumulate, tm_stream stream) {
  if (!dY || !X || !dW) return TM_EINVAL;
  if (accumulate != 0 && accumulate != 1) return TM_EINVAL;
  if (M < 1 || N < 1 || N % 8 != 0 || K < 1 || K % 64 != 0) return TM_ESHAPE;
  int64_t yb, xb, wb;
  if (!bytes_of(M, N, 2, &yb) || !bytes_of(M, K, 2, &xb) || !bytes_of(N, K, 4, &wb))
    return TM_ESHAPE;
  if (((N + 255) / 256) * ((K + 255) / 256) * ((M + 255) / 256) > kMaxGridBlocks) return TM_ESHAPE;
  if (N > (int64_t(1) << 26) || K > (int64_t(1) << 26)) return TM_ESHAPE;  // 32-bit row offsets
  if (!aligned(dY, 16) || !aligned(X, 16) || !aligned(dW, 16)) return TM_EALIGN;
  const Span o = span(dW, wb);
  if (overlap(o, span(dY, yb)) || overlap(o, span(X, xb))) return TM_EINVAL;
  return hip_status(tmk::launch_tgemm_bwd_dw(dY, X, M, N, K, dW, accumulate, to_hip(stream)));
}

tm_status tm_dgemv(const uint16_t* x, const uint16_t* W16, int32_t count, int32_t B, int64_t N,
                   int64_t K, float* y, tm_stream stream) {
  if (!x || !W16 || !y) return TM_EINVAL;
  if (count < 1 || count > 65535 || B < 1 || B > 8 || N < 1) return TM_ESHAPE;
  if (K < 64 || K % 64 != 0 || (int64_t)B * K > 16384) return TM_ESHAPE;
  int64_t xb, wb, yb;
  if (!bytes_of((int64_t)count * B, K, 2, &xb) || !bytes_of((int64_t)count * N, K, 2, &wb) ||
      !bytes_of((int64_t)count * B, N, 4, &yb))
    return TM_ESHAPE;
  if ((N + 7) / 8 > kMaxGridBlocks) return TM_ESHAPE;
  if (!aligned(x, 16) || !aligned(W16, 16) || !aligned(y, 4)) return TM_EALIGN;
  const Span o = span(y, yb);
  if (overlap(o, span(x, xb)) || overlap(o, span(W16, wb))) return TM_EINVAL;
  return hip_status(tmk::launch_dgemv(x, W16, count, B, N, K, y, to_hip(stream)));
}

tm_status tm_residual_rmsnorm(float* residual, const float* y, int32_t B, int64_t D,
                              const float* w, float eps, uint16_t* x, tm_stream stream) {
  if (!residual || !w || !x) return TM_EINVAL;
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return TM_EINVAL;
  if (B < 1 || B > 65535 || D < 1) return TM_ESHAPE;
  int64_t rb, xb, wb;
  if (!bytes_of(B, D, 4, &rb) || !bytes_of(B, D, 2, &xb) || !bytes_of(1, D, 4, &wb))
    return TM_ESHAPE;
  if (!aligned(residual, 4) || !aligned(y, 4) || !aligned(w, 4) || !aligned(x, 2))
    return TM_EALIGN;
  const Span r = span(residual, rb), o = span(x, xb), yy = span(y, y ? rb : 0), ww = span(w, wb);
  if (overlap(r, o) || overlap(r, yy) || overlap(r, ww) || overlap(o, yy) || overlap(o, ww))
    return TM_EINVAL;
  return hip_status(tmk::launch_residual_rmsnorm(residual, y, B, D, w, eps, x, to_hip(stream)));
}

tm_status tm_mixer_step(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                        int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                        uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                        const float* dt_bias, const float* A_log, const float* D,
                        const float* norm_w, float eps, float* workspace, uint16_t* out,
                        tm_stream stream) {
  if (!workspace) return TM_EINVAL;
  if (tm_status st = mixer_checked(zxbcdt, B, nheads, headdim, d_state, conv_state, conv_pos,
                                   ssm_state, conv_w, conv_b, dt_bias, A_log, D, norm_w, eps,
                                   workspace, out))
    return st;
  return hip_status(tmk::launch_mixer_step(zxbcdt, B, nheads, conv_state, conv_pos, ssm_state,
                                           conv_w, conv_b, dt_bias, A_log, D, norm_w, eps,
                                           workspace, out, to_hip(stream)));
}

tm_status tm_mixer_step_noalloc(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                                int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                                uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                                const float* dt_bias, const float* A_log, const float* D,
                                const float* norm_w, float eps, uint16_t* out,
                                tm_stream stream) {
  if (tm_status st = mixer_checked(zxbcdt, B, nheads, headdim, d_state, conv_state, conv_pos,
                                   ssm_state, conv_w, conv_b, dt_bias, A_log, D, norm_w, eps,
                                   nullptr, out))
    return st;
  if ((int64_t)B * ((int64_t)nheads * headdim + nheads) > tmk::mixer_scratch_floats())
    return TM_ESHAPE;
  return hip_status(tmk::launch_mixer_step_noalloc(zxbcdt, B, nheads, conv_state, conv_pos,
                                                   ssm_state, conv_w, conv_b, dt_bias, A_log, D,
                                                   norm_w, eps, out, to_hip(stream)));
}

tm_status tm_tgemv(const uint16_t* x, const uint8_t* codes, const uint16_t* scales_f16,
                   int32_t count, int32_t B, int64_t N, int64_t K, int32_t g, float* y,
                   tm_stream stream) {
  Span out, ins[3];
  if (tm_status st = tgemv_checked(x, codes, scales_f16, count, B, N, K, g, y, &out, ins))
    return st;
  if (tgemv_on_bf16_mfma(count, B, N, g))
    return hip_status(
        tmk::launch_tgemv_b16(x, codes, scales_f16, count, B, N, K, g, y, to_hip(stream)));
  return hip_status(tmk::launch_tgemv(x, codes, scales_f16, count, B, N, K, g, y, to_hip(stream)));
}

tm_status tm_tgemv_pair(const uint16_t* x0, const uint8_t* codes0, const uint16_t* scales0,
                        int32_t count0, int64_t N0, int64_t K0, float* y0, const uint16_t* x1,
                        const uint8_t* codes1, const uint16_t* scales1, int32_t count1,
                        int64_t N1, int64_t K1, float* y1, int32_t B, int32_t g,
                        tm_stream stream) {
  Span o0, o1, i0[3], i1[3];
  if (tm_status st = tgemv_checked(x0, codes0, scales0, count0, B, N0, K0, g, y0, &o0, i0))
    return st;
  if (tm_status st = tgemv_checked(x1, codes1, scales1, count1, B, N1, K1, g, y1, &o1, i1))
    return st;
  if (overlap(o0, o1)) return TM_EINVAL;
  for (int i = 0; i < 3; ++i)
    if (overlap(o0, i1[i]) || overlap(o1, i0[i])) return TM_EINVAL;
  if (tgemv_on_bf16_mfma(count0, B, N0, g) && tgemv_on_bf16_mfma(count1, B, N1, g)) {
    const hipError_t e = tmk::launch_tgemv_b16(x0, codes0, scales0, count0, B, N0, K0, g, y0,
                                               to_hip(stream));
    if (e != hipSuccess) return hip_status(e);
    return hip_status(tmk::launch_tgemv_b16(x1, codes1, scales1, count1, B, N1, K1, g, y1,
                                            to_hip(stream)));
  }
  return hip_status(tmk::launch_tgemv_pair(x0, codes0, scales0, count0, N0, K0, y0, x1, codes1,
                                           scales1, count1, N1, K1, y1, B, g, to_hip(stream)));
}

tm_status tm_tgemv_rms(const float* src, const float* norm_w, float eps, const uint8_t* codes,
                       const uint16_t* scales_f16, int32_t B, int64_t N, int64_t K, int32_t g,
                       float* y, int32_t accumulate, tm_stream stream) {
  if (!src || !norm_w || !codes || !scales_f16 || !y) return TM_EINVAL;
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return TM_EINVAL;
  if (accumulate != 0 && accumulate != 1) return TM_EINVAL;
  if (B < 1 || B > 16 || N < 1) return TM_ESHAPE;
  if (tm_status st = shape_kg(K, g)) return st;
  if (!tmk::tgemv_rms_fits(B, K, g)) return TM_ESHAPE;
  int64_t xb, wb, cb, sb, yb;
  if (!bytes_of(B, K, 4, &xb) || !bytes_of(1, K, 4, &wb) || !bytes_of(N, K / 4, 1, &cb) ||
      !bytes_of(N, K / g, 2, &sb) || !bytes_of(B, N, 4, &yb))
    return TM_ESHAPE;
  if ((N + 31) / 32 > kMaxGridBlocks) return TM_ESHAPE;
  if (cb > (int64_t(1) << 31)) return TM_ESHAPE;  // 32-bit offsets inside the matrix
  if (!aligned(src, 16) || !aligned(norm_w, 16) || !aligned(codes, 16) ||
      !aligned(scales_f16, 2) || !aligned(y, 16))
    return TM_EALIGN;
  const Span o = span(y, yb);
  if (overlap(o, span(src, xb)) || overlap(o, span(norm_w, wb)) || overlap(o, span(codes, cb)) ||
      overlap(o, span(scales_f16, sb)))
    return TM_EINVAL;
  return hip_status(tmk::launch_tgemv_rms(src, norm_w, eps, codes, scales_f16, B, N, K, g, y,
                                          accumulate, to_hip(stream)));
}

tm_status tm_dgemv_rms(const float* src, const float* norm_w, float eps, const uint16_t* W16,
                       int32_t B, int64_t N, int64_t K, float* y, int32_t accumulate,
                       tm_stream stream) {
  if (!src || !norm_w || !W16 || !y) return TM_EINVAL;
  if (!(eps >= 0.0f) || !std::isfinite(eps)) return TM_EINVAL;
  if (accumulate != 0 && accumulate != 1) return TM_EINVAL;
  if (B < 1 || B > 8 || N < 1) return TM_ESHAPE;
  if (K < 64 || K % 64 != 0 || (int64_t)B * K > 16384) return TM_ESHAPE;
  int64_t xb, wb, mb, yb;
  if (!bytes_of(B, K, 4, &xb) || !bytes_of(1, K, 4, &wb) || !bytes_of(N, K, 2, &mb) ||
      !bytes_of(B, N, 4, &yb))
    return TM_ESHAPE;
  if ((N + 7) / 8 > kMaxGridBlocks) return TM_ESHAPE;
  if (!aligned(src, 16) || !aligned(norm_w, 16) || !aligned(W16, 16) || !aligned(y, 4))
    return TM_EALIGN;
  const Span o = span(y, yb);
  if (overlap(o, span(src, xb)) || overlap(o, span(norm_w, wb)) || overlap(o, span(W16, mb)))
    return TM_EINVAL;
  return hip_status(
      tmk::launch_dgemv_rms(src, norm_w, eps, W16, B, N, K, y, accumulate, to_hip(stream)));
}

tm_status tm_mixer_gate(const float* zxbcdt, int32_t B, int32_t nheads, int32_t headdim,
                        int32_t d_state, uint16_t* conv_state, int32_t* conv_pos,
                        uint16_t* ssm_state, const float* conv_w, const float* conv_b,
                        const float* dt_bias, const float* A_log, const float* D, float* gated,
                        tm_stream stream) {
  if (tm_status st = mixer_checked(zxbcdt, B, nheads, headdim, d_state, conv_state, conv_pos,
                                   ssm_state, conv_w, conv_b, dt_bias, A_log, D, nullptr, 0.f,
                                   nullptr, gated, true))
    return st;
  if ((int64_t)B * nheads >= (int64_t(1) << 29)) return TM_ESHAPE;  // the arrival count fits
  return hip_status(tmk::launch_mixer_gate(zxbcdt, B, nheads, conv_state, conv_pos, ssm_state,
                                           conv_w, conv_b, dt_bias, A_log, D, gated,
                                           to_hip(stream)));
}

int64_t tm_mamba2_decode_workspace(int32_t d_model, int32_t nheads, int32_t batch) {
  if (d_model < 1 || d_model > 4096 || nheads < 1 || nheads > 128 || batch < 1 ||
      batch > tmk::kDecodeStackMaxBatch)
    return -1;
  return tmk::decode_stack_workspace_bytes(d_model, nheads, batch);
}

tm_status tm_mamba2_decode_token(const tm_mamba2_stack* st, const float* emb, uint16_t* x_out,
                                 void* workspace, int64_t workspace_bytes, tm_stream stream) {
  if (!st || !emb || !x_out || !workspace) return TM_EINVAL;
  const tm_mamba2_stack& s = *st;
  if (!s.in_codes || !s.in_scales || !s.out_codes || !s.out_scales || !s.pre_w || !s.conv_w ||
      !s.conv_b || !s.dt_bias || !s.A_log || !s.D || !s.norm_w || !s.final_w ||
      !s.conv_state || !s.conv_pos || !s.ssm_state)
    return TM_EINVAL;
  if (!(s.eps >= 0.0f) || !std::isfinite(s.eps)) return TM_EINVAL;
  if (s.g != 64 && s.g != 128 && s.g != 256) return TM_ESHAPE;
  if (s.n_layers < 1 || s.n_layers > 65535 || s.nheads < 1 || s.nheads > 128) return TM_ESHAPE;
  const int64_t L = s.n_layers, Dm = s.d_model, H = s.nheads, DI = 64 * H, B = s.batch;
  if (Dm < 64 || Dm > 4096 || Dm % 64 != 0 || Dm % s.g != 0 || DI % s.g != 0) return TM_ESHAPE;
  if (B < 1 || B > tmk::kDecodeStackMaxBatch || (B > 1 && (Dm > 2048 || DI > 4096)))
    return TM_ESHAPE;
  // one workgroup per head and batch row
  if (H * B > tmk::current_cu_count()) return TM_ESHAPE;
  const int64_t Z = 2 * DI + 256 + H, CD = DI + 256;
  int64_t icb, isb, ocb, osb, csb, ssb;
  if (!bytes_of(L * Z, Dm / 4, 1, &icb) || !bytes_of(L * Z, Dm / s.g, 2, &isb) ||
      !bytes_of(L * Dm, DI / 4, 1, &ocb) || !bytes_of(L * Dm, DI / s.g, 2, &osb) ||
      !bytes_of(L * B * CD, 4, 2, &csb) || !bytes_of(L * B * H * 64, 128, 2, &ssb))
    return TM_ESHAPE;
  if (Z * (Dm / 4) > (int64_t(1) << 31) || Dm * (DI / 4) > (int64_t(1) << 31))
    return TM_ESHAPE;  // 32-bit offsets inside one matrix
  const int64_t need = tmk::decode_stack_workspace_bytes((int)Dm, (int)H, (int)B);
  if (workspace_bytes < need) return TM_ESHAPE;
  if (!aligned(s.in_codes, 16) || !aligned(s.out_codes, 16) || !aligned(s.in_scales, 2) ||
      !aligned(s.out_scales, 2) || !aligned(s.pre_w, 16) || !aligned(s.conv_w, 4) ||
      !aligned(s.conv_b, 4) || !aligned(s.dt_bias, 4) || !aligned(s.A_log, 4) ||
      !aligned(s.D, 4) || !aligned(s.norm_w, 16) || !aligned(s.final_w, 16) ||
      !aligned(s.conv_state, 8) || !aligned(s.conv_pos, 4) || !aligned(s.ssm_state, 16) ||
      !aligned(emb, 16) || !aligned(x_out, 4) || !aligned(workspace, 256))
    return TM_EALIGN;
  // blocks kept in FP16
  if (s.n_kept < 0 || s.n_kept > tmk::kDecodeStackMaxKept) return TM_ESHAPE;
  int64_t iwb = 0, owb = 0;
  if (s.n_kept > 0) {
    if (!s.kept || !s.in_w16 || !s.out_w16) return TM_EINVAL;
    for (int i = 0; i < s.n_kept; ++i)
      if (s.kept[i] < 0 || s.kept[i] >= L || (i > 0 && s.kept[i] <= s.kept[i - 1]))
        return TM_ESHAPE;
    if (!bytes_of((int64_t)s.n_kept * Z, Dm, 2, &iwb) ||
        !bytes_of((int64_t)s.n_kept * Dm, DI, 2, &owb))
      return TM_ESHAPE;
    if (!aligned(s.in_w16, 16) || !aligned(s.out_w16, 16)) return TM_EALIGN;
  }
  const Span outs[5] = {span(s.conv_state, csb), span(s.conv_pos, L * 4), span(s.ssm_state, ssb),
                        span(x_out, B * Dm * 2), span(workspace, need)};
  const Span ins[13] = {span(s.in_codes, icb), span(s.in_scales, isb), span(s.out_codes, ocb),
                        span(s.out_scales, osb), span(s.pre_w, L * Dm * 4),
                        span(s.conv_w, L * CD * 16), span(s.conv_b, L * CD * 4),
                        span(s.dt_bias, L * H * 4), span(s.A_log, L * H * 4),
                        span(s.D, L * H * 4), span(s.norm_w, L * DI * 4),
                        span(s.final_w, Dm * 4), span(emb, B * Dm * 4)};
  for (int i = 0; i < 5; ++i) {
    for (int j = i + 1; j < 5; ++j)
      if (overlap(outs[i], outs[j])) return TM_EINVAL;
    for (const Span& in : ins)
      if (overlap(outs[i], in)) return TM_EINVAL;
    if (s.n_kept > 0 && (overlap(outs[i], span(s.in_w16, iwb)) ||
                         overlap(outs[i], span(s.out_w16, owb))))
      return TM_EINVAL;
  }
  tmk::DecodeStackDesc d;
  d.n_layers = s.n_layers;
  d.d_model = s.d_model;
  d.nheads = s.nheads;
  d.g = s.g;
  d.batch = s.batch;
  d.eps = s.eps;
  d.in_codes = s.in_codes;
  d.in_s16 = s.in_scales;
  d.out_codes = s.out_codes;
  d.out_s16 = s.out_scales;
  d.pre_w = s.pre_w;
  d.conv_w = s.conv_w;
  d.conv_b = s.conv_b;
  d.dt_bias = s.dt_bias;
  d.A_log = s.A_log;
  d.D = s.D;
  d.norm_w = s.norm_w;
  d.final_w = s.final_w;
  d.conv_state = s.conv_state;
  d.conv_pos = s.conv_pos;
  d.ssm_state = s.ssm_state;
  d.n_kept = s.n_kept;
  for (int i = 0; i < tmk::kDecodeStackMaxKept; ++i) d.kept[i] = i < s.n_kept ? s.kept[i] : -1;
  d.in_w16 = s.n_kept > 0 ? s.in_w16 : nullptr;
  d.out_w16 = s.n_kept > 0 ? s.out_w16 : nullptr;
  return hip_status(tmk::launch_decode_stack(d, emb, x_out, workspace, to_hip(stream)));
}

}  // extern "C"
