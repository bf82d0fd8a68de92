"""CPU oracle for the grouped-absmean ternary (W1.58A16) linear layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports or calls this
module: only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may.  It shares no code with the HIP kernels.

What it computes, and where the paper defines it
-------------------------------------------------
Paper: "Ternary Mamba: Grouped Quantization-Aware Training of W1.58A16 State
Space Models", Sec. 3.1 (TernaryLinear Module).

* The weight matrix W [N, K] (out x in) is cut into groups of ``g`` consecutive
  input-dimension elements of one output row.
* Group scale: the mean absolute value of the group, recomputed on every call
  and never learned (Sec. 3.1, second paragraph; Sec. 4 explains why).
* Code: the weight divided by its group scale, clipped to [-1, 1] and rounded,
  giving a value in {-1, 0, +1}.
* Dequantized weight: scale times code.  Forward: Y = X * What^T.
* Backward: gradients pass the quantizer unchanged (straight-through
  estimator, Sec. 3.1; hard quantization in the forward pass, App. A.3), so
  dX = dY * What and dW = dY^T * X.
* Zero ratio: the fraction of zero codes (Sec. 3.1 and Table 1).
* Deployment storage: 2-bit codes plus per-group scales (Sec. 8, Table 11).
* Weight NRMSE: per-layer weight quantization error (Sec. 7, App. A.7).

Readings taken where the paper is silent:

* groups run along the input dimension K, contiguous, K % g == 0;
* a non-negative ``eps`` is added to the scale before the division (eps = 0 is
  the paper's literal formula); dequantization multiplies by the scale itself;
* "round" is round-half-to-even (PyTorch semantics);
* the division, clip and round are taken in float32, the precision the kernel
  works in, on the float32-rounded scale; the mean itself is taken in float64;
* the straight-through estimator is the identity (no clip mask, no gradient
  through the scale);
* 2-bit storage format, see ``pack`` below.

Every floating-point reference product (GEMM, GEMV) is computed in float64.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_bits_to_f64",
    "group_scales_f64",
    "group_scales_f32",
    "scales_f16",
    "ternary_codes",
    "boundary_mask",
    "zero_count",
    "pack",
    "unpack",
    "dequantize",
    "gemm_fwd",
    "gemm_bwd_dx",
    "gemm_bwd_dw",
    "gemv",
    "dense_gemv",
    "nrmse",
    "rel_fro_error",
    "ternarize",
]


def _check_finite(W: np.ndarray) -> None:
    if not np.all(np.isfinite(W)):
        raise ValueError("oracle: NaN or Inf in W is outside the method's domain")


def _groups(W: np.ndarray, g: int) -> np.ndarray:
    """View W [N, K] as [N, K/g, g]: contiguous groups along the input dim."""
    N, K = W.shape
    if g <= 0 or K % g:
        raise ValueError(f"oracle: K={K} is not a multiple of the group size g={g}")
    return W.reshape(N, K // g, g)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact float64 values."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Quantizer (Sec. 3.1)
# --------------------------------------------------------------------------

def group_scales_f64(W: np.ndarray, g: int) -> np.ndarray:
    """s[n, j] = (1/g) * sum_i |W[n, j*g + i]|, accumulated in float64.

    Sec. 3.1: the per-group scale is the mean absolute weight of its group.
    numpy's float64 sum of at most 512 float32 magnitudes is exact to far
    below float32 resolution.
    """
    W = np.asarray(W, dtype=np.float32)
    _check_finite(W)
    Wg = _groups(W, g).astype(np.float64)
    return np.abs(Wg).sum(axis=2) / g


def group_scales_f32(W: np.ndarray, g: int) -> np.ndarray:
    """The float32 rounding of the float64 group mean (the stored scale)."""
    return group_scales_f64(W, g).astype(np.float32)


def scales_f16(s32: np.ndarray) -> np.ndarray:
    """Deployment scales: float16 round-to-nearest-even of the float32 scale."""
    return np.asarray(s32, dtype=np.float32).astype(np.float16)


def ternary_codes(W: np.ndarray, s32: np.ndarray, g: int, eps: float) -> np.ndarray:
    """q = round(clip(W / (s + eps), -1, 1)) in {-1, 0, +1}, as int8.

    Sec. 3.1 gives round(clip(w / s_g, -1, 1)).  The division, the clip and
    the half-to-even round are taken in float32 on the float32 scale, as a
    float32 PyTorch module would compute them.
    """
    W = np.asarray(W, dtype=np.float32)
    _check_finite(W)
    if not (np.isfinite(eps) and eps >= 0.0):
        raise ValueError("oracle: eps must be finite and >= 0")
    N, K = W.shape
    s32 = np.asarray(s32, dtype=np.float32).reshape(N, K // g)
    d = (s32 + np.float32(eps)).astype(np.float32)            # float32 add
    Wg = _groups(W, g)
    with np.errstate(divide="ignore", invalid="ignore"):
        x = (Wg / d[:, :, None]).astype(np.float32)            # float32 divide
    # 0/0 (an all-zero group at eps = 0): the code is 0 by definition of the
    # zero group; the dequantized weight is 0 either way.
    x = np.where(Wg == 0, np.float32(0.0), x)
    x = np.clip(x, np.float32(-1.0), np.float32(1.0))
    q = np.round(x)                                            # half to even
    return q.reshape(N, K).astype(np.int8)


def boundary_mask(W: np.ndarray, s64: np.ndarray, g: int, eps: float,
                  rel: float = 1e-6) -> np.ndarray:
    """Elements whose |W| lies within ``rel`` (relative) of the +-0.5 rounding
    boundary |W| = (s + eps)/2, judged in float64 with the float64 scale.

    On these elements a code may legitimately differ between two correct
    implementations; everywhere else it is fixed by the definition.
    """
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    half = 0.5 * (np.asarray(s64, dtype=np.float64).reshape(N, K // g) + eps)
    a = np.abs(_groups(W, g))
    return (np.abs(a - half[:, :, None]) <= rel * half[:, :, None]).reshape(N, K)


def zero_count(q: np.ndarray) -> int:
    """Number of zero codes (the zero ratio of Sec. 3.1 / Table 1 times N*K)."""
    return int(np.count_nonzero(np.asarray(q) == 0))


def ternarize(W: np.ndarray, g: int, eps: float):
    """Convenience: (s64, s32, q, zero count) for one weight matrix."""
    s64 = group_scales_f64(W, g)
    s32 = s64.astype(np.float32)
    q = ternary_codes(W, s32, g, eps)
    return s64, s32, q, zero_count(q)


# --------------------------------------------------------------------------
# 2-bit storage (Sec. 8: packed 2-bit weights plus group scales)
# --------------------------------------------------------------------------
# Format (written out here from its specification; the paper fixes only
# "2 bits per weight"):
#   * codes are a uint8 array [N, K/4]; each row is K/16 little-endian 32-bit
#     words, word w holding elements k = 16*w + e, e = 0..15;
#   * element e = 2*i   sits at bits [2*i,      2*i + 2);
#     element e = 2*i+1 sits at bits [16 + 2*i, 16 + 2*i + 2);
#   * the 2-bit value is the two's complement of the code:
#     0b00 -> 0, 0b01 -> +1, 0b11 -> -1; 0b10 is never written.

def _bit_position(e: int) -> int:
    return 2 * (e // 2) + 16 * (e % 2)


def pack(q: np.ndarray) -> np.ndarray:
    """int8 codes [N, K] in {-1, 0, 1} -> packed uint8 [N, K/4]."""
    q = np.asarray(q)
    N, K = q.shape
    if K % 16:
        raise ValueError("oracle: packing needs K to be a multiple of 16")
    if not np.all((q >= -1) & (q <= 1)):
        raise ValueError("oracle: codes must lie in {-1, 0, +1}")
    two_bit = (q.astype(np.int64) & 3).astype(np.uint32)      # -1 -> 3
    two_bit = two_bit.reshape(N, K // 16, 16)
    words = np.zeros((N, K // 16), dtype=np.uint32)
    for e in range(16):
        words |= two_bit[:, :, e] << np.uint32(_bit_position(e))
    return words.astype("<u4").view(np.uint8).reshape(N, K // 4)


def unpack(codes: np.ndarray, K: int) -> np.ndarray:
    """Packed uint8 [N, K/4] -> int8 codes [N, K]; rejects the unused 0b10."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    N = c.shape[0]
    if c.shape[1] * 4 != K or K % 16:
        raise ValueError("oracle: packed row length does not match K")
    words = c.view("<u4").reshape(N, K // 16).astype(np.uint32)
    out = np.empty((N, K // 16, 16), dtype=np.int8)
    for e in range(16):
        v = (words >> np.uint32(_bit_position(e))) & np.uint32(3)
        if np.any(v == 2):
            raise ValueError("oracle: invalid 2-bit code 0b10")
        out[:, :, e] = np.where(v == 3, -1, v).astype(np.int8)
    return out.reshape(N, K)


# --------------------------------------------------------------------------
# Linear maps (Sec. 3.1: forward with What = s * q, straight-through backward)
# --------------------------------------------------------------------------

def dequantize(q: np.ndarray, s: np.ndarray, g: int) -> np.ndarray:
    """What[n, k] = s[n, k // g] * q[n, k] in float64 (Sec. 3.1)."""
    q = np.asarray(q, dtype=np.float64)
    N, K = q.shape
    s = np.asarray(s, dtype=np.float64).reshape(N, K // g)
    return (q.reshape(N, K // g, g) * s[:, :, None]).reshape(N, K)


def gemm_fwd(X: np.ndarray, q: np.ndarray, s: np.ndarray, g: int) -> np.ndarray:
    """Y[M, N] = X[M, K] . What[N, K]^T in float64.  X may be bf16 bits."""
    Xf = bf16_bits_to_f64(X) if X.dtype == np.uint16 else np.asarray(X, np.float64)
    return Xf @ dequantize(q, s, g).T


def gemm_bwd_dx(dY: np.ndarray, q: np.ndarray, s: np.ndarray, g: int) -> np.ndarray:
    """dX[M, K] = dY[M, N] . What[N, K]: straight-through gradient w.r.t. X."""
    dYf = bf16_bits_to_f64(dY) if dY.dtype == np.uint16 else np.asarray(dY, np.float64)
    return dYf @ dequantize(q, s, g)


def gemm_bwd_dw(dY: np.ndarray, X: np.ndarray) -> np.ndarray:
    """dW[N, K] = dY[M, N]^T . X[M, K]: the identity straight-through
    estimator passes dL/dWhat to the latent weight unchanged."""
    dYf = bf16_bits_to_f64(dY) if dY.dtype == np.uint16 else np.asarray(dY, np.float64)
    Xf = bf16_bits_to_f64(X) if X.dtype == np.uint16 else np.asarray(X, np.float64)
    return dYf.T @ Xf


def gemv(x: np.ndarray, q: np.ndarray, s16: np.ndarray, g: int) -> np.ndarray:
    """y[B, N] = x[B, K] . (q * s16)^T for decode, with float16 scales."""
    xf = bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, np.float64)
    return xf @ dequantize(q, np.asarray(s16).astype(np.float64), g).T


def dense_gemv(x: np.ndarray, W16: np.ndarray) -> np.ndarray:
    """y[B, N] = x[B, K] . W16[N, K]^T in float64: the decode product of a
    layer kept in FP16 (Sec. 7, layer-selective quantization: the first and
    last blocks stay unquantized).  x may be bf16 bits; W16 is float16."""
    xf = bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, np.float64)
    W = np.asarray(W16)
    if W.dtype != np.float16:
        raise ValueError("oracle: the kept layers' weights are float16")
    return xf @ W.astype(np.float64).T


# --------------------------------------------------------------------------
# Metrics
# --------------------------------------------------------------------------

def nrmse(W: np.ndarray, q: np.ndarray, s: np.ndarray, g: int) -> float:
    """||W - s*q||_F / ||W||_F: the weight quantization error of Sec. 7."""
    W = np.asarray(W, dtype=np.float64)
    return float(np.linalg.norm(W - dequantize(q, s, g)) / np.linalg.norm(W))


def rel_fro_error(got: np.ndarray, ref: np.ndarray) -> float:
    """||got - ref||_F / ||ref||_F in float64 (0 when both are zero)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)
