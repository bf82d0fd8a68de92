"""CPU oracle for the scale-parameterization variants of the ternary layer.

TEST INFRASTRUCTURE ONLY (see ``oracle/ternary.py``): only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline may use it.  It
shares no code with the HIP kernels.

The paper's appendix (Decoupled Quantization Ablations) and Sec. 4
(Zero-Ratio Collapse) test three changes to the standard layer:

* Asymmetric gate thresholds: the rows of ``in_proj`` that feed the gate
  (rows 0-4095) round against 0.8 x absmean instead of the absmean, while the
  code is still scaled by the absmean.  Written here as a per-row threshold
  multiplier m[n]: the code divides by m[n] * s + eps instead of s + eps.
* Decoupled quantization: a fixed absmean threshold tau_g decides the codes and
  an independent, learnable magnitude alpha_g scales them, What = alpha_g * q.
  Its gradient is d alpha_g = sum_i q_i * dWhat_i over the group's elements
  (the codes do not depend on alpha).
* Learnable scale: s_g itself an nn.Parameter.  Two readings of its
  gradient are kept.  (a) Magnitude only: sum_i q_i * dWhat_i, the threshold
  path through the rounding cut by the hard forward quantization.  (b) The
  straight-through estimator applied to the rounding alone (round passes
  the gradient unchanged, clip keeps its derivative), which is what a PyTorch
  layer computing s * ste(round(clip(w / (s + eps)))) gives: the threshold
  term feeds back into s and the weights' gradient is clip-masked
  (``scale_ste_grad``).

Readings: the multiplied threshold is rounded to
float32 once (fl32(m * s)), then eps is added in float32, then the quotient is
taken in float32 as for the standard code; dWhat is the gradient with respect
to the dequantized weight, dY^T * X.
"""

from __future__ import annotations

import numpy as np

from . import ternary as T

__all__ = ["ternary_codes_thresh", "boundary_mask_thresh", "group_code_dot",
           "scale_ste_grad"]


def ternary_codes_thresh(W: np.ndarray, s32: np.ndarray, g: int, eps: float,
                         row_mult: np.ndarray) -> np.ndarray:
    """q = round(clip(W / (m[n] * s + eps), -1, 1)) in {-1, 0, +1}, as int8.

    With every m[n] = 1 this is the standard code of Sec. 3.1.
    """
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    m = np.asarray(row_mult, dtype=np.float32).reshape(N)
    if not np.all(np.isfinite(m)) or np.any(m <= 0):
        raise ValueError("oracle: threshold multipliers must be finite and > 0")
    s32 = np.asarray(s32, dtype=np.float32).reshape(N, K // g)
    tau = (m[:, None] * s32).astype(np.float32)               # float32 product
    return T.ternary_codes(W, tau, g, eps)


def boundary_mask_thresh(W: np.ndarray, s64: np.ndarray, g: int, eps: float,
                         row_mult: np.ndarray, rel: float = 1e-6) -> np.ndarray:
    """Elements within ``rel`` of the rounding boundary |W| = (m s + eps) / 2."""
    N, K = np.asarray(W).shape
    m = np.asarray(row_mult, dtype=np.float64).reshape(N)
    tau64 = m[:, None] * np.asarray(s64, dtype=np.float64).reshape(N, K // g)
    return T.boundary_mask(W, tau64, g, eps, rel)


def group_code_dot(q: np.ndarray, dWhat: np.ndarray, g: int) -> np.ndarray:
    """out[n, j] = sum_{i < g} q[n, j g + i] * dWhat[n, j g + i], in float64:
    the gradient of a per-group magnitude that multiplies the codes."""
    q = np.asarray(q, dtype=np.float64)
    d = np.asarray(dWhat, dtype=np.float64)
    N, K = q.shape
    if d.shape != (N, K) or K % g:
        raise ValueError("oracle: q and dWhat must be [N, K] with K % g == 0")
    return (q * d).reshape(N, K // g, g).sum(axis=2)


def scale_ste_grad(W: np.ndarray, q: np.ndarray, s32: np.ndarray, dWhat: np.ndarray, g: int,
                   eps: float):
    """Gradients of a learnable scale s (Sec. 4) and of the latent weights
    when only the rounding is straight-through:

        x = clip(w / (s + eps), -1, 1),  q = round(x),  What = s * q,
        d What / d s = q - m * s * w / (s + eps)^2,
        d What / d w = m * s / (s + eps),

    with m = 1 where the float32 quotient |w| / fl32(s + eps) is at most 1
    (clip passes the gradient on its closed range) and 0 elsewhere; s + eps
    is the float32 sum the codes are decided with.  Returns (ds [N, K/g],
    dw [N, K]) in float64: ds[n, j] = sum over group j of dWhat * dWhat/ds,
    dw = dWhat * dWhat/dw.  q are the layer's codes (ternarized against s)."""
    W = np.asarray(W, dtype=np.float32)
    N, K = W.shape
    if K % g:
        raise ValueError("oracle: K must be a multiple of g")
    s32 = np.asarray(s32, dtype=np.float32).reshape(N, K // g)
    if not np.all(np.isfinite(s32)) or np.any(s32 <= 0):
        raise ValueError("oracle: a learnable scale must be finite and > 0")
    d32 = (s32 + np.float32(eps)).astype(np.float32)
    d_full = np.repeat(d32, g, axis=1)
    quot = (np.abs(W) / d_full).astype(np.float32)          # float32 quotient
    m = (quot <= np.float32(1.0)).astype(np.float64)
    s64 = np.repeat(s32.astype(np.float64), g, axis=1)
    d64 = d_full.astype(np.float64)
    dwh = np.asarray(dWhat, dtype=np.float64)
    qf = np.asarray(q, dtype=np.float64)
    terms = dwh * (qf - m * s64 * W.astype(np.float64) / (d64 * d64))
    ds = terms.reshape(N, K // g, g).sum(axis=2)
    dw = dwh * m * s64 / d64
    return ds, dw
