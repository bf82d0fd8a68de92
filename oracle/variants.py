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
* Learnable scale: s_g itself an nn.Parameter.  Its magnitude path has the
  same gradient, sum_i q_i * dWhat_i; the threshold path through the rounding
  is cut by the hard forward quantization (the straight-through estimator of
  Sec. 3.1 passes gradients to W only), which is the reading taken here.

Readings: the multiplied threshold is rounded to
float32 once (fl32(m * s)), then eps is added in float32, then the quotient is
taken in float32 as for the standard code; dWhat is the gradient with respect
to the dequantized weight, dY^T * X.
"""

from __future__ import annotations

import numpy as np

from . import ternary as T

__all__ = ["ternary_codes_thresh", "boundary_mask_thresh", "group_code_dot"]


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
