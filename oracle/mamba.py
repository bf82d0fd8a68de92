"""CPU oracle of one Mamba-2 mixer decode step between the two projections.

TEST INFRASTRUCTURE ONLY (see ``oracle/ternary.py``): only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline may use it.  It
shares no code with the HIP kernels.

The paper ternarizes only the projections and keeps the selective-state-space
part in FP16 (Sec. 3.2: convolution, SSM parameters and state stay in
float16; Sec. 8: batch-1 decode).  A decoding layer therefore runs
in_proj -> the step below -> out_proj.  Written from the Mamba-2 layer the
paper builds on (d_model 2048, d_inner 4096 = 64 heads of 64, d_state 128,
one group of B/C, d_conv 4, gated RMSNorm before out_proj):

* in_proj output per token: z [d_inner] | xBC [d_inner + 2 d_state] | dt [nheads];
* causal depthwise convolution step: the per-channel window of the last
  d_conv inputs (the conv state, oldest first) shifts by one and takes the
  new xBC; out = sum_t window[t] * w[c, t] + b[c], then SiLU;
* x, B, C = split(out); dt' = softplus(dt + dt_bias); a = exp(dt' * A), with
  A = -exp(A_log) per head;
* state[h, p, n] <- a_h * state[h, p, n] + dt'_h * x[h, p] * B[n];
  y[h, p] = sum_n state[h, p, n] * C[n] + D_h * x[h, p];
* gate and normalize: g = y * silu(z); out = g / sqrt(mean(g^2) + eps) * w_norm
  (one normalization group over all d_inner channels).

Readings: states are stored in float16 (the FP16 SSM), each update computed
from the stored float16 values and rounded to float16 once when stored; the
parameters are given as float32 arrays; every other quantity is float64
here.  The normalized output is returned in float64; the layer feeds its
bfloat16 rounding to out_proj.
"""

from __future__ import annotations

import numpy as np

__all__ = ["split_in_proj", "conv_step", "ssm_step", "gated_rmsnorm", "mixer_step",
           "softplus", "silu", "rmsnorm"]


def softplus(v: np.ndarray) -> np.ndarray:
    """log(1 + e^v), evaluated stably."""
    v = np.asarray(v, dtype=np.float64)
    return np.where(v > 20.0, v, np.log1p(np.exp(np.minimum(v, 20.0))))


def silu(v: np.ndarray) -> np.ndarray:
    """v * sigmoid(v)."""
    v = np.asarray(v, dtype=np.float64)
    return v / (1.0 + np.exp(-v))


def split_in_proj(zxbcdt: np.ndarray, d_inner: int, d_state: int, nheads: int):
    """[B, 2 d_inner + 2 d_state + nheads] -> z, xBC, dt."""
    zxbcdt = np.asarray(zxbcdt, dtype=np.float64)
    conv_dim = d_inner + 2 * d_state
    if zxbcdt.shape[-1] != d_inner + conv_dim + nheads:
        raise ValueError("oracle: in_proj width does not match the layer shape")
    return (zxbcdt[..., :d_inner], zxbcdt[..., d_inner:d_inner + conv_dim],
            zxbcdt[..., d_inner + conv_dim:])


def conv_step(conv_state: np.ndarray, xBC: np.ndarray, w: np.ndarray, b: np.ndarray):
    """One causal depthwise convolution step.

    conv_state float16 [B, C, d_conv] (oldest first), xBC [B, C], w [C, d_conv],
    b [C] -> (SiLU of the convolution output [B, C] float64, the new state
    as float16)."""
    st = np.asarray(conv_state, dtype=np.float16)
    window = np.concatenate([st[..., 1:].astype(np.float64),
                             np.asarray(xBC, np.float64)[..., None]], axis=-1)
    out = (window * np.asarray(w, np.float64)[None]).sum(-1) + np.asarray(b, np.float64)[None]
    return silu(out), window.astype(np.float16)


def ssm_step(state: np.ndarray, x: np.ndarray, Bv: np.ndarray, Cv: np.ndarray,
             dt: np.ndarray, dt_bias: np.ndarray, A_log: np.ndarray, D: np.ndarray):
    """One selective-state-space step.

    state float16 [B, H, P, N]; x [B, H, P]; Bv, Cv [B, N]; dt [B, H];
    dt_bias, A_log, D [H].  Returns (y [B, H, P] float64, new state float16)."""
    s = np.asarray(state, dtype=np.float16).astype(np.float64)
    dtp = softplus(np.asarray(dt, np.float64) + np.asarray(dt_bias, np.float64)[None])
    a = np.exp(dtp * -np.exp(np.asarray(A_log, np.float64))[None])          # [B, H]
    x = np.asarray(x, np.float64)
    new = (s * a[:, :, None, None]
           + (dtp[:, :, None] * x)[..., None] * np.asarray(Bv, np.float64)[:, None, None, :])
    y = (new * np.asarray(Cv, np.float64)[:, None, None, :]).sum(-1) \
        + np.asarray(D, np.float64)[None, :, None] * x
    return y, new.astype(np.float16)


def gated_rmsnorm(y: np.ndarray, z: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """g = y * silu(z); g / sqrt(mean(g^2) + eps) * w, per token."""
    g = np.asarray(y, np.float64) * silu(z)
    r = 1.0 / np.sqrt((g * g).mean(axis=-1, keepdims=True) + eps)
    return g * r * np.asarray(w, np.float64)[None]


def mixer_step(zxbcdt, conv_state, ssm_state, conv_w, conv_b, dt_bias, A_log, D, norm_w,
               eps: float, headdim: int, d_state: int):
    """The whole step between in_proj and out_proj for a batch of tokens.

    Returns (out [B, d_inner] float64, new conv state float16, new SSM state
    float16)."""
    nheads = np.asarray(A_log).shape[0]
    d_inner = nheads * headdim
    z, xBC, dt = split_in_proj(zxbcdt, d_inner, d_state, nheads)
    u, conv_new = conv_step(conv_state, xBC, conv_w, conv_b)
    x = u[:, :d_inner].reshape(-1, nheads, headdim)
    Bv, Cv = u[:, d_inner:d_inner + d_state], u[:, d_inner + d_state:]
    y, ssm_new = ssm_step(ssm_state, x, Bv, Cv, dt, dt_bias, A_log, D)
    out = gated_rmsnorm(y.reshape(-1, d_inner), z, norm_w, eps)
    return out, conv_new, ssm_new


def rmsnorm(residual: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """The block's pre-norm: residual / sqrt(mean(residual^2) + eps) * w, per token
    (the next layer's in_proj input before its bfloat16 rounding)."""
    r = np.asarray(residual, np.float64)
    return r / np.sqrt((r * r).mean(axis=-1, keepdims=True) + eps) * np.asarray(w, np.float64)[None]
