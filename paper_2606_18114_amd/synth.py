"""Seeded synthetic inputs shaped like the Mamba-2 1.3B projections.

This module only draws random numbers and converts float32 to bfloat16 bit
patterns; it holds none of the quantizer's or the linear layer's arithmetic.
Tests, the bench and the oracle checks all draw their inputs from here, so
the HIP path and the oracle see identical bits.

Distributions (numpy ``default_rng``, PCG64):

* weights: float32 N(0, 0.02) (standard deviation 0.02);
* ``outliers=True``: a Bernoulli(0.01) mask, masked entries replaced by
  Laplace(0, 0.2) draws (ten times the weight scale);
* activations: float32 N(0, 1) rounded to bfloat16 (round-to-nearest-even);
* upstream gradients dY: float32 N(0, 0.01) rounded to bfloat16.

Shapes: d_model 2048, d_inner 4096, in_proj 8512 x 2048, out_proj
2048 x 4096, 48 layers (Mamba-2 1.3B, Sec. 3.2 and App. A.2 of the paper).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

D_MODEL = 2048
D_INNER = 4096
IN_PROJ_N = 8512
N_LAYERS = 48
WEIGHT_STD = 0.02


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def weights(rng: np.random.Generator, N: int, K: int, outliers: bool = False,
            std: float = WEIGHT_STD) -> np.ndarray:
    W = rng.standard_normal((N, K), dtype=np.float32) * np.float32(std)
    if outliers:
        mask = rng.random((N, K), dtype=np.float32) < np.float32(0.01)
        n = int(mask.sum())
        W[mask] = rng.laplace(0.0, 10.0 * std, n).astype(np.float32)
    return W


def activations(rng: np.random.Generator, M: int, K: int, std: float = 1.0) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32) * np.float32(std))


@dataclass(frozen=True)
class Config:
    """One workload: a weight [N, K], activations [M, K], group size g."""
    name: str
    N: int
    K: int
    M: int
    g: int
    outliers: bool
    eps: float = 1e-5


# Single ternary linear, out_proj, in_proj (forward + STE backward) and the
# group-size sweep on in_proj with 2048 tokens.
C1 = Config("single_linear_256x512_m16", 256, 512, 16, 128, False)
C2 = Config("out_proj_2048x4096_m4096", D_MODEL, D_INNER, 4096, 128, False)
C3 = Config("in_proj_8512x2048_m16384", IN_PROJ_N, D_MODEL, 16384, 128, True)
C5_GROUPS = (32, 64, 128, 256, 512)


def c5(g: int) -> Config:
    return Config(f"in_proj_8512x2048_m2048_g{g}", IN_PROJ_N, D_MODEL, 2048, g, True)


def single_linear_inputs(cfg: Config, seed: int = 0):
    """C1 recipe: one generator, W drawn first, then X."""
    rng = np.random.default_rng(seed)
    W = weights(rng, cfg.N, cfg.K, cfg.outliers)
    X = activations(rng, cfg.M, cfg.K)
    return W, X


def layer_weight(cfg: Config, seed: int) -> np.ndarray:
    return weights(np.random.default_rng(seed), cfg.N, cfg.K, cfg.outliers)


def layer_acts(M: int, K: int, seed: int, std: float = 1.0) -> np.ndarray:
    return activations(np.random.default_rng(seed), M, K, std)


# Seeds of the projection configs: W 0, X 1, dY 2.
SEED_W, SEED_X, SEED_DY = 0, 1, 2
DY_STD = 0.01

# Decode over all 48 layers: in_proj layer l seed 1000+l, out_proj 2000+l,
# decode input x of layer l 3000+l (in_proj) / 4000+l (out_proj).
DECODE_IN = Config("decode_in_proj", IN_PROJ_N, D_MODEL, 1, 128, True)
DECODE_OUT = Config("decode_out_proj", D_MODEL, D_INNER, 1, 128, False)


def decode_seed(kind: str, layer: int) -> int:
    return {"in_w": 1000, "out_w": 2000, "in_x": 3000, "out_x": 4000}[kind] + layer


# Mamba-2 mixer parameters and states for the decode step between the
# projections (64 heads of 64 channels, d_state 128, d_conv 4):
#   conv taps and bias U(-1/2, 1/2); step sizes dt log-uniform in
#   [1e-3, 1e-1] stored as dt_bias = softplus^-1(dt); A_log = log U(1, 16);
#   D = 1; norm weight 1 + N(0, 0.1); conv state N(0, 1) and SSM state
#   N(0, 0.5), both rounded to float16.
HEADDIM, D_STATE, D_CONV = 64, 128, 4


def mixer_params(rng: np.random.Generator, nheads: int):
    d_inner = nheads * HEADDIM
    conv_dim = d_inner + 2 * D_STATE
    dt = np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), nheads))
    return dict(
        conv_w=rng.uniform(-0.5, 0.5, (conv_dim, D_CONV)).astype(np.float32),
        conv_b=rng.uniform(-0.5, 0.5, conv_dim).astype(np.float32),
        dt_bias=(dt + np.log(-np.expm1(-dt))).astype(np.float32),
        A_log=np.log(rng.uniform(1.0, 16.0, nheads)).astype(np.float32),
        D=np.ones(nheads, np.float32),
        norm_w=(1.0 + 0.1 * rng.standard_normal(d_inner)).astype(np.float32))


def mixer_states(rng: np.random.Generator, B: int, nheads: int):
    d_inner = nheads * HEADDIM
    conv_dim = d_inner + 2 * D_STATE
    return (rng.standard_normal((B, conv_dim, D_CONV)).astype(np.float16),
            (0.5 * rng.standard_normal((B, nheads, HEADDIM, D_STATE))).astype(np.float16))


def in_proj_out(rng: np.random.Generator, B: int, nheads: int) -> np.ndarray:
    """A float32 stand-in for in_proj's output [B, 2 d_inner + 2 d_state + nheads]."""
    d_inner = nheads * HEADDIM
    return rng.standard_normal((B, 2 * d_inner + 2 * D_STATE + nheads)).astype(np.float32)
