"""Quantization-aware training with the ternary linear layer (paper Sec. 3.1).

``TernaryLinear`` replaces a Mamba-2 ``in_proj`` / ``out_proj``: it keeps
float32 latent weights, and on every forward call

  * recomputes the group scales and ternary codes from the current weights
    (``tm_ternarize_pack``; the scale is not a learned parameter),
  * applies the dequantized weights to the bfloat16 activations
    (``tm_tgemm_fwd``, float32 output);

and its backward pass is the straight-through estimator: the gradient passes
the quantizer unchanged, so ``dX = dY . (q s)`` (``tm_tgemm_bwd_dx``) and
``dW = dY^T . X`` (``tm_tgemm_bwd_dw_ste``).  The incoming gradient is taken
in bfloat16, the precision the backward kernels read.

Every product runs in the library's kernels; this module only wires them
into autograd (a dtype cast of the gradient and reshapes are the only torch
operations on the data).  ``pack_for_decode`` returns the deployment format
(2-bit codes and float16 group scales) that ``ops.tgemv`` reads.
"""

from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import ops


class TernaryLinearFn(torch.autograd.Function):
    """y = x . (q s)^T with q, s recomputed from `weight`; straight-through backward."""

    @staticmethod
    def forward(ctx, x: torch.Tensor, weight: torch.Tensor, g: int, eps: float,
                zero_count: Optional[torch.Tensor]) -> torch.Tensor:
        N, K = weight.shape
        if x.shape[-1] != K:
            raise ValueError(f"x has {x.shape[-1]} features, the layer takes {K}")
        lead = x.shape[:-1]
        x2 = x.reshape(-1, K)
        if x2.dtype != torch.bfloat16:
            raise TypeError(f"x must be bfloat16 (got {x2.dtype}): the layer is W1.58A16")
        x2 = x2.contiguous()
        codes, scales, _, _ = ops.ternarize_pack(weight.detach().contiguous(), g, eps,
                                                 zero_count=zero_count, want_f16=False,
                                                 want_zero_count=zero_count is not None)
        y = ops.tgemm_fwd(x2, codes, scales, g)
        ctx.save_for_backward(x2, codes, scales)
        ctx.g = g
        ctx.lead = lead
        ctx.x_dtype = x.dtype
        return y.reshape(*lead, N)

    @staticmethod
    def backward(ctx, gy: torch.Tensor):
        x2, codes, scales = ctx.saved_tensors
        N = codes.shape[0]
        dy = gy.reshape(-1, N)
        if dy.dtype != torch.bfloat16:
            dy = dy.to(torch.bfloat16)
        dy = dy.contiguous()
        dx = dw = None
        if ctx.needs_input_grad[0]:
            dx = ops.tgemm_bwd_dx(dy, codes, scales, ctx.g)
            dx = dx.to(ctx.x_dtype).reshape(*ctx.lead, x2.shape[1])
        if ctx.needs_input_grad[1]:
            dw = ops.tgemm_bwd_dw_ste(dy, x2)
        return dx, dw, None, None, None


class TernaryLinear(torch.nn.Module):
    """Grouped-absmean ternary linear layer (no bias; the Mamba-2 projections
    have none).  weight: float32 [out_features, in_features]; groups of `g`
    consecutive input features of one output row share a scale."""

    def __init__(self, in_features: int, out_features: int, g: int = 128, eps: float = 1e-5,
                 device: Optional[torch.device] = None, track_zero_ratio: bool = True):
        super().__init__()
        if in_features % g or in_features % 64:
            raise ValueError(f"in_features={in_features} must be a multiple of g={g} and of 64")
        self.in_features, self.out_features, self.g, self.eps = in_features, out_features, g, eps
        self.weight = torch.nn.Parameter(
            torch.empty((out_features, in_features), dtype=torch.float32, device=device))
        torch.nn.init.normal_(self.weight, 0.0, 0.02)
        self._zc = (torch.zeros((1,), dtype=torch.int64, device=device)
                    if track_zero_ratio else None)

    @classmethod
    def from_weight(cls, weight: torch.Tensor, g: int = 128, eps: float = 1e-5) -> "TernaryLinear":
        """Wrap existing (e.g. pretrained) float weights [out, in]."""
        m = cls(weight.shape[1], weight.shape[0], g, eps, device=weight.device)
        with torch.no_grad():
            m.weight.copy_(weight.float())
        return m

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        if self._zc is not None and self._zc.device != self.weight.device:
            self._zc = self._zc.to(self.weight.device)
        return TernaryLinearFn.apply(x, self.weight, self.g, self.eps, self._zc)

    def zero_ratio(self) -> float:
        """Fraction of zero codes in the last forward call (Sec. 3.1 tracks it
        during training); reading it synchronizes with the device."""
        if self._zc is None:
            raise RuntimeError("zero-ratio tracking is off for this layer")
        return int(self._zc.item()) / (self.in_features * self.out_features)

    @torch.no_grad()
    def pack_for_decode(self) -> Tuple[torch.Tensor, torch.Tensor]:
        """(codes uint8 [out, in/4], scales float16 [out, in/g]) of the current
        weights: the storage format of the decode GEMV."""
        codes, _, s16, _ = ops.ternarize_pack(self.weight.detach().contiguous(), self.g,
                                              self.eps, want_zero_count=False)
        return codes, s16

    def extra_repr(self) -> str:
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"g={self.g}, eps={self.eps}")


def flops_per_step(tokens: int, layer: TernaryLinear) -> float:
    """Algorithmic flops of one forward + straight-through backward (three
    dense products of 2 * tokens * in * out each; zeros not discounted)."""
    return 3.0 * 2.0 * tokens * layer.in_features * layer.out_features


__all__ = ["TernaryLinear", "TernaryLinearFn", "flops_per_step"]
