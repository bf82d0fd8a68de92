"""Quantization-aware training with the ternary linear layer (paper Sec. 3.1).

``TernaryLinear`` replaces a Mamba-2 ``in_proj`` / ``out_proj``: it keeps
float32 latent weights, and on every forward call

  * recomputes the group scales and ternary codes from the current weights
    (``tm_ternarize_pack``; the scale is not a learned parameter),
  * applies the dequantized weights to the bfloat16 activations
    (``tm_tgemm_fwd``, float32 output);

and its backward pass is the straight-through estimator: the gradient passes
the quantizer unchanged, so ``dX = dY . (q s)`` (``tm_tgemm_bwd_dx_f16``:
one float16 pass, each dequantized weight within 2^-11 relative; or the
two-pass ``tm_tgemm_bwd_dx`` with ``dx_precision="exact"``) and
``dW = dY^T . X`` (``tm_tgemm_bwd_dw_ste``).  The incoming gradient is taken
in bfloat16, the precision the backward kernels read.

The scale variants the paper tests against this layer are options of the
same module: a learned magnitude next to the absmean threshold (decoupled),
a learned scale that is threshold and magnitude at once (learnable, whose
zero ratio collapses in Sec. 4), and per-row threshold multipliers (the
appendix's 0.8 x absmean on the gate rows).  Their extra calls are
``tm_ternarize_pack_thresh``, ``tm_ternarize_codes`` and, in the backward,
``tm_group_code_dot`` for the gradient of the learned scale.

Every product runs in the library's kernels; this module only wires them
into autograd (a dtype cast of the gradient and reshapes are the only torch
operations on the data).  ``pack_for_decode`` returns the deployment format
(2-bit codes and float16 group scales) that ``ops.tgemv`` reads.
"""

from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import ops


SCALE_MODES = ("absmean", "decoupled", "learnable", "learnable_ste")


class TernaryLinearFn(torch.autograd.Function):
    """y = x . (q m)^T with straight-through backward.

    mode "absmean": q and the magnitude m = s are recomputed from `weight`
    (Sec. 3.1); `scale` is None.  mode "decoupled": q from the recomputed
    absmean threshold, m = `scale` (a learned alpha_g, appendix Decoupled
    Quantization Ablations).  mode "learnable": `scale` is the learned s_g of
    Sec. 4, used as the rounding threshold and as the magnitude.  `row_mult`
    (float32 [out] or None) multiplies each row's absmean threshold.
    In "decoupled" and "learnable" the gradient of the learned scale is
    sum_group q * dWhat (the hard forward rounding passes nothing back
    through the threshold) and the weights get dWhat.  "learnable_ste" has
    the same forward as "learnable", with only the rounding straight-through:
    the scale also receives the threshold term, and the weights' gradient is
    clip-masked (``tm_scale_ste_grad``).
    """

    @staticmethod
    def forward(ctx, x: torch.Tensor, weight: torch.Tensor, scale: Optional[torch.Tensor],
                g: int, eps: float, zero_count: Optional[torch.Tensor], mode: str,
                row_mult: Optional[torch.Tensor],
                out_dtype: torch.dtype = torch.float32,
                dx_precision: str = "f16") -> torch.Tensor:
        N, K = weight.shape
        if x.shape[-1] != K:
            raise ValueError(f"x has {x.shape[-1]} features, the layer takes {K}")
        lead = x.shape[:-1]
        x2 = x.reshape(-1, K)
        if x2.dtype != torch.bfloat16:
            raise TypeError(f"x must be bfloat16 (got {x2.dtype}): the layer is W1.58A16")
        x2 = x2.contiguous()
        w = weight.detach().contiguous()
        want_zc = zero_count is not None
        if mode in ("learnable", "learnable_ste"):
            mag = scale.detach().contiguous()
            codes, _ = ops.ternarize_codes(w, mag, g, eps, zero_count=zero_count,
                                           want_zero_count=want_zc)
        else:
            codes, absmean, _, _ = ops.ternarize_pack(w, g, eps, zero_count=zero_count,
                                                      want_f16=False, want_zero_count=want_zc,
                                                      row_mult=row_mult)
            mag = absmean if mode == "absmean" else scale.detach().contiguous()
        y = ops.tgemm_fwd(x2, codes, mag, g, out_dtype=out_dtype)
        ctx.save_for_backward(x2, codes, mag, w if mode == "learnable_ste" else None)
        ctx.g = g
        ctx.eps = eps
        ctx.ste_scale = mode == "learnable_ste"
        ctx.lead = lead
        ctx.x_dtype = x.dtype
        ctx.learned = mode != "absmean"
        ctx.dx_precision = dx_precision
        return y.reshape(*lead, N)

    @staticmethod
    def backward(ctx, gy: torch.Tensor):
        x2, codes, mag, w = ctx.saved_tensors
        N = codes.shape[0]
        dy = gy.reshape(-1, N)
        if dy.dtype != torch.bfloat16:
            dy = dy.to(torch.bfloat16)
        dy = dy.contiguous()
        dx = dw = dscale = None
        if ctx.needs_input_grad[0]:
            dx = ops.tgemm_bwd_dx(dy, codes, mag, ctx.g, precision=ctx.dx_precision)
            dx = dx.to(ctx.x_dtype).reshape(*ctx.lead, x2.shape[1])
        want_scale = ctx.learned and ctx.needs_input_grad[2]
        if ctx.needs_input_grad[1] or want_scale:
            dw_hat = ops.tgemm_bwd_dw_ste(dy, x2)   # gradient w.r.t. the dequantized weights
            if ctx.ste_scale:
                # scale gradient with the threshold term; the weights' gradient
                # clip-masked, written over dWhat
                dscale, dw_m = ops.scale_ste_grad(w, codes, mag, dw_hat, ctx.g, ctx.eps,
                                                  in_place=ctx.needs_input_grad[1],
                                                  want_dW=ctx.needs_input_grad[1])
                if ctx.needs_input_grad[1]:
                    dw = dw_m
                if not want_scale:
                    dscale = None
            else:
                if want_scale:
                    dscale = ops.group_code_dot(codes, dw_hat, ctx.g)
                if ctx.needs_input_grad[1]:
                    dw = dw_hat
        return dx, dw, dscale, None, None, None, None, None, None, None


class TernaryLinear(torch.nn.Module):
    """Grouped-absmean ternary linear layer (no bias; the Mamba-2 projections
    have none).  weight: float32 [out_features, in_features]; groups of `g`
    consecutive input features of one output row share a scale.

    scale_mode "absmean" (the paper's layer): the scale is recomputed from
    the weights on every call and is not a parameter.  "decoupled": codes
    from the recomputed absmean, magnitude the parameter `scale`.
    "learnable": the parameter `scale` is both threshold and magnitude;
    "learnable_ste": the same with only the rounding straight-through (the
    scale's gradient keeps the threshold term, the weights' is clip-masked).
    The parameter starts at the absmean of the weights (``reset_scale``, run on
    the first call unless it was run before or the scale was loaded with
    ``load_state_dict``).  threshold_mult (float32 [out]) scales
    each row's absmean threshold (e.g. 0.8 on the gate rows of in_proj).
    out_dtype: float32 (default) or bfloat16, the output rounded once as a
    bfloat16 model stores it; the incoming gradient then needs no cast.
    dx_precision: "f16" (default, one float16 pass for the input gradient)
    or "exact" (two bfloat16 passes, 16 bits of every scale).
    """

    def __init__(self, in_features: int, out_features: int, g: int = 128, eps: float = 1e-5,
                 device: Optional[torch.device] = None, track_zero_ratio: bool = True,
                 scale_mode: str = "absmean", threshold_mult: Optional[torch.Tensor] = None,
                 out_dtype: torch.dtype = torch.float32, dx_precision: str = "f16"):
        super().__init__()
        if dx_precision not in ("f16", "exact"):
            raise ValueError("dx_precision must be 'f16' or 'exact'")
        self.dx_precision = dx_precision
        if out_dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("out_dtype must be torch.float32 or torch.bfloat16")
        self.out_dtype = out_dtype
        if in_features % g or in_features % 64:
            raise ValueError(f"in_features={in_features} must be a multiple of g={g} and of 64")
        if scale_mode not in SCALE_MODES:
            raise ValueError(f"scale_mode must be one of {SCALE_MODES}")
        if threshold_mult is not None:
            if scale_mode in ("learnable", "learnable_ste"):
                raise ValueError("a learnable scale is its own threshold: no threshold_mult")
            if threshold_mult.shape != (out_features,):
                raise ValueError(f"threshold_mult must have shape ({out_features},)")
        self.in_features, self.out_features, self.g, self.eps = in_features, out_features, g, eps
        self.scale_mode = scale_mode
        self.weight = torch.nn.Parameter(
            torch.empty((out_features, in_features), dtype=torch.float32, device=device))
        torch.nn.init.normal_(self.weight, 0.0, 0.02)
        if scale_mode == "absmean":
            self.scale = None
        else:
            self.scale = torch.nn.Parameter(
                torch.zeros((out_features, in_features // g), dtype=torch.float32, device=device))
        self._scale_ready = scale_mode == "absmean"
        # a scale that arrives through load_state_dict (a checkpoint, a resumed
        # run) is the trained one: it must not be reset to the absmean
        self.register_load_state_dict_pre_hook(TernaryLinear._mark_scale_loaded)
        self.register_buffer(
            "threshold_mult",
            None if threshold_mult is None
            else threshold_mult.detach().to(device=device, dtype=torch.float32).contiguous())
        self._zc = (torch.zeros((1,), dtype=torch.int64, device=device)
                    if track_zero_ratio else None)

    @classmethod
    def from_weight(cls, weight: torch.Tensor, g: int = 128, eps: float = 1e-5,
                    **kw) -> "TernaryLinear":
        """Wrap existing (e.g. pretrained) float weights [out, in]."""
        m = cls(weight.shape[1], weight.shape[0], g, eps, device=weight.device, **kw)
        with torch.no_grad():
            m.weight.copy_(weight.float())
        if m.scale is not None and weight.is_cuda:
            m.reset_scale()
        return m

    @staticmethod
    def _mark_scale_loaded(module, state_dict, prefix, *args) -> None:
        if module.scale is not None and (prefix + "scale") in state_dict:
            module._scale_ready = True

    @torch.no_grad()
    def reset_scale(self) -> None:
        """Set the learned scale to the absmean of the current weights."""
        if self.scale is None:
            raise RuntimeError("the absmean layer has no scale parameter")
        ops.ternarize_pack(self.weight.detach().contiguous(), self.g, self.eps,
                           scales=self.scale.data, want_f16=False, want_zero_count=False)
        self._scale_ready = True

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        if self._zc is not None and self._zc.device != self.weight.device:
            self._zc = self._zc.to(self.weight.device)
        if not self._scale_ready:
            self.reset_scale()
        return TernaryLinearFn.apply(x, self.weight, self.scale, self.g, self.eps, self._zc,
                                     self.scale_mode, self.threshold_mult, self.out_dtype,
                                     self.dx_precision)

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
        w = self.weight.detach().contiguous()
        if self.scale_mode == "absmean":
            codes, _, s16, _ = ops.ternarize_pack(w, self.g, self.eps, want_zero_count=False,
                                                  row_mult=self.threshold_mult)
            return codes, s16
        if self.scale_mode in ("learnable", "learnable_ste"):
            codes, _ = ops.ternarize_codes(w, self.scale.detach().contiguous(), self.g, self.eps,
                                           want_zero_count=False)
        else:
            codes, _, _, _ = ops.ternarize_pack(w, self.g, self.eps, want_f16=False,
                                                want_zero_count=False,
                                                row_mult=self.threshold_mult)
        return codes, self.scale.detach().to(torch.float16)

    def extra_repr(self) -> str:
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"g={self.g}, eps={self.eps}, scale_mode={self.scale_mode}, "
                f"out_dtype={self.out_dtype}")


def flops_per_step(tokens: int, layer: TernaryLinear) -> float:
    """Algorithmic flops of one forward + straight-through backward (three
    dense products of 2 * tokens * in * out each; zeros not discounted)."""
    return 3.0 * 2.0 * tokens * layer.in_features * layer.out_features


__all__ = ["SCALE_MODES", "TernaryLinear", "TernaryLinearFn", "flops_per_step"]
