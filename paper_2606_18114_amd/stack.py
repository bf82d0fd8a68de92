"""Layer-selective quantization of a Mamba-2 projection stack (paper Sec. 7,
Table 10: keeping the first and last blocks in FP16 recovers most of the
quality lost to ternarization).

* ``keep_first_last(n_layers, n)``: the layer indices the paper's setting
  keeps unquantized (the first n and the last n blocks).
* ``quantize_projections(blocks, keep, ...)``: QAT wiring.  Every block
  outside ``keep`` gets its ``in_proj`` / ``out_proj`` replaced by a
  ``TernaryLinear`` initialised from the existing weights; the kept blocks'
  projections stay the model's own dense layers.
* ``DecodeStack``: the deployment form of the projections of all layers,
  2-bit codes + float16 group scales for the ternary layers and float16
  weights for the kept ones, and one decode token over them
  (``tm_tgemv`` for the ternary layers, ``tm_dgemv`` for the kept ones).

Only argument marshalling and packing happen here; every product runs in
the library's kernels.
"""

from __future__ import annotations

from typing import Callable, Dict, Iterable, List, Optional, Sequence

import torch

from . import ops
from .qat import TernaryLinear

PROJECTIONS = ("in_proj", "out_proj")


def keep_first_last(n_layers: int, n: int) -> List[int]:
    """Indices of the first n and the last n of n_layers blocks."""
    if n < 0 or 2 * n > n_layers:
        raise ValueError(f"cannot keep {n} blocks at each end of {n_layers}")
    return sorted(set(range(n)) | set(range(n_layers - n, n_layers)))


def quantize_projections(blocks: Sequence[torch.nn.Module], keep: Iterable[int] = (),
                         g: int = 128, eps: float = 1e-5, **layer_kw) -> List[int]:
    """Replace in_proj / out_proj of every block not in ``keep`` by a
    TernaryLinear holding the same weights; returns the quantized indices.
    A projection must be a bias-free torch.nn.Linear (Mamba-2's are)."""
    keep = set(keep)
    if any(i < 0 or i >= len(blocks) for i in keep):
        raise ValueError("keep holds an index outside the stack")
    done = []
    for i, blk in enumerate(blocks):
        if i in keep:
            continue
        for name in PROJECTIONS:
            lin = getattr(blk, name)
            if not isinstance(lin, torch.nn.Linear) or lin.bias is not None:
                raise TypeError(f"block {i}.{name} must be a bias-free torch.nn.Linear")
            setattr(blk, name, TernaryLinear.from_weight(lin.weight.detach(), g=g, eps=eps,
                                                         **layer_kw))
        done.append(i)
    return done


class DecodeStack:
    """Packed decode weights of an L-layer stack of (in_proj, out_proj) pairs.

    weight(kind, layer) -> float32 [N, K] on the GPU gives the master weights
    (kind "in" or "out"); layers in ``keep`` are stored as float16, the
    others ternarized (``tm_ternarize_pack``) into codes + float16 scales.
    Each kind's ternary layers and kept layers form two contiguous arenas in
    layer order, so a token is four launches.  Inputs and outputs of a token
    live in per-kind buffers ``x[kind]`` [L, B, K] and ``y[kind]`` [L, B, N]
    in layer order; the launches read and write views of them.
    """

    def __init__(self, weight: Callable[[str, int], torch.Tensor], n_layers: int,
                 shapes: Dict[str, tuple], keep: Iterable[int] = (), g: int = 128,
                 eps: float = 1e-5, batch: int = 1, device: Optional[torch.device] = None):
        self.L = n_layers
        self.keep = sorted(set(keep))
        self.tern = [i for i in range(n_layers) if i not in set(self.keep)]
        self.g, self.batch = g, batch
        dev = device or torch.device("cuda")
        self.shapes = dict(shapes)
        self.codes, self.s16, self.w16, self.x, self.y = {}, {}, {}, {}, {}
        self._xt, self._xd, self._yt, self._yd = {}, {}, {}, {}
        for kind, (N, K) in self.shapes.items():
            T, D = len(self.tern), len(self.keep)
            self.codes[kind] = torch.empty((T, N, K // 4), dtype=torch.uint8, device=dev)
            self.s16[kind] = torch.empty((T, N, K // g), dtype=torch.float16, device=dev)
            self.w16[kind] = torch.empty((D, N, K), dtype=torch.float16, device=dev)
            tmp = torch.empty((N, K // g), dtype=torch.float32, device=dev)
            for t, layer in enumerate(self.tern):
                ops.ternarize_pack(weight(kind, layer).contiguous(), g, eps,
                                   codes=self.codes[kind][t], scales=tmp,
                                   scales_f16=self.s16[kind][t], want_zero_count=False)
            for d, layer in enumerate(self.keep):
                self.w16[kind][d].copy_(weight(kind, layer))   # float16 storage
            # token buffers grouped as the launches read them
            self._xt[kind] = torch.zeros((T, batch, K), dtype=torch.bfloat16, device=dev)
            self._xd[kind] = torch.zeros((D, batch, K), dtype=torch.bfloat16, device=dev)
            self._yt[kind] = torch.empty((T, batch, N), dtype=torch.float32, device=dev)
            self._yd[kind] = torch.empty((D, batch, N), dtype=torch.float32, device=dev)

    def set_inputs(self, kind: str, x: torch.Tensor) -> None:
        """x bf16 [L, B, K] in layer order -> the grouped input buffers."""
        if self.tern:
            self._xt[kind].copy_(x[self.tern])
        if self.keep:
            self._xd[kind].copy_(x[self.keep])

    def outputs(self, kind: str) -> torch.Tensor:
        """float32 [L, B, N] in layer order (gathered from the grouped buffers)."""
        N = self.shapes[kind][0]
        out = torch.empty((self.L, self.batch, N), dtype=torch.float32,
                          device=self._yt[kind].device)
        if self.tern:
            out[self.tern] = self._yt[kind]
        if self.keep:
            out[self.keep] = self._yd[kind]
        return out

    def token(self, kinds: Sequence[str] = ("in", "out"), arenas: Optional[dict] = None) -> None:
        """One decode token: every layer's projections of the given kinds.
        ``arenas`` (optional) replaces the weight arenas, e.g. copies used to
        keep the caches cold."""
        a = arenas or {}
        for kind in kinds:
            if self.tern:
                ops.tgemv(self._xt[kind], a.get(("codes", kind), self.codes[kind]),
                          a.get(("s16", kind), self.s16[kind]), self.g, y=self._yt[kind])
            if self.keep:
                ops.dgemv(self._xd[kind], a.get(("w16", kind), self.w16[kind]),
                          y=self._yd[kind])

    def arena_copy(self) -> dict:
        """Copies of all weight arenas (for cold-cache timing)."""
        out = {}
        for kind in self.shapes:
            out[("codes", kind)] = self.codes[kind].clone()
            out[("s16", kind)] = self.s16[kind].clone()
            out[("w16", kind)] = self.w16[kind].clone()
        return out

    def bytes_per_token(self, batch: Optional[int] = None) -> float:
        """Algorithmic bytes of one token: weights, scales, x and y."""
        B = self.batch if batch is None else batch
        total = 0.0
        for kind, (N, K) in self.shapes.items():
            total += len(self.tern) * (N * K / 4 + 2 * N * K / self.g)
            total += len(self.keep) * 2 * N * K
            total += self.L * (2 * B * K + 4 * B * N)
        return total


__all__ = ["keep_first_last", "quantize_projections", "DecodeStack", "PROJECTIONS"]
