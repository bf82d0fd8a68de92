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
* ``Mamba2Decoder``: decode in layer order through whole Mamba-2 blocks
  (pre-norm, in_proj, the FP16 mixer step of Sec. 3.2, out_proj), one token
  capturable as a HIP graph, or the whole stack in one launch (Sec. 8:
  small-batch decode).

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
    layer order, so a token is three launches: both kinds' ternary arenas in
    one (``tm_tgemv_pair``), then each kind's kept layers.  Inputs and outputs of a token
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
        cs = {k: (a.get(("codes", k), self.codes[k]), a.get(("s16", k), self.s16[k]))
              for k in kinds}
        pair = self.tern and len(kinds) == 2
        if pair:  # both kinds' ternary layers in one launch
            k0, k1 = kinds
            ops.tgemv_pair(self._xt[k0], *cs[k0], self._xt[k1], *cs[k1], self.g,
                           y0=self._yt[k0], y1=self._yt[k1])
        for kind in kinds:
            if self.tern and not pair:
                ops.tgemv(self._xt[kind], *cs[kind], self.g, y=self._yt[kind])
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


MAX_KEPT_STACK = 64  # kept layers the one-launch decode takes


def stack_fits(B: int, d_model: int, nheads: int, g: int) -> bool:
    """Whether tm_mamba2_decode_token takes this stack (its declaration's
    limits; nheads must also not exceed the device's CU count)."""
    d_inner = nheads * ops.MIXER_HEADDIM
    shapes = (1 <= B <= 4 and g in (64, 128, 256) and 64 <= d_model <= 4096
              and d_model % 64 == 0 and d_model % g == 0 and d_inner % g == 0
              and 1 <= nheads <= 128 and (B == 1 or (d_model <= 2048 and d_inner <= 4096)))
    return (shapes and torch.cuda.is_available()
            and nheads * B <= torch.cuda.get_device_properties(
                torch.cuda.current_device()).multi_processor_count)


def rms_fused_fits(B: int, K: int, g: int) -> bool:
    """Whether tm_tgemv_rms takes B rows of K columns at group size g (the
    rule its declaration states: one workgroup stages all rows at once)."""
    H = 128 // g if g < 128 else 1
    pieces = (K + 127) // 128 * 8
    waves = 8 if (K + 511) // 512 >= 8 else 4
    return 4 * B * H <= 16 and B * pieces <= 2 * 64 * waves


class Mamba2Decoder:
    """Batch-B decode through L Mamba-2 blocks in layer order, every step on
    the library's kernels.  Fused (the default where the shapes allow it),
    three launches per layer:

        zx  = in_proj(rmsnorm(residual) * w_pre[l])       tm_tgemv_rms / tm_dgemv_rms
        g   = mixer step up to the gate (conv, FP16 SSM)  tm_mixer_gate
        residual += out_proj(rmsnorm(g) * norm_w[l])      tm_tgemv_rms / tm_dgemv_rms

    or unfused, five (each normalization its own launch):

        x   = rmsnorm(residual += y_prev) * w_pre[l]      tm_residual_rmsnorm
        zx  = in_proj(x)                                  tm_tgemv / tm_dgemv (kept)
        m   = mixer step (conv, FP16 SSM, gated norm)     tm_mixer_step
        y   = out_proj(m)                                 tm_tgemv / tm_dgemv (kept)

    After the last layer the final norm of the residual gives ``x_out`` (the
    lm head is outside).  All launches go to the current stream with fixed
    buffers, so a token can be captured once as a HIP graph (``capture``) and
    replayed.

    or the whole stack in one launch (``tm_mamba2_decode_token``: the three
    phases of every block separated by grid barriers instead of launches;
    batch 1 .. 4, kept blocks included).

    weight(kind, l) -> float32 [N, K] master weights (kind "in": [Z, d_model],
    "out": [d_model, d_inner]); mixer(l) -> dict of float32 arrays conv_w,
    conv_b, dt_bias, A_log, D, norm_w (see ops.mixer_step); pre_norm(l) ->
    float32 [d_model].  Layers in ``keep`` stay in float16 (Sec. 7).
    fused: None picks the fused form whenever every projection's shape
    allows it (batch up to 4 at g >= 128 for the Mamba-2 1.3B shapes).
    stack: None picks the one-launch form whenever it applies (at most
    ``MAX_KEPT_STACK`` kept layers, ``stack_fits``); it keeps the residual in
    its own workspace (``residual`` is not updated).
    The packed weights, mixer parameters and states of all layers live in
    layer-stacked arrays (``arena``); each layer's entries are views of them,
    so every form reads and advances the same states.
    """

    def __init__(self, weight: Callable[[str, int], torch.Tensor], mixer: Callable[[int], dict],
                 pre_norm: Callable[[int], torch.Tensor], n_layers: int, d_model: int,
                 nheads: int, keep: Iterable[int] = (), g: int = 128, eps: float = 1e-5,
                 batch: int = 1, device: Optional[torch.device] = None,
                 fused: Optional[bool] = None, stack: Optional[bool] = None):
        dev = device or torch.device("cuda")
        self.L, self.B, self.g, self.eps = n_layers, batch, g, eps
        self.keep = set(keep)
        self.d_model, self.nheads = d_model, nheads
        P, N = ops.MIXER_HEADDIM, ops.MIXER_DSTATE
        self.d_inner = nheads * P
        self.Z = 2 * self.d_inner + 2 * N + nheads
        conv_dim = self.d_inner + 2 * N
        if self.keep and not (1 <= batch <= 8 and
                              batch * max(d_model, self.d_inner) <= 16384):
            raise ValueError(f"blocks kept in FP16 decode at batch 1 .. 8 with batch x K "
                             f"<= 16384 (tm_dgemv); got batch {batch}")
        fits = all(rms_fused_fits(batch, k, g) if l not in self.keep else batch * k <= 16384
                   for l in range(n_layers) for k in (d_model, self.d_inner))
        if fused and not fits:
            raise ValueError(f"batch {batch} does not fit the fused decode at g = {g}")
        self.fused = fits if fused is None else bool(fused)
        st_ok = stack_fits(batch, d_model, nheads, g) and len(self.keep) <= MAX_KEPT_STACK
        if stack and not st_ok:
            raise ValueError(f"the one-launch stack decode needs at most {MAX_KEPT_STACK} "
                             f"kept layers and shapes stack_fits accepts")
        self.stack = st_ok if stack is None else bool(stack)
        L, f32, f16 = n_layers, torch.float32, torch.float16
        ar = {"pre_w": torch.empty((L, d_model), dtype=f32, device=dev),
              "conv_w": torch.empty((L, conv_dim, 4), dtype=f32, device=dev),
              "conv_b": torch.empty((L, conv_dim), dtype=f32, device=dev),
              "dt_bias": torch.empty((L, nheads), dtype=f32, device=dev),
              "A_log": torch.empty((L, nheads), dtype=f32, device=dev),
              "D": torch.empty((L, nheads), dtype=f32, device=dev),
              "norm_w": torch.empty((L, self.d_inner), dtype=f32, device=dev),
              "conv_state": torch.zeros((L, batch, conv_dim, 4), dtype=f16, device=dev),
              "conv_pos": torch.zeros((L,), dtype=torch.int32, device=dev),
              "ssm_state": torch.zeros((L, batch, nheads, P, N), dtype=f16, device=dev)}
        # packed weights of every layer (a kept layer's entries stay zero and
        # unread), and the float16 projections of the kept layers, in order
        ar["in_codes"] = torch.zeros((L, self.Z, d_model // 4), dtype=torch.uint8, device=dev)
        ar["in_scales"] = torch.zeros((L, self.Z, d_model // g), dtype=f16, device=dev)
        ar["out_codes"] = torch.zeros((L, d_model, self.d_inner // 4), dtype=torch.uint8,
                                      device=dev)
        ar["out_scales"] = torch.zeros((L, d_model, self.d_inner // g), dtype=f16, device=dev)
        self.kept = sorted(self.keep)
        nk = len(self.kept)
        ar["in_w16"] = torch.empty((nk, self.Z, d_model), dtype=f16, device=dev)
        ar["out_w16"] = torch.empty((nk, d_model, self.d_inner), dtype=f16, device=dev)
        self.arena = ar
        self.layers = []
        for l in range(n_layers):
            lay = {}
            for kind, (n, k) in (("in", (self.Z, d_model)), ("out", (d_model, self.d_inner))):
                w = weight(kind, l).contiguous()
                if tuple(w.shape) != (n, k):
                    raise ValueError(f"layer {l} {kind}_proj has shape {tuple(w.shape)}")
                if l in self.keep:
                    d = self.kept.index(l)
                    w16 = ar[f"{kind}_w16"][d:d + 1]
                    w16.copy_(w.to(torch.float16)[None])
                    lay[kind] = ("dense", w16)
                else:
                    codes = ar[f"{kind}_codes"][l:l + 1]
                    s16 = ar[f"{kind}_scales"][l:l + 1]
                    ops.ternarize_pack(w, g, eps, codes=codes[0], scales_f16=s16[0],
                                       want_zero_count=False)
                    lay[kind] = ("ternary", codes, s16)
            prm = mixer(l)
            lay["mixer"] = {}
            for k, v in prm.items():
                v = v if isinstance(v, torch.Tensor) else torch.from_numpy(v)
                ar[k][l].copy_(v.to(dev, torch.float32).reshape(ar[k][l].shape))
                lay["mixer"][k] = ar[k][l]
            ar["pre_w"][l].copy_(pre_norm(l).to(dev, torch.float32))
            lay["pre"] = ar["pre_w"][l]
            lay["conv"] = ar["conv_state"][l]
            lay["pos"] = ar["conv_pos"][l:l + 1]
            lay["ssm"] = ar["ssm_state"][l]
            self.layers.append(lay)
        self.final_norm = torch.ones((d_model,), dtype=torch.float32, device=dev)
        # token buffers (reused by every layer: the layers run one after another)
        self.emb = torch.zeros((batch, d_model), dtype=torch.float32, device=dev)
        self.residual = torch.zeros((batch, d_model), dtype=torch.float32, device=dev)
        self.x = torch.empty((1, batch, d_model), dtype=torch.bfloat16, device=dev)
        self.zx = torch.empty((1, batch, self.Z), dtype=torch.float32, device=dev)
        self.m = torch.empty((1, batch, self.d_inner), dtype=torch.bfloat16, device=dev)
        self.y = torch.empty((1, batch, d_model), dtype=torch.float32, device=dev)
        self.gated = torch.empty((batch, self.d_inner), dtype=torch.float32, device=dev)
        self.ws = ops.mixer_workspace(batch, nheads, dev)
        self.x_out = torch.empty((batch, d_model), dtype=torch.bfloat16, device=dev)
        self.arena["final_w"] = self.final_norm
        self.stack_ws = (ops.mamba2_decode_workspace(d_model, nheads, dev, batch)
                         if self.stack else None)
        self.graph = None

    def set_states(self, l: int, conv: torch.Tensor, ssm: torch.Tensor, pos: int = 0) -> None:
        """Layer l's convolution ring (float16 [B, conv_dim, 4], slot (pos + j) % 4
        the j-th oldest) and SSM state (float16 [B, nheads, 64, 128])."""
        lay = self.layers[l]
        lay["conv"].copy_(conv)
        lay["ssm"].copy_(ssm)
        lay["pos"].fill_(pos)

    def _proj(self, lay, kind, x, y) -> None:
        p = lay[kind]
        if p[0] == "dense":
            ops.dgemv(x, p[1], y=y)
        else:
            ops.tgemv(x, p[1], p[2], self.g, y=y)

    def _proj_rms(self, lay, kind, src, norm_w, y, accumulate) -> None:
        p = lay[kind]
        if p[0] == "dense":
            ops.dgemv_rms(src, p[1][0], norm_w, self.eps, y=y, accumulate=accumulate)
        else:
            ops.tgemv_rms(src, p[1][0], p[2][0], self.g, norm_w, self.eps, y=y,
                          accumulate=accumulate)

    def layer_step(self, l: int) -> None:
        """Layer l of a token.  Fused: in_proj of the normalized residual,
        the mixer up to the gate, out_proj of the normalized gate added into
        the residual.  Unfused: pre-norm (taking the previous layer's output
        into the residual), in_proj, mixer step, out_proj into ``y``."""
        lay = self.layers[l]
        if l == 0:
            self.residual.copy_(self.emb)
        mp = lay["mixer"]
        if self.fused:
            self._proj_rms(lay, "in", self.residual, lay["pre"], self.zx[0], False)
            ops.mixer_gate(self.zx[0], lay["conv"], lay["pos"], lay["ssm"], mp["conv_w"],
                           mp["conv_b"], mp["dt_bias"], mp["A_log"], mp["D"], gated=self.gated)
            self._proj_rms(lay, "out", self.gated, mp["norm_w"], self.residual, True)
            return
        ops.residual_rmsnorm(self.residual, None if l == 0 else self.y[0], lay["pre"], self.eps,
                             x=self.x[0])
        self._proj(lay, "in", self.x, self.zx)
        ops.mixer_step(self.zx[0], lay["conv"], lay["pos"], lay["ssm"], mp["conv_w"],
                       mp["conv_b"], mp["dt_bias"], mp["A_log"], mp["D"], mp["norm_w"], self.eps,
                       workspace=self.ws, out=self.m[0])
        self._proj(lay, "out", self.m, self.y)

    def token_stack(self) -> torch.Tensor:
        """One token per batch row through every block in a single launch."""
        a = {k: self.arena[k] for k in ops.STACK_FIELDS}
        ops.mamba2_decode_token(a, self.g, self.eps, self.emb, x_out=self.x_out,
                                workspace=self.stack_ws, kept=self.kept,
                                in_w16=self.arena["in_w16"], out_w16=self.arena["out_w16"])
        return self.x_out

    def token(self) -> torch.Tensor:
        """One decode token from ``emb`` (float32 [B, d_model]) through every
        layer; returns ``x_out`` = final norm of the residual (bfloat16)."""
        if self.stack:
            return self.token_stack()
        for l in range(self.L):
            self.layer_step(l)
        ops.residual_rmsnorm(self.residual, None if self.fused else self.y[0], self.final_norm,
                             self.eps, x=self.x_out)
        return self.x_out

    def capture(self) -> None:
        """Record one token (all layers) as a HIP graph on a side stream."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(self.graph, stream=side):
                self.token()
        torch.cuda.current_stream().wait_stream(side)

    def replay(self) -> torch.Tensor:
        if self.graph is None:
            raise RuntimeError("capture() first")
        self.graph.replay()
        return self.x_out

    def launches_per_token(self) -> int:
        # one launch (and the clear of its barrier counter); else per layer:
        # in_proj, mixer, out_proj (fused) or pre-norm, in_proj, mixer (2),
        # out_proj; then the residual copy and the final norm
        if self.stack:
            return 2
        return (3 if self.fused else 5) * self.L + 2

    def bytes_per_token(self) -> float:
        """Algorithmic HBM bytes of one token: packed or float16 projection
        weights, both SSM/conv state passes (read + write), mixer parameters
        and the activations, per batch of B tokens."""
        total = 0.0
        P, N = ops.MIXER_HEADDIM, ops.MIXER_DSTATE
        for l, lay in enumerate(self.layers):
            for kind in ("in", "out"):
                p = lay[kind]
                total += p[1].numel() * p[1].element_size()
                if p[0] == "ternary":
                    total += p[2].numel() * 2
            total += 2 * self.B * self.nheads * P * N * 2          # SSM state read + write
            total += self.B * (self.d_inner + 2 * N) * 4 * 2       # conv ring read, new slot
            total += sum(v.numel() * 4 for v in lay["mixer"].values()) + self.d_model * 4
            total += self.B * (4 * self.Z + 2 * self.Z + 4 * self.d_inner + 2 * self.d_inner
                               + 12 * self.d_model)                # activations, roughly
        return total


__all__ += ["Mamba2Decoder", "rms_fused_fits", "stack_fits"]
