"""Thin ctypes binding of ``libtmamba.so`` (declared in ``include/tmamba.h``).

Argument marshalling only: every function checks the dtype, device,
contiguity and exact shape of every tensor it is given (inputs and
caller-supplied outputs: the C ABI sees only pointers, so a wrong size here
would become an out-of-bounds access on the device), allocates missing
outputs with torch (the library itself allocates nothing), and passes raw
device pointers plus the current HIP stream to the C ABI.  All arithmetic
runs in the library's HIP kernels.  There is no fallback: if the library is missing, every call raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtmamba.so")
_lib = None

TM_STATUS = {0: "TM_OK", 1: "TM_EINVAL", 2: "TM_ESHAPE", 3: "TM_EALIGN", 4: "TM_EHIP",
             5: "TM_ENOTIMPL"}

# exported symbol -> (restype, argtypes)
_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
class Mamba2Stack(ctypes.Structure):
    """``tm_mamba2_stack``: the device arrays of a stack of ternary Mamba-2
    blocks for whole-stack decoding (layer-stacked, see include/tmamba.h)."""
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("nheads", ctypes.c_int32), ("g", ctypes.c_int32), ("eps", ctypes.c_float),
                ("in_codes", ctypes.c_void_p), ("in_scales", ctypes.c_void_p),
                ("out_codes", ctypes.c_void_p), ("out_scales", ctypes.c_void_p),
                ("pre_w", ctypes.c_void_p), ("conv_w", ctypes.c_void_p),
                ("conv_b", ctypes.c_void_p), ("dt_bias", ctypes.c_void_p),
                ("A_log", ctypes.c_void_p), ("D", ctypes.c_void_p), ("norm_w", ctypes.c_void_p),
                ("final_w", ctypes.c_void_p), ("conv_state", ctypes.c_void_p),
                ("conv_pos", ctypes.c_void_p), ("ssm_state", ctypes.c_void_p),
                ("n_kept", ctypes.c_int32), ("kept", ctypes.POINTER(ctypes.c_int32)),
                ("in_w16", ctypes.c_void_p), ("out_w16", ctypes.c_void_p),
                ("batch", ctypes.c_int32)]


SIGNATURES = {
    "tm_abi_version": (ctypes.c_int, []),
    "tm_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "tm_ternarize_pack": (ctypes.c_int, [_P, _I64, _I64, _I32, ctypes.c_float, _P, _P, _P, _P, _P]),
    "tm_tgemm_fwd": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I64, _I32, _P, _P]),
    "tm_tgemm_fwd_ws": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I64, _I32, _P, _P, _I64, _P]),
    "tm_tgemm_fwd_workspace": (ctypes.c_int64, []),
    "tm_tgemm_bwd_dx": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I64, _I32, _P, _P]),
    "tm_tgemm_bwd_dx_f16": (ctypes.c_int,
                            [_P, _P, _P, _I64, _I64, _I64, _I32, _P, _P, _I64, _P]),
    "tm_tgemm_bwd_dx_f16_workspace": (ctypes.c_int64, [_I64, _I64]),
    "tm_tgemm_bwd_dw_ste": (ctypes.c_int, [_P, _P, _I64, _I64, _I64, _P, _I32, _P]),
    "tm_tgemv": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _I64, _I64, _I32, _P, _P]),
    "tm_tgemv_pair": (ctypes.c_int, [_P, _P, _P, _I32, _I64, _I64, _P, _P, _P, _P, _I32, _I64,
                                     _I64, _P, _I32, _I32, _P]),
    "tm_ternarize_pack_thresh": (ctypes.c_int,
                                 [_P, _I64, _I64, _I32, ctypes.c_float, _P, _P, _P, _P, _P, _P]),
    "tm_group_code_dot": (ctypes.c_int, [_P, _P, _I64, _I64, _I32, _P, _P]),
    "tm_ternarize_codes": (ctypes.c_int, [_P, _I64, _I64, _I32, ctypes.c_float, _P, _P, _P, _P]),
    "tm_tgemm_fwd_bf16": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _I64, _I32, _P, _P]),
    "tm_dgemv": (ctypes.c_int, [_P, _P, _I32, _I32, _I64, _I64, _P, _P]),
    "tm_residual_rmsnorm": (ctypes.c_int, [_P, _P, _I32, _I64, _P, ctypes.c_float, _P, _P]),
    "tm_mixer_step_noalloc": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                             _P, _P, _P, ctypes.c_float, _P, _P]),
    "tm_mixer_step": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P,
                                     _P, ctypes.c_float, _P, _P, _P]),
    "tm_scale_ste_grad": (ctypes.c_int,
                          [_P, _P, _P, _P, _I64, _I64, _I32, ctypes.c_float, _P, _P, _P]),
    "tm_tgemv_rms": (ctypes.c_int, [_P, _P, ctypes.c_float, _P, _P, _I32, _I64, _I64, _I32, _P,
                                    _I32, _P]),
    "tm_dgemv_rms": (ctypes.c_int, [_P, _P, ctypes.c_float, _P, _I32, _I64, _I64, _P, _I32, _P]),
    "tm_mixer_gate": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P,
                                     _P, _P]),
    "tm_mamba2_decode_token": (ctypes.c_int, [ctypes.POINTER(Mamba2Stack), _P, _P, _P, _I64, _P]),
    "tm_mamba2_decode_workspace": (ctypes.c_int64, [_I32, _I32, _I32]),
}


class TernaryError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = lib().tm_status_str(status).decode() if status in TM_STATUS else "unknown"
        super().__init__(f"{fn} failed: {msg}")


def lib_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load the HIP library once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(
                f"{_LIB_PATH} is missing: build it with `python -m paper_2606_18114_amd.build` "
                "(or __graft_entry__.build()); there is no fallback implementation")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise TernaryError(fn, status)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtypes, ndim: int) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on the GPU (got {t.device})")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims (got shape {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shape(t: torch.Tensor, name: str, shape, device: torch.device) -> None:
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the other operands on {device}")


def _groups(K: int, g: int) -> int:
    """K / g for the shape checks; a K that g does not divide is left to the
    library, which rejects it (TM_ESHAPE) before launching anything."""
    return K // g if g > 0 and K % g == 0 else max(K // max(g, 1), 1)


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)
_U8 = (torch.uint8,)
_F32 = (torch.float32,)
_F16 = (torch.float16, torch.int16, torch.uint16)
_INT64 = (torch.int64,)


def ternarize_pack(W: torch.Tensor, g: int = 128, eps: float = 1e-5, *,
                   codes: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None,
                   scales_f16: Optional[torch.Tensor] = None,
                   zero_count: Optional[torch.Tensor] = None, want_f16: bool = True,
                   want_zero_count: bool = True, row_mult: Optional[torch.Tensor] = None):
    """W float32 [N, K] -> (codes uint8 [N, K/4], scales f32 [N, K/g],
    scales_f16 float16 [N, K/g] or None, zero_count int64 [1] or None).

    row_mult (float32 [N], optional) multiplies each row's rounding threshold
    (``tm_ternarize_pack_thresh``); the stored scales stay the absmean."""
    _need(W, "W", _F32, 2)
    N, K = W.shape
    dev = W.device
    G = _groups(K, g)
    if row_mult is not None:
        _need(row_mult, "row_mult", _F32, 1)
        _shape(row_mult, "row_mult", (N,), dev)
    if codes is None:
        codes = torch.empty((N, K // 4), dtype=torch.uint8, device=dev)
    _need(codes, "codes", _U8, 2)
    _shape(codes, "codes", (N, K // 4), dev)
    if scales is None:
        scales = torch.empty((N, G), dtype=torch.float32, device=dev)
    _need(scales, "scales", _F32, 2)
    _shape(scales, "scales", (N, G), dev)
    if scales_f16 is None and want_f16:
        scales_f16 = torch.empty((N, G), dtype=torch.float16, device=dev)
    if scales_f16 is not None:
        _need(scales_f16, "scales_f16", _F16, 2)
        _shape(scales_f16, "scales_f16", (N, G), dev)
    if zero_count is None and want_zero_count:
        zero_count = torch.empty((1,), dtype=torch.int64, device=dev)
    if zero_count is not None:
        _need(zero_count, "zero_count", _INT64, 1)
        _shape(zero_count, "zero_count", (1,), dev)
    if row_mult is None:
        st = lib().tm_ternarize_pack(_ptr(W), N, K, g, eps, _ptr(codes), _ptr(scales),
                                     _ptr(scales_f16), _ptr(zero_count), _stream())
        _check("tm_ternarize_pack", st)
    else:
        st = lib().tm_ternarize_pack_thresh(_ptr(W), N, K, g, eps, _ptr(row_mult), _ptr(codes),
                                            _ptr(scales), _ptr(scales_f16), _ptr(zero_count),
                                            _stream())
        _check("tm_ternarize_pack_thresh", st)
    return codes, scales, scales_f16, zero_count


def ternarize_codes(W: torch.Tensor, tau: torch.Tensor, g: int = 128, eps: float = 1e-5, *,
                    codes: Optional[torch.Tensor] = None,
                    zero_count: Optional[torch.Tensor] = None, want_zero_count: bool = True):
    """Codes of W against the given per-group thresholds tau float32 [N, K/g]
    -> (codes uint8 [N, K/4], zero_count int64 [1] or None)."""
    _need(W, "W", _F32, 2)
    _need(tau, "tau", _F32, 2)
    N, K = W.shape
    _shape(tau, "tau", (N, _groups(K, g)), W.device)
    if codes is None:
        codes = torch.empty((N, K // 4), dtype=torch.uint8, device=W.device)
    _need(codes, "codes", _U8, 2)
    _shape(codes, "codes", (N, K // 4), W.device)
    if zero_count is None and want_zero_count:
        zero_count = torch.empty((1,), dtype=torch.int64, device=W.device)
    if zero_count is not None:
        _need(zero_count, "zero_count", _INT64, 1)
        _shape(zero_count, "zero_count", (1,), W.device)
    st = lib().tm_ternarize_codes(_ptr(W), N, K, g, eps, _ptr(tau), _ptr(codes),
                                  _ptr(zero_count), _stream())
    _check("tm_ternarize_codes", st)
    return codes, zero_count


def group_code_dot(codes: torch.Tensor, dW: torch.Tensor, g: int = 128,
                   out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """out[n, j] = sum over group j of row n of q * dW (float32 [N, K/g]): the
    gradient of a per-group magnitude that multiplies the codes."""
    _need(codes, "codes", _U8, 2)
    _need(dW, "dW", _F32, 2)
    N, K = dW.shape
    _shape(codes, "codes", (N, K // 4), dW.device)
    if out is None:
        out = torch.empty((N, _groups(K, g)), dtype=torch.float32, device=dW.device)
    _need(out, "out", _F32, 2)
    _shape(out, "out", (N, _groups(K, g)), dW.device)
    st = lib().tm_group_code_dot(_ptr(codes), _ptr(dW), N, K, g, _ptr(out), _stream())
    _check("tm_group_code_dot", st)
    return out


def scale_ste_grad(W: torch.Tensor, codes: torch.Tensor, scale: torch.Tensor,
                   dWhat: torch.Tensor, g: int = 128, eps: float = 1e-5, *,
                   ds: Optional[torch.Tensor] = None, dW: Optional[torch.Tensor] = None,
                   want_dW: bool = True, in_place: bool = False):
    """Learnable-scale gradients with the rounding straight-through:
    (ds float32 [N, K/g], dW float32 [N, K] or None).  in_place=True writes
    dW over dWhat."""
    _need(W, "W", _F32, 2)
    _need(codes, "codes", _U8, 2)
    _need(scale, "scale", _F32, 2)
    _need(dWhat, "dWhat", _F32, 2)
    N, K = W.shape
    G = _groups(K, g)
    _shape(codes, "codes", (N, K // 4), W.device)
    _shape(scale, "scale", (N, G), W.device)
    _shape(dWhat, "dWhat", (N, K), W.device)
    if ds is None:
        ds = torch.empty((N, G), dtype=torch.float32, device=W.device)
    _need(ds, "ds", _F32, 2)
    _shape(ds, "ds", (N, G), W.device)
    if in_place:
        dW = dWhat
    elif dW is None and want_dW:
        dW = torch.empty((N, K), dtype=torch.float32, device=W.device)
    if dW is not None:
        _need(dW, "dW", _F32, 2)
        _shape(dW, "dW", (N, K), W.device)
    st = lib().tm_scale_ste_grad(_ptr(W), _ptr(codes), _ptr(scale), _ptr(dWhat), N, K, g, eps,
                                 _ptr(ds), _ptr(dW), _stream())
    _check("tm_scale_ste_grad", st)
    return ds, dW


def tgemm_fwd(X: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor, g: int = 128,
              Y: Optional[torch.Tensor] = None,
              out_dtype: torch.dtype = torch.float32, *,
              workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Y[M, N] = X . (q * s)^T in float32 (``tm_tgemm_fwd_ws``: the two parts of
    a cut tile meet through a small workspace, uint8 of at least
    ``fwd_workspace_bytes()`` bytes; when not given, one kept per stream), or
    rounded once to bfloat16 (out_dtype=torch.bfloat16,
    ``tm_tgemm_fwd_bf16``)."""
    _need(X, "X", _BF16, 2)
    _need(codes, "codes", _U8, 2)
    _need(scales, "scales", _F32, 2)
    if out_dtype not in (torch.float32, torch.bfloat16):
        raise TypeError(f"out_dtype must be float32 or bfloat16 (got {out_dtype})")
    M, K = X.shape
    N = codes.shape[0]
    _shape(codes, "codes", (N, K // 4), X.device)
    _shape(scales, "scales", (N, _groups(K, g)), X.device)
    if Y is None:
        Y = torch.empty((M, N), dtype=out_dtype, device=X.device)
    _need(Y, "Y", _BF16 if out_dtype == torch.bfloat16 else _F32, 2)
    _shape(Y, "Y", (M, N), X.device)
    if out_dtype == torch.bfloat16:
        st = lib().tm_tgemm_fwd_bf16(_ptr(X), _ptr(codes), _ptr(scales), M, N, K, g, _ptr(Y),
                                     _stream())
        _check("tm_tgemm_fwd_bf16", st)
    else:
        need = fwd_workspace_bytes()
        stream = _stream()
        if workspace is None:
            workspace = _stream_workspace(X.device, stream, need)
        _need(workspace, "workspace", _U8, 1)
        if workspace.numel() < need:
            raise ValueError(f"workspace has {workspace.numel()} bytes, {need} needed")
        if workspace.device != X.device:
            raise ValueError(f"workspace is on {workspace.device}, the operands on {X.device}")
        st = lib().tm_tgemm_fwd_ws(_ptr(X), _ptr(codes), _ptr(scales), M, N, K, g, _ptr(Y),
                                   _ptr(workspace), workspace.numel(), stream)
        _check("tm_tgemm_fwd_ws", st)
    return Y


_STREAM_WS: dict = {}


def _stream_workspace(device: torch.device, stream: int, nbytes: int) -> torch.Tensor:
    """A small scratch buffer kept per (device, stream): calls on one stream
    run in order, so they may share it (calls on different streams get
    their own)."""
    key = (device.index, stream)
    ws = _STREAM_WS.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = _STREAM_WS[key] = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws


_FWD_WS_BYTES: list = []


def fwd_workspace_bytes() -> int:
    """Workspace bytes of ``tm_tgemm_fwd_ws`` (a constant of the library)."""
    if not _FWD_WS_BYTES:
        _FWD_WS_BYTES.append(int(lib().tm_tgemm_fwd_workspace()))
    return _FWD_WS_BYTES[0]


def tgemm_bwd_dx(dY: torch.Tensor, codes: torch.Tensor, scales: torch.Tensor, g: int = 128,
                 dX: Optional[torch.Tensor] = None, *, precision: str = "f16",
                 workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """dX[M, K] = dY . (q * s) in float32.

    precision "f16" (``tm_tgemm_bwd_dx_f16``): one float16 pass, each
    dequantized weight within 2^-11 relative; the workspace (uint8, at least
    ``dx_f16_workspace_bytes(M, N)`` bytes) is allocated here when not given.
    precision "exact" (``tm_tgemm_bwd_dx``): two bfloat16 passes carrying 16
    bits of every scale."""
    _need(dY, "dY", _BF16, 2)
    _need(codes, "codes", _U8, 2)
    _need(scales, "scales", _F32, 2)
    M, N = dY.shape
    K = codes.shape[1] * 4
    _shape(codes, "codes", (N, K // 4), dY.device)
    _shape(scales, "scales", (N, _groups(K, g)), dY.device)
    if dX is None:
        dX = torch.empty((M, K), dtype=torch.float32, device=dY.device)
    _need(dX, "dX", _F32, 2)
    _shape(dX, "dX", (M, K), dY.device)
    if precision == "exact":
        st = lib().tm_tgemm_bwd_dx(_ptr(dY), _ptr(codes), _ptr(scales), M, N, K, g, _ptr(dX),
                                   _stream())
        _check("tm_tgemm_bwd_dx", st)
        return dX
    if precision != "f16":
        raise ValueError(f"precision must be 'f16' or 'exact' (got {precision!r})")
    need = dx_f16_workspace_bytes(M, N)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dY.device)
    _need(workspace, "workspace", _U8, 1)
    if workspace.numel() < need:
        raise ValueError(f"workspace has {workspace.numel()} bytes, {need} needed")
    if workspace.device != dY.device:
        raise ValueError(f"workspace is on {workspace.device}, the operands on {dY.device}")
    st = lib().tm_tgemm_bwd_dx_f16(_ptr(dY), _ptr(codes), _ptr(scales), M, N, K, g, _ptr(dX),
                                   _ptr(workspace), workspace.numel(), _stream())
    _check("tm_tgemm_bwd_dx_f16", st)
    return dX


def dx_f16_workspace_bytes(M: int, N: int) -> int:
    """Workspace bytes of the float16 dX call for an M x N gradient."""
    n = int(lib().tm_tgemm_bwd_dx_f16_workspace(M, N))
    if n < 0:
        raise ValueError(f"no workspace size for M={M}, N={N}")
    return n


def tgemm_bwd_dw_ste(dY: torch.Tensor, X: torch.Tensor, dW: Optional[torch.Tensor] = None,
                     accumulate: bool = False) -> torch.Tensor:
    """dW[N, K] (+)= dY^T . X in float32 (identity straight-through estimator)."""
    _need(dY, "dY", _BF16, 2)
    _need(X, "X", _BF16, 2)
    M, N = dY.shape
    K = X.shape[1]
    _shape(X, "X", (M, K), dY.device)
    if dW is None:
        if accumulate:
            raise ValueError("accumulate=True needs an existing dW")
        dW = torch.empty((N, K), dtype=torch.float32, device=dY.device)
    _need(dW, "dW", _F32, 2)
    _shape(dW, "dW", (N, K), dY.device)
    st = lib().tm_tgemm_bwd_dw_ste(_ptr(dY), _ptr(X), M, N, K, _ptr(dW), int(accumulate),
                                   _stream())
    _check("tm_tgemm_bwd_dw_ste", st)
    return dW


def tgemv(x: torch.Tensor, codes: torch.Tensor, scales_f16: torch.Tensor, g: int = 128,
          y: Optional[torch.Tensor] = None) -> torch.Tensor:
    """x bf16 [count, B, K], codes uint8 [count, N, K/4], scales_f16 [count, N, K/g]
    -> y float32 [count, B, N]."""
    _need(x, "x", _BF16, 3)
    _need(codes, "codes", _U8, 3)
    _need(scales_f16, "scales_f16", _F16, 3)
    count, B, K = x.shape
    N = codes.shape[1]
    _shape(codes, "codes", (count, N, K // 4), x.device)
    _shape(scales_f16, "scales_f16", (count, N, _groups(K, g)), x.device)
    if y is None:
        y = torch.empty((count, B, N), dtype=torch.float32, device=x.device)
    _need(y, "y", _F32, 3)
    _shape(y, "y", (count, B, N), x.device)
    st = lib().tm_tgemv(_ptr(x), _ptr(codes), _ptr(scales_f16), count, B, N, K, g, _ptr(y),
                        _stream())
    _check("tm_tgemv", st)
    return y


def _gemv_stack(x, codes, scales_f16, g, y, tag):
    _need(x, f"x{tag}", _BF16, 3)
    _need(codes, f"codes{tag}", _U8, 3)
    _need(scales_f16, f"scales{tag}", _F16, 3)
    count, B, K = x.shape
    N = codes.shape[1]
    _shape(codes, f"codes{tag}", (count, N, K // 4), x.device)
    _shape(scales_f16, f"scales{tag}", (count, N, _groups(K, g)), x.device)
    if y is None:
        y = torch.empty((count, B, N), dtype=torch.float32, device=x.device)
    _need(y, f"y{tag}", _F32, 3)
    _shape(y, f"y{tag}", (count, B, N), x.device)
    return count, B, N, K, y


def tgemv_pair(x0: torch.Tensor, codes0: torch.Tensor, scales0: torch.Tensor,
               x1: torch.Tensor, codes1: torch.Tensor, scales1: torch.Tensor, g: int = 128,
               y0: Optional[torch.Tensor] = None, y1: Optional[torch.Tensor] = None):
    """Two strided stacks of ``tgemv`` in one launch (``tm_tgemv_pair``), e.g. a
    decode token's in_proj and out_proj layers; returns (y0, y1)."""
    c0, B, N0, K0, y0 = _gemv_stack(x0, codes0, scales0, g, y0, "0")
    c1, B1, N1, K1, y1 = _gemv_stack(x1, codes1, scales1, g, y1, "1")
    if B1 != B:
        raise ValueError(f"the stacks have batches {B} and {B1}; tm_tgemv_pair needs one")
    if x1.device != x0.device:
        raise ValueError("the two stacks live on different devices")
    st = lib().tm_tgemv_pair(_ptr(x0), _ptr(codes0), _ptr(scales0), c0, N0, K0, _ptr(y0),
                             _ptr(x1), _ptr(codes1), _ptr(scales1), c1, N1, K1, _ptr(y1), B, g,
                             _stream())
    _check("tm_tgemv_pair", st)
    return y0, y1


def dgemv(x: torch.Tensor, W16: torch.Tensor, y: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Dense decode product of layers kept in FP16: x bf16 [count, B, K],
    W16 float16 [count, N, K] -> y float32 [count, B, N]."""
    _need(x, "x", _BF16, 3)
    _need(W16, "W16", _F16, 3)
    count, B, K = x.shape
    N = W16.shape[1]
    _shape(W16, "W16", (count, N, K), x.device)
    if y is None:
        y = torch.empty((count, B, N), dtype=torch.float32, device=x.device)
    _need(y, "y", _F32, 3)
    _shape(y, "y", (count, B, N), x.device)
    st = lib().tm_dgemv(_ptr(x), _ptr(W16), count, B, N, K, _ptr(y), _stream())
    _check("tm_dgemv", st)
    return y


def _rms_args(src, norm_w, y, N):
    _need(src, "src", _F32, 2)
    B, K = src.shape
    _need(norm_w, "norm_w", _F32, 1)
    _shape(norm_w, "norm_w", (K,), src.device)
    if y is None:
        y = torch.empty((B, N), dtype=torch.float32, device=src.device)
    _need(y, "y", _F32, 2)
    _shape(y, "y", (B, N), src.device)
    return B, K, y


def tgemv_rms(src: torch.Tensor, codes: torch.Tensor, scales_f16: torch.Tensor, g: int,
              norm_w: torch.Tensor, eps: float = 1e-5, y: Optional[torch.Tensor] = None,
              accumulate: bool = False) -> torch.Tensor:
    """Fused decode projection (tm_tgemv_rms): src float32 [B, K] is
    normalized per row (RMSNorm with weight norm_w, rounded to bfloat16) and
    multiplied by one packed matrix (codes uint8 [N, K/4], scales_f16
    [N, K/g]); y float32 [B, N] = the product, or += it when accumulate."""
    _need(codes, "codes", _U8, 2)
    N = codes.shape[0]
    B, K, y = _rms_args(src, norm_w, y, N)
    _need(scales_f16, "scales_f16", _F16, 2)
    _shape(codes, "codes", (N, K // 4), src.device)
    _shape(scales_f16, "scales_f16", (N, _groups(K, g)), src.device)
    st = lib().tm_tgemv_rms(_ptr(src), _ptr(norm_w), eps, _ptr(codes), _ptr(scales_f16), B, N, K,
                            g, _ptr(y), int(bool(accumulate)), _stream())
    _check("tm_tgemv_rms", st)
    return y


def dgemv_rms(src: torch.Tensor, W16: torch.Tensor, norm_w: torch.Tensor, eps: float = 1e-5,
              y: Optional[torch.Tensor] = None, accumulate: bool = False) -> torch.Tensor:
    """tgemv_rms for one matrix kept in float16: W16 float16 [N, K]."""
    _need(W16, "W16", _F16, 2)
    N = W16.shape[0]
    B, K, y = _rms_args(src, norm_w, y, N)
    _shape(W16, "W16", (N, K), src.device)
    st = lib().tm_dgemv_rms(_ptr(src), _ptr(norm_w), eps, _ptr(W16), B, N, K, _ptr(y),
                            int(bool(accumulate)), _stream())
    _check("tm_dgemv_rms", st)
    return y


MIXER_HEADDIM = 64
MIXER_DSTATE = 128


def _mixer_args(zxbcdt, conv_state, conv_pos, ssm_state, A_log, params):
    """Shape and dtype checks shared by mixer_step and mixer_gate; params:
    (tensor, name) pairs of the per-channel and per-head parameters."""
    _need(zxbcdt, "zxbcdt", _F32, 2)
    B = zxbcdt.shape[0]
    _need(A_log, "A_log", _F32, 1)
    H = A_log.shape[0]
    P, N = MIXER_HEADDIM, MIXER_DSTATE
    di, cd = H * P, H * P + 2 * N
    dev = zxbcdt.device
    _shape(zxbcdt, "zxbcdt", (B, 2 * di + 2 * N + H), dev)
    _need(conv_state, "conv_state", _F16, 3)
    _shape(conv_state, "conv_state", (B, cd, 4), dev)
    _need(conv_pos, "conv_pos", (torch.int32,), 1)
    _shape(conv_pos, "conv_pos", (1,), dev)
    _need(ssm_state, "ssm_state", _F16, 4)
    _shape(ssm_state, "ssm_state", (B, H, P, N), dev)
    shapes = {"conv_w": (cd, 4), "conv_b": (cd,), "dt_bias": (H,), "D": (H,), "norm_w": (di,)}
    for t, name in params:
        _need(t, name, _F32, len(shapes[name]))
        _shape(t, name, shapes[name], dev)
    return B, H, P, N, di, dev


def mixer_gate(zxbcdt: torch.Tensor, conv_state: torch.Tensor, conv_pos: torch.Tensor,
               ssm_state: torch.Tensor, conv_w: torch.Tensor, conv_b: torch.Tensor,
               dt_bias: torch.Tensor, A_log: torch.Tensor, D: torch.Tensor,
               gated: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The mixer step up to the gated values (tm_mixer_gate): zxbcdt float32
    [B, Z] -> gated float32 [B, d_inner] = y * SiLU(z), not normalized; the
    states and conv_pos are updated in place as by mixer_step."""
    B, H, P, N, di, dev = _mixer_args(
        zxbcdt, conv_state, conv_pos, ssm_state, A_log,
        ((conv_w, "conv_w"), (conv_b, "conv_b"), (dt_bias, "dt_bias"), (D, "D")))
    if gated is None:
        gated = torch.empty((B, di), dtype=torch.float32, device=dev)
    _need(gated, "gated", _F32, 2)
    _shape(gated, "gated", (B, di), dev)
    st = lib().tm_mixer_gate(_ptr(zxbcdt), B, H, P, N, _ptr(conv_state), _ptr(conv_pos),
                             _ptr(ssm_state), _ptr(conv_w), _ptr(conv_b), _ptr(dt_bias),
                             _ptr(A_log), _ptr(D), _ptr(gated), _stream())
    _check("tm_mixer_gate", st)
    return gated


def mixer_workspace(B: int, nheads: int, device) -> torch.Tensor:
    """Scratch for mixer_step: the gated values and per-head sums of squares."""
    return torch.empty((B * (nheads * MIXER_HEADDIM + nheads),), dtype=torch.float32,
                       device=device)


def mixer_step(zxbcdt: torch.Tensor, conv_state: torch.Tensor, conv_pos: torch.Tensor,
               ssm_state: torch.Tensor, conv_w: torch.Tensor, conv_b: torch.Tensor,
               dt_bias: torch.Tensor, A_log: torch.Tensor, D: torch.Tensor,
               norm_w: torch.Tensor, eps: float = 1e-5, *,
               workspace: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None, noalloc: bool = False) -> torch.Tensor:
    """One Mamba-2 mixer decode step between the projections (tm_mixer_step):
    zxbcdt float32 [B, Z] -> out bfloat16 [B, d_inner]; conv_state (float16
    ring [B, conv_dim, 4]), conv_pos (int32 [1]) and ssm_state (float16
    [B, nheads, 64, 128]) are updated in place.  noalloc=True calls
    tm_mixer_step_noalloc (the library's own scratch array, no workspace)."""
    B, H, P, N, di, dev = _mixer_args(
        zxbcdt, conv_state, conv_pos, ssm_state, A_log,
        ((conv_w, "conv_w"), (conv_b, "conv_b"), (dt_bias, "dt_bias"), (D, "D"),
         (norm_w, "norm_w")))
    if out is None:
        out = torch.empty((B, di), dtype=torch.bfloat16, device=dev)
    _need(out, "out", _BF16, 2)
    _shape(out, "out", (B, di), dev)
    if noalloc:
        if workspace is not None:
            raise ValueError("noalloc=True takes no workspace")
        st = lib().tm_mixer_step_noalloc(_ptr(zxbcdt), B, H, P, N, _ptr(conv_state),
                                         _ptr(conv_pos), _ptr(ssm_state), _ptr(conv_w),
                                         _ptr(conv_b), _ptr(dt_bias), _ptr(A_log), _ptr(D),
                                         _ptr(norm_w), eps, _ptr(out), _stream())
        _check("tm_mixer_step_noalloc", st)
        return out
    if workspace is None:
        workspace = mixer_workspace(B, H, dev)
    _need(workspace, "workspace", _F32, 1)
    if workspace.numel() < B * (di + H):
        raise ValueError(f"workspace holds {workspace.numel()} floats, needs {B * (di + H)}")
    st = lib().tm_mixer_step(_ptr(zxbcdt), B, H, P, N, _ptr(conv_state), _ptr(conv_pos),
                             _ptr(ssm_state), _ptr(conv_w), _ptr(conv_b), _ptr(dt_bias),
                             _ptr(A_log), _ptr(D), _ptr(norm_w), eps, _ptr(workspace), _ptr(out),
                             _stream())
    _check("tm_mixer_step", st)
    return out


def residual_rmsnorm(residual: torch.Tensor, y: Optional[torch.Tensor], w: torch.Tensor,
                     eps: float = 1e-5, x: Optional[torch.Tensor] = None) -> torch.Tensor:
    """residual float32 [B, D] += y (if given); returns x = bf16(rmsnorm(residual) * w)."""
    _need(residual, "residual", _F32, 2)
    B, D = residual.shape
    dev = residual.device
    if y is not None:
        _need(y, "y", _F32, 2)
        _shape(y, "y", (B, D), dev)
    _need(w, "w", _F32, 1)
    _shape(w, "w", (D,), dev)
    if x is None:
        x = torch.empty((B, D), dtype=torch.bfloat16, device=dev)
    _need(x, "x", _BF16, 2)
    _shape(x, "x", (B, D), dev)
    st = lib().tm_residual_rmsnorm(_ptr(residual), _ptr(y), B, D, _ptr(w), eps, _ptr(x),
                                   _stream())
    _check("tm_residual_rmsnorm", st)
    return x


STACK_FIELDS = ("in_codes", "in_scales", "out_codes", "out_scales", "pre_w", "conv_w", "conv_b",
                "dt_bias", "A_log", "D", "norm_w", "final_w", "conv_state", "conv_pos",
                "ssm_state")


def mamba2_decode_workspace(d_model: int, nheads: int, device, batch: int = 1) -> torch.Tensor:
    """Scratch for mamba2_decode_token (uint8)."""
    n = int(lib().tm_mamba2_decode_workspace(d_model, nheads, batch))
    if n < 0:
        raise ValueError(f"no stack decode for d_model={d_model}, nheads={nheads}, "
                         f"batch={batch}")
    return torch.empty((n,), dtype=torch.uint8, device=device)


def mamba2_decode_token(arrays: dict, g: int, eps: float, emb: torch.Tensor,
                        x_out: Optional[torch.Tensor] = None,
                        workspace: Optional[torch.Tensor] = None, kept=(),
                        in_w16: Optional[torch.Tensor] = None,
                        out_w16: Optional[torch.Tensor] = None) -> torch.Tensor:
    """One decode token per batch row through a stack of Mamba-2 blocks in a
    single launch (``tm_mamba2_decode_token``).  arrays: the stacked device
    tensors named as ``tm_mamba2_stack``'s fields (``STACK_FIELDS``).  emb
    float32 [d_model] (batch 1; the states then [L, conv_dim, 4] and [L,
    nheads, 64, 128]) or [B, d_model] with B = 1 .. 4 (the states [L, B,
    ...]); returns x_out bfloat16 of emb's shape (the final norm).  kept: the
    indices (ascending) of blocks kept in FP16, whose projections are in_w16
    float16 [len(kept), Z, d_model] and out_w16 [len(kept), d_model,
    d_inner]."""
    P, N = MIXER_HEADDIM, MIXER_DSTATE
    L, Z, d4 = arrays["in_codes"].shape
    D = 4 * d4
    H = arrays["dt_bias"].shape[1]
    di, cd = H * P, H * P + 2 * N
    dev = emb.device
    if emb.dim() not in (1, 2):
        raise ValueError(f"emb must be [d_model] or [B, d_model], got {tuple(emb.shape)}")
    B = 1 if emb.dim() == 1 else emb.shape[0]
    lead = (L,) if emb.dim() == 1 else (L, B)
    want = {"in_codes": ((L, Z, D // 4), _U8), "in_scales": ((L, Z, _groups(D, g)), _F16),
            "out_codes": ((L, D, di // 4), _U8), "out_scales": ((L, D, _groups(di, g)), _F16),
            "pre_w": ((L, D), _F32), "conv_w": ((L, cd, 4), _F32), "conv_b": ((L, cd), _F32),
            "dt_bias": ((L, H), _F32), "A_log": ((L, H), _F32), "D": ((L, H), _F32),
            "norm_w": ((L, di), _F32), "final_w": ((D,), _F32),
            "conv_state": (lead + (cd, 4), _F16), "conv_pos": ((L,), (torch.int32,)),
            "ssm_state": (lead + (H, P, N), _F16)}
    if Z != 2 * di + 2 * N + H:
        raise ValueError(f"in_codes has {Z} rows; nheads={H} needs {2 * di + 2 * N + H}")
    for name, (shape, dtypes) in want.items():
        t = arrays[name]
        _need(t, name, dtypes, len(shape))
        _shape(t, name, shape, dev)
    shp = tuple(emb.shape[:-1]) + (D,)
    _need(emb, "emb", _F32, emb.dim())
    _shape(emb, "emb", shp, dev)
    if x_out is None:
        x_out = torch.empty(shp, dtype=torch.bfloat16, device=dev)
    _need(x_out, "x_out", _BF16, emb.dim())
    _shape(x_out, "x_out", shp, dev)
    if workspace is None:
        workspace = mamba2_decode_workspace(D, H, dev, B)
    _need(workspace, "workspace", _U8, 1)
    if workspace.device != dev:
        raise ValueError(f"workspace is on {workspace.device}, the operands on {dev}")
    kept = [int(i) for i in kept]
    nk = len(kept)
    kept_arr = (ctypes.c_int32 * max(nk, 1))(*kept)
    if nk:
        _need(in_w16, "in_w16", _F16, 3)
        _shape(in_w16, "in_w16", (nk, Z, D), dev)
        _need(out_w16, "out_w16", _F16, 3)
        _shape(out_w16, "out_w16", (nk, D, di), dev)
    st = Mamba2Stack(L, D, H, g, eps, *(arrays[k].data_ptr() for k in STACK_FIELDS),
                     nk, kept_arr if nk else None, _ptr(in_w16) if nk else None,
                     _ptr(out_w16) if nk else None, B)
    rc = lib().tm_mamba2_decode_token(ctypes.byref(st), _ptr(emb), _ptr(x_out), _ptr(workspace),
                                      workspace.numel(), _stream())
    _check("tm_mamba2_decode_token", rc)
    return x_out
