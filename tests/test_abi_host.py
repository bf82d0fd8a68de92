"""The C ABI on the host: the library loads, exports every declared symbol,
and rejects bad arguments with the documented status codes before any HIP
call.  No test here passes arguments that would reach a kernel launch."""

import ctypes
import os
import re

import pytest

from paper_2606_18114_amd import ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tmamba.h")

OK, EINVAL, ESHAPE, EALIGN = 0, 1, 2, 3
P = 0x7F0000000000  # a 4 KiB-aligned fake device address, never dereferenced


@pytest.fixture(scope="module")
def L():
    # TM_ABI_TEST_LIB: a host-only sanitizer build of the same C ABI
    # (tests/test_abi_sanitized.py), loaded with the binding's signatures
    alt = os.environ.get("TM_ABI_TEST_LIB")
    if alt:
        lib = ctypes.CDLL(alt)
        for name, (res, args) in ops.SIGNATURES.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        return lib
    if not os.path.exists(ops.lib_path()):
        from paper_2606_18114_amd import build
        build.build(verbose=False)
    return ops.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:tm_status|int|int64_t|const char\*)\s+(tm_[a-z0-9_]+)\(",
                                 text, re.M)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) == 26
    for n in names:
        assert hasattr(L, n), n
        assert n in ops.SIGNATURES, n
    assert L.tm_abi_version() == 15


def test_status_strings(L):
    for code, name in ops.TM_STATUS.items():
        assert L.tm_status_str(code).decode().startswith(name)
    assert L.tm_status_str(99).decode() == "unknown tm_status"


def tp(L, W=P, N=8, K=128, g=128, eps=1e-5, codes=P + 2 ** 20, scales=P + 2 ** 21,
       s16=0, zc=0):
    return L.tm_ternarize_pack(W, N, K, g, eps, codes, scales, s16, zc, None)


def test_ternarize_pack_validation(L):
    assert tp(L, W=0) == EINVAL
    assert tp(L, codes=0) == EINVAL
    assert tp(L, scales=0) == EINVAL
    assert tp(L, eps=-1.0) == EINVAL
    assert tp(L, eps=float("nan")) == EINVAL
    assert tp(L, eps=float("inf")) == EINVAL
    assert tp(L, N=0) == ESHAPE
    assert tp(L, K=0) == ESHAPE
    assert tp(L, g=100) == ESHAPE
    assert tp(L, g=16) == ESHAPE
    assert tp(L, K=96, g=32) == ESHAPE          # K % 64
    assert tp(L, K=192, g=128) == ESHAPE        # K % g
    assert tp(L, N=2 ** 40, K=2 ** 20) == ESHAPE  # size overflow
    assert tp(L, W=P + 4) == EALIGN
    assert tp(L, codes=P + 2 ** 20 + 8) == EALIGN
    assert tp(L, scales=P + 2 ** 21 + 2) == EALIGN
    assert tp(L, s16=P + 2 ** 22 + 1) == EALIGN
    assert tp(L, zc=P + 2 ** 23 + 4) == EALIGN
    # outputs overlapping the input or each other
    assert tp(L, codes=P + 64) == EINVAL
    assert tp(L, scales=P + 2 ** 20 + 16) == EINVAL
    assert tp(L, s16=P + 2 ** 21) == EINVAL
    assert tp(L, zc=P + 2 ** 20) == EINVAL


def tpt(L, W=P, N=8, K=128, g=128, eps=1e-5, mult=P + 2 ** 23, codes=P + 2 ** 20,
        scales=P + 2 ** 21, s16=0, zc=0):
    return L.tm_ternarize_pack_thresh(W, N, K, g, eps, mult, codes, scales, s16, zc, None)


def test_ternarize_pack_thresh_validation(L):
    # the standard checks apply unchanged
    assert tpt(L, W=0) == EINVAL
    assert tpt(L, eps=float("nan")) == EINVAL
    assert tpt(L, g=100) == ESHAPE
    assert tpt(L, K=192, g=128) == ESHAPE
    assert tpt(L, W=P + 4) == EALIGN
    assert tpt(L, codes=P + 64) == EINVAL
    # the multiplier array: 4-byte aligned, not overlapping an output
    assert tpt(L, mult=P + 2 ** 23 + 2) == EALIGN
    assert tpt(L, mult=P + 2 ** 21) == EINVAL            # overlaps the scales
    assert tpt(L, mult=P + 2 ** 20 + 4) == EINVAL        # overlaps the codes


def tc(L, W=P, N=8, K=128, g=128, eps=1e-5, tau=P + 2 ** 23, codes=P + 2 ** 20, zc=0):
    return L.tm_ternarize_codes(W, N, K, g, eps, tau, codes, zc, None)


def test_ternarize_codes_validation(L):
    for kw in ("W", "tau", "codes"):
        assert tc(L, **{kw: 0}) == EINVAL, kw
    assert tc(L, eps=-1.0) == EINVAL
    assert tc(L, N=0) == ESHAPE
    assert tc(L, K=192, g=128) == ESHAPE
    assert tc(L, g=48) == ESHAPE
    assert tc(L, W=P + 8) == EALIGN
    assert tc(L, tau=P + 2 ** 23 + 2) == EALIGN
    assert tc(L, codes=P + 2 ** 20 + 4) == EALIGN
    assert tc(L, zc=P + 2 ** 22 + 4) == EALIGN
    assert tc(L, codes=P + 512) == EINVAL               # overlaps W
    assert tc(L, codes=P + 2 ** 23) == EINVAL           # overlaps tau
    assert tc(L, zc=P + 2 ** 20 + 8) == EINVAL          # overlaps the codes


def gcd(L, codes=P, dW=P + 2 ** 24, N=8, K=512, g=128, out=P + 2 ** 26):
    return L.tm_group_code_dot(codes, dW, N, K, g, out, None)


def test_group_code_dot_validation(L):
    for kw in ("codes", "dW", "out"):
        assert gcd(L, **{kw: 0}) == EINVAL, kw
    assert gcd(L, N=0) == ESHAPE
    assert gcd(L, K=96, g=32) == ESHAPE
    assert gcd(L, K=256, g=512) == ESHAPE
    assert gcd(L, g=16) == ESHAPE
    assert gcd(L, N=2 ** 40, K=2 ** 20) == ESHAPE
    assert gcd(L, codes=P + 8) == EALIGN
    assert gcd(L, dW=P + 2 ** 24 + 4) == EALIGN
    assert gcd(L, out=P + 2 ** 26 + 2) == EALIGN
    assert gcd(L, out=P + 256) == EINVAL                 # overlaps the codes
    assert gcd(L, out=P + 2 ** 24 + 1024) == EINVAL      # overlaps dW


def ssg(L, W=P, codes=P + 2 ** 22, scale=P + 2 ** 23, dWhat=P + 2 ** 24, N=8, K=256, g=128,
        eps=1e-5, ds=P + 2 ** 25, dW=P + 2 ** 26):
    return L.tm_scale_ste_grad(W, codes, scale, dWhat, N, K, g, eps, ds, dW, None)


def test_scale_ste_grad_validation(L):
    for kw in ("W", "codes", "scale", "dWhat", "ds"):
        assert ssg(L, **{kw: 0}) == EINVAL, kw
    assert ssg(L, eps=-1.0) == EINVAL
    assert ssg(L, eps=float("nan")) == EINVAL
    assert ssg(L, N=0) == ESHAPE
    assert ssg(L, K=96, g=32) == ESHAPE
    assert ssg(L, g=16) == ESHAPE
    assert ssg(L, N=2 ** 40, K=2 ** 20) == ESHAPE
    assert ssg(L, W=P + 4) == EALIGN
    assert ssg(L, dWhat=P + 2 ** 24 + 8) == EALIGN
    assert ssg(L, dW=P + 2 ** 26 + 4) == EALIGN
    assert ssg(L, ds=P + 2 ** 25 + 2) == EALIGN
    assert ssg(L, ds=P + 64) == EINVAL                    # ds overlaps W
    assert ssg(L, ds=P + 2 ** 24 + 64) == EINVAL          # ds overlaps dWhat
    assert ssg(L, dW=P + 2 ** 22) == EINVAL               # dW overlaps the codes
    assert ssg(L, dW=P + 2 ** 24 + 16) == EINVAL          # partly over dWhat
    assert ssg(L, dW=P + 2 ** 25 - 4 * 1024) == EINVAL    # dW [8, 256] (8 KiB) reaches ds


def dg(L, x=P, W=P + 2 ** 24, count=2, B=1, N=300, K=2048, y=P + 2 ** 28):
    return L.tm_dgemv(x, W, count, B, N, K, y, None)


def test_dgemv_validation(L):
    for kw in ("x", "W", "y"):
        assert dg(L, **{kw: 0}) == EINVAL, kw
    assert dg(L, count=0) == ESHAPE
    assert dg(L, count=65536) == ESHAPE
    assert dg(L, B=0) == ESHAPE
    assert dg(L, B=9) == ESHAPE
    assert dg(L, N=0) == ESHAPE
    assert dg(L, K=2000) == ESHAPE
    assert dg(L, B=5, K=4096) == ESHAPE          # x staging beyond 64 KiB of LDS
    assert dg(L, x=P + 8) == EALIGN
    assert dg(L, W=P + 2 ** 24 + 8) == EALIGN
    assert dg(L, y=P + 2 ** 28 + 2) == EALIGN
    assert dg(L, y=P + 2048) == EINVAL           # y overlaps x
    assert dg(L, y=P + 2 ** 24 + 4096) == EINVAL  # y overlaps W


def mx(L, z=P, B=1, H=64, hd=64, ds=128, cs=P + 2 ** 20, pos=P + 2 ** 21, ss=P + 2 ** 22,
       cw=P + 2 ** 24, cb=P + 2 ** 25, dtb=P + 2 ** 26, al=P + 2 ** 26 + 4096,
       D=P + 2 ** 26 + 8192, nw=P + 2 ** 27, eps=1e-5, ws=P + 2 ** 28, out=P + 2 ** 29):
    return L.tm_mixer_step(z, B, H, hd, ds, cs, pos, ss, cw, cb, dtb, al, D, nw, eps, ws, out,
                           None)


def test_mixer_step_noalloc_validation(L):
    def na(**kw):
        S = 2 ** 27   # arrays far apart, so that only the size check can fail
        a = dict(z=P, B=1, H=64, hd=64, ds=128, cs=P + S, pos=P + 2 * S, ss=P + 3 * S,
                 cw=P + 4 * S, cb=P + 5 * S, dtb=P + 6 * S, al=P + 7 * S, D=P + 8 * S,
                 nw=P + 9 * S, eps=1e-5, out=P + 10 * S)
        a.update(kw)
        return L.tm_mixer_step_noalloc(a["z"], a["B"], a["H"], a["hd"], a["ds"], a["cs"],
                                       a["pos"], a["ss"], a["cw"], a["cb"], a["dtb"], a["al"],
                                       a["D"], a["nw"], a["eps"], a["out"], None)
    assert na(z=0) == EINVAL
    assert na(out=0) == EINVAL
    assert na(hd=32) == ESHAPE
    # the scratch array holds 16 * (8192 + 128) = 133120 floats
    assert na(B=33) == ESHAPE          # 33 * (4096 + 64) = 137280 floats
    assert na(B=1, H=2049) == ESHAPE   # 2049 * 65 = 133185 floats
    assert na(ss=P + 3 * 2 ** 27 + 8) == EALIGN
    assert na(out=P + 3 * 2 ** 27) == EINVAL    # out over the SSM state


def test_mixer_step_validation(L):
    for kw in ("z", "cs", "pos", "ss", "cw", "cb", "dtb", "al", "D", "nw", "ws", "out"):
        assert mx(L, **{kw: 0}) == EINVAL, kw
    assert mx(L, eps=-1.0) == EINVAL
    assert mx(L, B=0) == ESHAPE
    assert mx(L, H=0) == ESHAPE
    assert mx(L, hd=32) == ESHAPE
    assert mx(L, ds=64) == ESHAPE
    assert mx(L, ss=P + 2 ** 22 + 8) == EALIGN
    assert mx(L, pos=P + 2 ** 21 + 2) == EALIGN
    assert mx(L, cs=P + 2 ** 20 + 4) == EALIGN            # conv ring: 8-byte aligned
    assert mx(L, out=P + 2 ** 29 + 1) == EALIGN
    assert mx(L, ss=P + 2 ** 20 + 64) == EINVAL           # SSM state over the conv state
    assert mx(L, out=P + 2 ** 22) == EINVAL               # out over the SSM state
    assert mx(L, ws=P + 16) == EINVAL                     # workspace over zxbcdt
    assert mx(L, pos=P + 2 ** 24 + 64) == EINVAL          # conv_pos inside conv_w


def tr(L, src=P, nw=P + 2 ** 20, eps=1e-5, codes=P + 2 ** 21, s16=P + 2 ** 24, B=1, N=8512,
       K=2048, g=128, y=P + 2 ** 25, acc=0):
    return L.tm_tgemv_rms(src, nw, eps, codes, s16, B, N, K, g, y, acc, None)


def test_tgemv_rms_validation(L):
    for kw in ("src", "nw", "codes", "s16", "y"):
        assert tr(L, **{kw: 0}) == EINVAL, kw
    assert tr(L, eps=-1.0) == EINVAL
    assert tr(L, eps=float("nan")) == EINVAL
    assert tr(L, acc=2) == EINVAL
    assert tr(L, B=0) == ESHAPE
    assert tr(L, N=0) == ESHAPE
    assert tr(L, K=2000) == ESHAPE
    assert tr(L, g=100) == ESHAPE
    assert tr(L, B=5) == ESHAPE                 # 20 A rows: more than one operand
    assert tr(L, B=3, g=64) == ESHAPE           # 4 * 3 * 2 = 24 A rows
    assert tr(L, B=4, K=3584) == ESHAPE         # 4 * 224 pieces > 512 (4 waves)
    assert tr(L, src=P + 8) == EALIGN
    assert tr(L, nw=P + 2 ** 20 + 4) == EALIGN
    assert tr(L, y=P + 2 ** 25 + 4) == EALIGN
    assert tr(L, y=P + 4096) == EINVAL          # y over src
    assert tr(L, y=P + 2 ** 20) == EINVAL       # y over the norm weight
    assert tr(L, y=P + 2 ** 21 + 2 ** 20) == EINVAL  # y over the codes


def dr(L, src=P, nw=P + 2 ** 20, eps=1e-5, W=P + 2 ** 21, B=1, N=2048, K=4096,
       y=P + 2 ** 26, acc=1):
    return L.tm_dgemv_rms(src, nw, eps, W, B, N, K, y, acc, None)


def test_dgemv_rms_validation(L):
    for kw in ("src", "nw", "W", "y"):
        assert dr(L, **{kw: 0}) == EINVAL, kw
    assert dr(L, eps=float("inf")) == EINVAL
    assert dr(L, acc=-1) == EINVAL
    assert dr(L, B=0) == ESHAPE
    assert dr(L, B=9, K=64) == ESHAPE
    assert dr(L, K=1000) == ESHAPE
    assert dr(L, B=5) == ESHAPE                 # 5 * 4096 > 16384
    assert dr(L, src=P + 4) == EALIGN
    assert dr(L, y=P + 2 ** 26 + 2) == EALIGN
    assert dr(L, y=P + 2 ** 21 + 64) == EINVAL  # y over W
    assert dr(L, y=P + 2 ** 20 + 4) == EINVAL   # y over the norm weight


def mg(L, z=P, B=1, H=64, hd=64, ds=128, cs=P + 2 ** 20, pos=P + 2 ** 21, ss=P + 2 ** 22,
       cw=P + 2 ** 24, cb=P + 2 ** 25, dtb=P + 2 ** 26, al=P + 2 ** 26 + 4096,
       D=P + 2 ** 26 + 8192, gated=P + 2 ** 28):
    return L.tm_mixer_gate(z, B, H, hd, ds, cs, pos, ss, cw, cb, dtb, al, D, gated, None)


def test_mixer_gate_validation(L):
    for kw in ("z", "cs", "pos", "ss", "cw", "cb", "dtb", "al", "D", "gated"):
        assert mg(L, **{kw: 0}) == EINVAL, kw
    assert mg(L, B=0) == ESHAPE
    assert mg(L, hd=128) == ESHAPE
    assert mg(L, gated=P + 2 ** 28 + 2) == EALIGN          # float32 output
    assert mg(L, gated=P + 2 ** 22 + 64) == EINVAL         # gated over the SSM state
    assert mg(L, gated=P + 8) == EINVAL                    # gated over zxbcdt
    assert mg(L, pos=P + 2 ** 28 + 4) == EINVAL            # conv_pos inside gated


def rn(L, r=P, y=P + 2 ** 20, B=2, D=2048, w=P + 2 ** 21, eps=1e-5, x=P + 2 ** 22):
    return L.tm_residual_rmsnorm(r, y, B, D, w, eps, x, None)


def test_residual_rmsnorm_validation(L):
    for kw in ("r", "w", "x"):
        assert rn(L, **{kw: 0}) == EINVAL, kw
    assert rn(L, eps=float("inf")) == EINVAL
    assert rn(L, B=0) == ESHAPE
    assert rn(L, D=0) == ESHAPE
    assert rn(L, r=P + 2) == EALIGN
    assert rn(L, x=P + 2 ** 22 + 1) == EALIGN
    assert rn(L, x=P + 64) == EINVAL          # x over the residual
    assert rn(L, y=P + 4096) == EINVAL        # y over the residual
    assert rn(L, w=P + 2 ** 22 + 64) == EINVAL  # w over x


def fwd(L, X=P, codes=P + 2 ** 24, scales=P + 2 ** 25, M=16, N=256, K=512, g=128, Y=P + 2 ** 26):
    return L.tm_tgemm_fwd(X, codes, scales, M, N, K, g, Y, None)


def test_tgemm_fwd_validation(L):
    for kw in ("X", "codes", "scales", "Y"):
        assert fwd(L, **{kw: 0}) == EINVAL, kw
    assert fwd(L, M=0) == ESHAPE
    assert fwd(L, N=-1) == ESHAPE
    assert fwd(L, K=544) == ESHAPE
    assert fwd(L, g=48) == ESHAPE
    assert fwd(L, K=256, g=512) == ESHAPE
    assert fwd(L, M=1, K=2 ** 22 + 128, N=8) == ESHAPE  # beyond the 32-bit tile offsets
    assert fwd(L, M=1, N=2 ** 26 + 8) == ESHAPE
    assert fwd(L, X=P + 2) == EALIGN
    assert fwd(L, codes=P + 2 ** 24 + 4) == EALIGN
    assert fwd(L, scales=P + 2 ** 25 + 2) == EALIGN
    assert fwd(L, Y=P + 2 ** 26 + 4) == EALIGN
    assert fwd(L, Y=P + 4096) == EINVAL                 # Y overlaps X
    assert fwd(L, Y=P + 2 ** 24 - 4096) == EINVAL       # Y overlaps codes


def test_tgemm_fwd_ws_validation(L):
    # ticket words of up to 1024 cut tiles, two per tile
    assert L.tm_tgemm_fwd_workspace() == 8192

    def f(X=P, codes=P + 2 ** 24, scales=P + 2 ** 25, M=16, N=256, K=512, g=128,
          Y=P + 2 ** 26, ws=P + 2 ** 27, wsb=8192):
        return L.tm_tgemm_fwd_ws(X, codes, scales, M, N, K, g, Y, ws, wsb, None)
    for kw in ("X", "codes", "scales", "Y", "ws"):
        assert f(**{kw: 0}) == EINVAL, kw
    assert f(M=0) == ESHAPE
    assert f(K=544) == ESHAPE
    assert f(wsb=8188) == ESHAPE                      # one word short
    assert f(ws=P + 2 ** 27 + 2) == EALIGN
    assert f(Y=P + 2 ** 26 + 4) == EALIGN
    assert f(ws=P + 2 ** 26) == EINVAL                # workspace over Y
    assert f(ws=P + 2 ** 25 - 4096) == EINVAL         # workspace runs into the scales
    assert f(ws=P + 64) == EINVAL                     # workspace over X


def test_tgemm_fwd_bf16_validation(L):
    def f(X=P, codes=P + 2 ** 24, scales=P + 2 ** 25, M=16, N=256, K=512, g=128, Y=P + 2 ** 26):
        return L.tm_tgemm_fwd_bf16(X, codes, scales, M, N, K, g, Y, None)
    for kw in ("X", "codes", "scales", "Y"):
        assert f(**{kw: 0}) == EINVAL, kw
    assert f(M=0) == ESHAPE
    assert f(K=544) == ESHAPE
    assert f(g=48) == ESHAPE
    assert f(Y=P + 2 ** 26 + 2) == EALIGN
    assert f(Y=P + 4096) == EINVAL                 # Y overlaps X
    # a bfloat16 Y of 16 x 256 is 8 KiB: one byte more reaches the codes
    assert f(Y=P + 2 ** 24 - 8192 + 16) == EINVAL


def dx(L, dY=P, codes=P + 2 ** 24, scales=P + 2 ** 25, M=16, N=256, K=512, g=128,
       dX=P + 2 ** 26):
    return L.tm_tgemm_bwd_dx(dY, codes, scales, M, N, K, g, dX, None)


def test_tgemm_bwd_dx_validation(L):
    for kw in ("dY", "codes", "scales", "dX"):
        assert dx(L, **{kw: 0}) == EINVAL, kw
    assert dx(L, N=250) == ESHAPE                        # dY rows not 16-byte multiples
    assert dx(L, M=0) == ESHAPE
    assert dx(L, K=100) == ESHAPE
    assert dx(L, N=2 ** 22 + 8) == ESHAPE                # 32-bit dY row offsets
    assert dx(L, dY=P + 8) == EALIGN
    assert dx(L, dX=P + 2 ** 26 + 8) == EALIGN
    assert dx(L, dX=P) == EINVAL


def gpair(L, x0=P, c0=P + 2 ** 24, s0=P + 2 ** 25, n0=2, N0=256, K0=512, y0=P + 2 ** 26,
          x1=P + 2 ** 27, c1=P + 2 ** 28, s1=P + 2 ** 29, n1=3, N1=128, K1=1024,
          y1=P + 2 ** 30, B=1, g=128):
    return L.tm_tgemv_pair(x0, c0, s0, n0, N0, K0, y0, x1, c1, s1, n1, N1, K1, y1, B, g, None)


def test_tgemv_pair_validation(L):
    for kw in ("x0", "c0", "s0", "y0", "x1", "c1", "s1", "y1"):
        assert gpair(L, **{kw: 0}) == EINVAL, kw
    assert gpair(L, n0=0) == ESHAPE
    assert gpair(L, n1=65536) == ESHAPE
    assert gpair(L, K1=1000) == ESHAPE                   # K % 64 in the second stack
    assert gpair(L, B=17) == ESHAPE
    assert gpair(L, g=96) == ESHAPE
    assert gpair(L, y1=P + 2 ** 30 + 4) == EALIGN
    assert gpair(L, y1=P + 2 ** 26) == EINVAL            # the two outputs overlap
    assert gpair(L, y1=P + 2 ** 24) == EINVAL            # y1 over the first stack's codes
    assert gpair(L, y0=P + 2 ** 28) == EINVAL            # y0 over the second stack's codes


def stack_desc(**kw):
    # fake device arrays 64 MiB apart (the checks never dereference them)
    names = ops.STACK_FIELDS
    vals = {n: P + (i + 1) * 2 ** 26 for i, n in enumerate(names)}
    vals.update({k: v for k, v in kw.items() if k in names})
    dims = dict(n_layers=2, d_model=256, nheads=2, g=128, eps=1e-5)
    dims.update({k: v for k, v in kw.items() if k in dims})
    st = ops.Mamba2Stack(dims["n_layers"], dims["d_model"], dims["nheads"], dims["g"],
                         dims["eps"], *(vals[n] for n in names))
    st.batch = kw.get("batch", 1)
    if "kept" in kw:  # host list of kept blocks; their float16 arrays after the others
        kept = kw["kept"]
        st.n_kept = kw.get("n_kept", len(kept))
        st._kept_keepalive = (ctypes.c_int32 * max(len(kept), 1))(*kept)
        st.kept = ctypes.cast(st._kept_keepalive, ctypes.POINTER(ctypes.c_int32)) if kept else None
        st.in_w16 = kw.get("in_w16", P + 20 * 2 ** 26)
        st.out_w16 = kw.get("out_w16", P + 21 * 2 ** 26)
    return st


def mdec(L, emb=P + 2 ** 31, x_out=P + 2 ** 31 + 2 ** 20, ws=P + 2 ** 32, wsb=None, **kw):
    st = stack_desc(**kw)
    if wsb is None:
        wsb = L.tm_mamba2_decode_workspace(st.d_model, st.nheads, max(st.batch, 1))
    return L.tm_mamba2_decode_token(ctypes.byref(st), emb, x_out, ws, wsb, None)


def test_mamba2_decode_token_validation(L):
    # [barrier words 32 KiB | zx Z | gated | partial | residual], 256-byte pieces
    z = 2 * 128 + 256 + 2
    ws = L.tm_mamba2_decode_workspace
    assert ws(256, 2, 1) == 32768 + 2304 + 512 + 256 + 1024 and z == 514
    # batch 3: every piece three rows
    assert ws(256, 2, 3) == 32768 + 6400 + 1536 + 256 + 3072
    assert ws(8192, 2, 1) == -1
    assert ws(256, 0, 1) == -1
    assert ws(256, 2, 0) == -1
    assert ws(256, 2, 5) == -1
    assert L.tm_mamba2_decode_token(None, P, P, P, 1 << 20, None) == EINVAL
    for name in ops.STACK_FIELDS:
        assert mdec(L, **{name: 0}) == EINVAL, name
    assert mdec(L, emb=0) == EINVAL
    assert mdec(L, eps=-1.0) == EINVAL
    assert mdec(L, eps=float("nan")) == EINVAL
    assert mdec(L, g=32) == ESHAPE                  # g in {64, 128, 256}
    assert mdec(L, d_model=4160) == ESHAPE          # beyond 4096
    assert mdec(L, d_model=320) == ESHAPE           # not a multiple of g = 128
    assert mdec(L, nheads=3) == ESHAPE              # d_inner 192 not a multiple of 128
    assert mdec(L, nheads=129) == ESHAPE
    assert mdec(L, n_layers=0) == ESHAPE
    assert mdec(L, wsb=1024) == ESHAPE              # workspace too small
    assert mdec(L, ws=P + 2 ** 32 + 128) == EALIGN
    assert mdec(L, ssm_state=P + 15 * 2 ** 26 + 8) == EALIGN
    assert mdec(L, conv_state=P + 13 * 2 ** 26 + 4) == EALIGN
    assert mdec(L, x_out=P + 2 ** 31 + 1) == EALIGN
    assert mdec(L, x_out=P + 2 ** 31 + 2) == EALIGN           # stored in bfloat16 pairs
    assert mdec(L, norm_w=P + 11 * 2 ** 26 + 4) == EALIGN   # the norm weights load 16 bytes
    assert mdec(L, emb=P + 2 ** 31 + 4) == EALIGN           # so does the embedding
    # batches: 1 .. 4 rows, up to d_model 2048 / d_inner 4096 above 1
    assert mdec(L, batch=0, wsb=1 << 20) == ESHAPE
    assert mdec(L, batch=5, wsb=1 << 20) == ESHAPE
    assert mdec(L, batch=2, d_model=4096) == ESHAPE
    assert mdec(L, batch=2, nheads=66) == ESHAPE            # d_inner 4224
    assert mdec(L, batch=2, wsb=ws(256, 2, 1)) == ESHAPE
    assert mdec(L, batch=2, x_out=P + 2 ** 32 - 512) == EINVAL   # second row over the workspace
    # a state array over a weight array, the output over the workspace
    assert mdec(L, ssm_state=P + 1 * 2 ** 26) == EINVAL
    assert mdec(L, x_out=P + 2 ** 32) == EINVAL
    assert mdec(L, conv_pos=P + 13 * 2 ** 26 + 64) == EINVAL   # inside the conv ring
    # blocks kept in FP16: a host list, ascending, below n_layers, at most 64
    assert mdec(L, kept=[0], n_layers=3, wsb=1024) == ESHAPE    # still checks the rest
    assert mdec(L, kept=[2], n_layers=2) == ESHAPE               # past the last block
    assert mdec(L, kept=[1, 0], n_layers=3) == ESHAPE            # not ascending
    assert mdec(L, kept=[1, 1], n_layers=3) == ESHAPE            # repeated
    assert mdec(L, kept=[0], n_kept=65, n_layers=3) == ESHAPE
    assert mdec(L, kept=[], n_kept=1, n_layers=3) == EINVAL      # no list
    assert mdec(L, kept=[0], n_layers=3, in_w16=0) == EINVAL
    assert mdec(L, kept=[0], n_layers=3, out_w16=P + 21 * 2 ** 26 + 8) == EALIGN
    assert mdec(L, kept=[0], n_layers=3, ssm_state=P + 20 * 2 ** 26) == EINVAL  # over in_w16


def dx16(L, dY=P, codes=P + 2 ** 24, scales=P + 2 ** 25, M=16, N=256, K=512, g=128,
         dX=P + 2 ** 26, ws=P + 2 ** 27, wsb=None):
    if wsb is None:
        wsb = L.tm_tgemm_bwd_dx_f16_workspace(M, N)
    return L.tm_tgemm_bwd_dx_f16(dY, codes, scales, M, N, K, g, dX, ws, wsb, None)


def test_tgemm_bwd_dx_f16_validation(L):
    # workspace bytes: float16 copy of dY, row exponents, scale maxima (256-byte pieces)
    assert L.tm_tgemm_bwd_dx_f16_workspace(16, 256) == 16 * 256 * 2 + 256 + 1024
    assert L.tm_tgemm_bwd_dx_f16_workspace(16384, 8512) == 16384 * 8512 * 2 + 65536 + 1024
    assert L.tm_tgemm_bwd_dx_f16_workspace(0, 256) == -1
    assert L.tm_tgemm_bwd_dx_f16_workspace(2 ** 40, 2 ** 40) == -1
    for kw in ("dY", "codes", "scales", "dX", "ws"):
        assert dx16(L, **{kw: 0}) == EINVAL, kw
    assert dx16(L, N=250) == ESHAPE
    assert dx16(L, K=100) == ESHAPE
    assert dx16(L, wsb=16 * 256 * 2) == ESHAPE            # one piece short
    assert dx16(L, ws=P + 2 ** 27 + 16) == EALIGN         # workspace needs 256 bytes
    assert dx16(L, dX=P + 2 ** 26 + 8) == EALIGN
    assert dx16(L, ws=P + 2 ** 26) == EINVAL              # workspace over dX
    assert dx16(L, ws=P + 2 ** 25 - 512) == EINVAL        # workspace runs into the scales
    assert dx16(L, ws=P) == EINVAL                        # workspace over dY


def dw(L, dY=P, X=P + 2 ** 24, M=16, N=256, K=512, dW=P + 2 ** 26, acc=0):
    return L.tm_tgemm_bwd_dw_ste(dY, X, M, N, K, dW, acc, None)


def test_tgemm_bwd_dw_validation(L):
    for kw in ("dY", "X", "dW"):
        assert dw(L, **{kw: 0}) == EINVAL, kw
    assert dw(L, acc=2) == EINVAL
    assert dw(L, M=0) == ESHAPE
    assert dw(L, N=12) == ESHAPE
    assert dw(L, K=96) == ESHAPE
    assert dw(L, X=P + 2 ** 24 + 2) == EALIGN
    assert dw(L, dW=P + 2 ** 24) == EINVAL


def gv(L, x=P, codes=P + 2 ** 24, s16=P + 2 ** 25, count=2, B=1, N=256, K=512, g=128,
       y=P + 2 ** 26):
    return L.tm_tgemv(x, codes, s16, count, B, N, K, g, y, None)


def test_tgemv_validation(L):
    for kw in ("x", "codes", "s16", "y"):
        assert gv(L, **{kw: 0}) == EINVAL, kw
    assert gv(L, count=0) == ESHAPE
    assert gv(L, count=65536) == ESHAPE
    assert gv(L, B=0) == ESHAPE
    assert gv(L, B=17) == ESHAPE
    assert gv(L, K=544, g=32) == ESHAPE
    assert gv(L, count=1, B=1, N=2 ** 20, K=2 ** 13 + 128) == ESHAPE  # > 2^31 code bytes per matrix
    assert gv(L, s16=P + 2 ** 25 + 1) == EALIGN
    assert gv(L, y=P + 2 ** 26 + 4) == EALIGN
    assert gv(L, y=P + 2 ** 24 + 256) == EINVAL          # y overlaps the codes


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(ops, "_lib", None)
    monkeypatch.setattr(ops, "_LIB_PATH", str(tmp_path / "libtmamba.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        ops.lib()


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2606_18114_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".hpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle", text, re.M), f
                assert "oracle/" not in text, f
