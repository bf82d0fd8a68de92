"""Pins of the oracle's decode product, its float16 scales, the boundary band
and the relative Frobenius error (the contract's measure).

Each oracle function is held to hand-worked values (tests/golden/
decode_examples.json, exact dyadic numbers with their derivations), to a
pure-Python twin written from the definitions (``brute.f16``: binary16
rounding from the format, ``brute.gemv``: fsum loops), and the last block
plants plausible mistakes in the oracle and checks that a pin catches each.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import brute
from oracle import ternary as O
from paper_2606_18114_amd import synth


def _f(v):
    return float("inf") if v == "inf" else float.fromhex(v)


@pytest.fixture(scope="module")
def dec(golden_dir):
    with open(os.path.join(golden_dir, "decode_examples.json")) as f:
        return json.load(f)


def _gemv_case(dec):
    c = dec["gemv"]
    W = np.array([[_f(v) for v in row] for row in c["W"]], np.float32)
    x = np.array([[_f(v) for v in row] for row in c["x"]], np.float64)
    return c, W, x


# --------------------------------------------------------------------------
# Decode product and float16 scales
# --------------------------------------------------------------------------

def test_hand_gemv(dec):
    """W -> float32 scales -> float16 scales -> codes -> y, all by hand."""
    c, W, x = _gemv_case(dec)
    g, eps = c["g"], c["eps"]
    s32 = O.group_scales_f32(W, g)
    np.testing.assert_array_equal(s32, np.array([[_f(v) for v in r] for r in c["s32"]], np.float32))
    s16 = O.scales_f16(s32)
    np.testing.assert_array_equal(s16.astype(np.float64),
                                  np.array([[_f(v) for v in r] for r in c["s16"]]))
    q = O.ternary_codes(W, s32, g, eps)
    np.testing.assert_array_equal(q, np.array(c["codes"]))
    y = O.gemv(x, q, s16, g)
    np.testing.assert_array_equal(y, np.array([[_f(v) for v in r] for r in c["y"]]))
    # the twin's loops agree with the hand values
    assert brute.gemv(x.tolist(), q.tolist(), s16.astype(float).tolist(), g) == y.tolist()


def test_hand_gemv_bf16_input(dec):
    """The same product with x given as bfloat16 bit patterns (the kernel's input)."""
    c, W, x = _gemv_case(dec)
    s16 = O.scales_f16(O.group_scales_f32(W, c["g"]))
    q = O.ternary_codes(W, O.group_scales_f32(W, c["g"]), c["g"], c["eps"])
    xb = synth.f32_to_bf16_bits(x.astype(np.float32))
    np.testing.assert_array_equal(O.gemv(xb, q, s16, c["g"]), O.gemv(x, q, s16, c["g"]))


def test_f16_rounding_cases(dec):
    for src, want, why in dec["f16_rounding"]["cases"]:
        got = O.scales_f16(np.array([_f(src)], np.float32))[0]
        assert float(got) == _f(want), why
        assert brute.f16(_f(src)) == _f(want), why


def test_f16_rounding_against_twin():
    """numpy's conversion against binary16 rounding written from the format:
    random float32 over 2^-30 .. 2^20 (subnormal, normal and overflowing
    float16), plus every float32 within 3 ulps of each float16 midpoint in
    [1, 2) and in the subnormal range (where ties are decided)."""
    rng = np.random.default_rng(16)
    vals = (rng.standard_normal(4000).astype(np.float32)
            * np.exp2(rng.integers(-30, 21, 4000)).astype(np.float32))
    mids = []
    for base, spacing in ((1.0, 2.0 ** -10), (0.0, 2.0 ** -24)):
        for m in range(0, 60):
            mid = np.float32(base + (m + 0.5) * spacing)
            for d in (-3, -2, -1, 0, 1, 2, 3):
                mids.append(np.nextafter(mid, np.float32(np.inf) if d > 0 else np.float32(0))
                            if d else mid)
                for _ in range(abs(d) - 1):
                    mids[-1] = np.nextafter(mids[-1], np.float32(np.inf) if d > 0
                                            else np.float32(0))
    vals = np.concatenate([vals, np.array(mids, np.float32)])
    with np.errstate(over="ignore"):
        got = O.scales_f16(vals).astype(np.float64)
    twin = np.array([brute.f16(float(v)) for v in vals])
    np.testing.assert_array_equal(got, twin)


def test_decode_scales_round_twice(dec):
    """The stored float16 scale is the float16 of the float32 scale, which can
    differ from the float16 of the exact mean (row 0, group 1 of the hand case)."""
    c, W, _ = _gemv_case(dec)
    s64 = O.group_scales_f64(W, c["g"])
    s16 = O.scales_f16(O.group_scales_f32(W, c["g"]))
    assert float(s16[0, 1]) == 1.0
    assert brute.f16(s64[0, 1]) == 1 + 2 ** -10      # the single rounding differs


@pytest.mark.parametrize("g", [32, 128])
def test_gemv_against_twin_random(g):
    """Random decode shapes (B = 3, ragged N) against the fsum twin."""
    rng = np.random.default_rng(40 + g)
    N, K, B = 5, 256, 3
    W = synth.weights(rng, N, K, outliers=True)
    x = synth.activations(rng, B, K)
    s32 = O.group_scales_f32(W, g)
    s16 = O.scales_f16(s32)
    q = O.ternary_codes(W, s32, g, 1e-5)
    y = O.gemv(x, q, s16, g)
    xf = O.bf16_bits_to_f64(x)
    twin = np.array(brute.gemv(xf.tolist(), q.tolist(), s16.astype(float).tolist(), g))
    np.testing.assert_allclose(y, twin, rtol=1e-12, atol=1e-15)


def test_gemv_exact_cases():
    """One +1 code per row with scale 1 selects columns of x; integer x with
    unit scales gives exact integers; all-zero codes give exact zeros."""
    rng = np.random.default_rng(9)
    N, K, g = 12, 64, 32
    q = np.zeros((N, K), np.int8)
    cols = rng.integers(0, K, N)
    q[np.arange(N), cols] = 1
    s16 = np.ones((N, K // g), np.float16)
    x = rng.standard_normal((2, K))
    np.testing.assert_array_equal(O.gemv(x, q, s16, g), x[:, cols])
    qi = rng.integers(-1, 2, (N, K)).astype(np.int8)
    xi = rng.integers(-8, 9, (3, K)).astype(float)
    np.testing.assert_array_equal(O.gemv(xi, qi, s16, g), xi @ qi.T.astype(float))
    assert not O.gemv(x, np.zeros_like(q), s16, g).any()


# --------------------------------------------------------------------------
# Boundary band and the error measure
# --------------------------------------------------------------------------

def test_boundary_band_width_and_centre(dec):
    b = dec["boundary_band"]
    W = np.array(b["W"], np.float32)
    got = O.boundary_mask(W, np.array(b["s64"]), b["g"], b["eps"], b["rel"])
    np.testing.assert_array_equal(got, np.array(b["inside"]))


def test_boundary_band_expected_size():
    """For Gaussian weights the band holds 2 * pdf(t) * t * 2e-6 of the
    elements, t = half the absmean over sigma = sqrt(2/pi)/2 (~ 0.399): about
    5.9e-7, i.e. ~10 of an 8192 x 2048 matrix.  A band ten times too wide, or
    one centred away from the code's threshold, misses this count."""
    W = synth.weights(np.random.default_rng(12), 8192, 2048)
    band = int(O.boundary_mask(W, O.group_scales_f64(W, 128), 128, 1e-5).sum())
    t = 0.5 * math.sqrt(2 / math.pi)
    expect = 2 * (math.exp(-t * t / 2) / math.sqrt(2 * math.pi)) * t * 2e-6 * W.size
    assert expect / 4 <= band <= 3 * expect, (band, expect)


def test_rel_fro_error_cases(dec):
    for case in dec["rel_fro_error"]["cases"]:
        v = O.rel_fro_error(np.array(case["got"]), np.array(case["ref"]))
        want = case["value"]
        if want == "inf":
            assert v == float("inf"), case["why"]
        else:
            assert v == pytest.approx(want, rel=1e-12, abs=1e-300), case["why"]


# --------------------------------------------------------------------------
# Planted mistakes: each must be caught by a pin above
# --------------------------------------------------------------------------

_ORIG_GEMV = O.gemv
_ORIG_F16 = O.scales_f16
_ORIG_MASK = O.boundary_mask
_ORIG_S32 = O.group_scales_f32


def _caught(fn, *args):
    try:
        fn(*args)
    except (AssertionError, ValueError):
        return True
    return False


@pytest.mark.parametrize("mutant", ["s32_not_s16", "no_transpose", "batch_rows_swapped",
                                    "codes_abs", "f16_truncates", "f16_half_away",
                                    "f16_from_exact_mean", "f16_no_subnormals"])
def test_planted_decode_mistakes_are_caught(dec, mutant, monkeypatch):
    if mutant == "s32_not_s16":
        monkeypatch.setattr(O, "scales_f16", lambda s: np.asarray(s, np.float32))
    elif mutant == "no_transpose":
        monkeypatch.setattr(O, "gemv", lambda x, q, s, g: (
            O.bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, float))
            @ O.dequantize(q, np.asarray(s).astype(float), g))
    elif mutant == "batch_rows_swapped":
        monkeypatch.setattr(O, "gemv", lambda x, q, s, g: _ORIG_GEMV(x, q, s, g)[::-1])
    elif mutant == "codes_abs":
        monkeypatch.setattr(O, "gemv", lambda x, q, s, g: _ORIG_GEMV(x, np.abs(q), s, g))
    elif mutant == "f16_truncates":
        def trunc(s):
            b = np.asarray(s, np.float32).astype(np.float16)
            # round toward zero: step back where nearest rounding went up
            up = np.abs(b.astype(np.float64)) > np.abs(np.asarray(s, np.float64))
            return np.where(up, np.nextafter(b, np.float16(0)), b).astype(np.float16)
        monkeypatch.setattr(O, "scales_f16", trunc)
    elif mutant == "f16_half_away":
        def away(s):
            s = np.asarray(s, np.float32)
            b = s.astype(np.float16)
            out = b.copy()
            for i, (sv, bv) in enumerate(zip(s.astype(np.float64).ravel(), b.ravel())):
                other = np.nextafter(bv, np.float16(np.inf) if bv < sv else np.float16(-np.inf))
                if np.isfinite(other) and abs(float(other) - sv) == abs(float(bv) - sv) \
                        and abs(float(other)) > abs(float(bv)):
                    out.ravel()[i] = other
            return out
        monkeypatch.setattr(O, "scales_f16", away)
    elif mutant == "f16_from_exact_mean":
        monkeypatch.setattr(O, "group_scales_f32", lambda W, g: O.group_scales_f64(W, g))
        monkeypatch.setattr(O, "scales_f16", lambda s: np.asarray(s, np.float64).astype(np.float16))
    elif mutant == "f16_no_subnormals":
        def ftz(s):
            b = _ORIG_F16(s)
            return np.where(np.abs(b) < np.float16(2.0 ** -14), np.float16(0), b).astype(np.float16)
        monkeypatch.setattr(O, "scales_f16", ftz)
    pins = [lambda: test_hand_gemv(dec), lambda: test_f16_rounding_cases(dec),
            lambda: test_decode_scales_round_twice(dec)]
    assert any(_caught(p) for p in pins), f"mutant {mutant} escaped the pins"


@pytest.mark.parametrize("mutant", ["width_1e-5", "centre_s_half", "no_eps", "absolute_width"])
def test_planted_band_mistakes_are_caught(dec, mutant, monkeypatch):
    if mutant == "width_1e-5":
        monkeypatch.setattr(O, "boundary_mask",
                            lambda W, s, g, eps, rel=1e-6: _ORIG_MASK(W, s, g, eps, 1e-5))
    elif mutant == "centre_s_half":
        monkeypatch.setattr(O, "boundary_mask",
                            lambda W, s, g, eps, rel=1e-6: _ORIG_MASK(W, s, g, 0.0, rel))
    elif mutant == "no_eps":
        monkeypatch.setattr(O, "boundary_mask",
                            lambda W, s, g, eps, rel=1e-6: _ORIG_MASK(W, np.asarray(s) + eps,
                                                                       g, -eps, rel))
    elif mutant == "absolute_width":
        def absw(W, s, g, eps, rel=1e-6):
            N, K = np.asarray(W).shape
            half = 0.5 * (np.asarray(s, float).reshape(N, K // g) + eps)
            a = np.abs(np.asarray(W, float)).reshape(N, K // g, g)
            return (np.abs(a - half[:, :, None]) <= rel).reshape(N, K)
        monkeypatch.setattr(O, "boundary_mask", absw)
    assert _caught(test_boundary_band_width_and_centre, dec), f"mutant {mutant} escaped"


@pytest.mark.parametrize("mutant", ["no_sqrt", "relative_to_got", "max_abs"])
def test_planted_error_measure_mistakes_are_caught(dec, mutant, monkeypatch):
    def no_sqrt(got, ref):
        got, ref = np.asarray(got, float), np.asarray(ref, float)
        den = np.sum(ref * ref)
        return 0.0 if den == 0 and not np.any(got) else (
            float("inf") if den == 0 else float(np.sum((got - ref) ** 2) / den))

    def rel_got(got, ref):
        got, ref = np.asarray(got, float), np.asarray(ref, float)
        den = np.linalg.norm(got)
        return 0.0 if den == 0 else float(np.linalg.norm(got - ref) / den)

    def max_abs(got, ref):
        got, ref = np.asarray(got, float), np.asarray(ref, float)
        den = np.linalg.norm(ref)
        if den == 0:
            return 0.0 if not np.any(got) else float("inf")
        return float(np.max(np.abs(got - ref)) / den)

    monkeypatch.setattr(O, "rel_fro_error", {"no_sqrt": no_sqrt, "relative_to_got": rel_got,
                                             "max_abs": max_abs}[mutant])
    assert _caught(test_rel_fro_error_cases, dec), f"mutant {mutant} escaped"


# --------------------------------------------------------------------------
# Dense FP16 decode product (the layers kept unquantized)
# --------------------------------------------------------------------------

def _dense_case(dec):
    c = dec["dense_gemv"]
    W16 = np.array([[_f(v) for v in r] for r in c["W16"]], np.float16)
    x = np.array([[_f(v) for v in r] for r in c["x"]], np.float64)
    y = np.array([[_f(v) for v in r] for r in c["y"]])
    return W16, x, y


def test_hand_dense_gemv(dec):
    """Float16 subnormal, largest and smallest normal weights, exact in float64."""
    W16, x, y = _dense_case(dec)
    assert np.array_equal(W16.astype(np.float64),
                          np.array([[_f(v) for v in r] for r in dec["dense_gemv"]["W16"]]))
    np.testing.assert_array_equal(O.dense_gemv(x, W16), y)
    assert brute.dense_gemv(x.tolist(), W16.astype(float).tolist()) == y.tolist()
    xb = synth.f32_to_bf16_bits(x.astype(np.float32))
    np.testing.assert_array_equal(O.dense_gemv(xb, W16), y)


def test_dense_gemv_against_twin_random():
    rng = np.random.default_rng(77)
    W16 = (rng.standard_normal((7, 192)) * 0.02).astype(np.float16)
    x = synth.activations(rng, 3, 192)
    twin = np.array(brute.dense_gemv(O.bf16_bits_to_f64(x).tolist(), W16.astype(float).tolist()))
    np.testing.assert_allclose(O.dense_gemv(x, W16), twin, rtol=1e-12, atol=1e-15)
    # one-hot rows select weight columns exactly
    eye = np.eye(192)[:5]
    np.testing.assert_array_equal(O.dense_gemv(eye, W16), W16.astype(np.float64)[:, :5].T)
    with pytest.raises(ValueError):
        O.dense_gemv(x, W16.astype(np.float32))


_ORIG_DENSE = O.dense_gemv


@pytest.mark.parametrize("mutant", ["no_transpose", "batch_rows_swapped", "weights_bf16",
                                    "x_as_float16"])
def test_planted_dense_mistakes_are_caught(dec, mutant, monkeypatch):
    if mutant == "no_transpose":
        monkeypatch.setattr(O, "dense_gemv", lambda x, W: (
            O.bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, float))
            @ np.asarray(W, np.float64))
    elif mutant == "batch_rows_swapped":
        monkeypatch.setattr(O, "dense_gemv", lambda x, W: _ORIG_DENSE(x, W)[::-1])
    elif mutant == "weights_bf16":
        def wbf(x, W):
            Wb = O.bf16_bits_to_f64(synth.f32_to_bf16_bits(np.asarray(W, np.float32)))
            xf = O.bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, float)
            return xf @ Wb.T
        monkeypatch.setattr(O, "dense_gemv", wbf)
    elif mutant == "x_as_float16":
        def xf16(x, W):
            xf = O.bf16_bits_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, float)
            with np.errstate(over="ignore"):
                return xf.astype(np.float16).astype(np.float64) @ np.asarray(W, np.float64).T
        monkeypatch.setattr(O, "dense_gemv", xf16)
    assert _caught(test_hand_dense_gemv, dec), f"mutant {mutant} escaped"
