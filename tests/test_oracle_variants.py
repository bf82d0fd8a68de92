"""Pins of the variant oracle (threshold multiplier, group-magnitude gradient).

Each check ties ``oracle/variants.py`` to something other than itself: the
hand-worked dyadic examples of ``tests/golden/variant_examples.json``, the
pure-Python twin with exact rational thresholds, the standard code it must
reduce to, monotonicity in the multiplier, and PyTorch's CPU autograd for the
gradient of a per-group magnitude.  Planted mistakes must fail a pin.
"""

import json
import os

import numpy as np
import pytest

from oracle import brute as BR
from oracle import ternary as T
from oracle import variants as V


@pytest.fixture(scope="module")
def ex(golden_dir):
    with open(os.path.join(golden_dir, "variant_examples.json")) as f:
        return json.load(f)


def test_hand_threshold_examples(ex):
    e = ex["threshold_multiplier"]
    W = np.array([e["W"]], np.float32)
    s = np.array([[e["scale"]]], np.float32)
    assert T.group_scales_f32(W, 4)[0, 0] == np.float32(e["scale"])
    for c in e["cases"]:
        q = V.ternary_codes_thresh(W, s, 4, 0.0, np.array([c["mult"]], np.float32))
        assert q.tolist() == [c["q"]], c
        assert BR.codes_thresh(W.tolist(), s.tolist(), 4, 0.0, [c["mult"]]) == [c["q"]], c


def test_hand_group_dot(ex):
    e = ex["group_code_dot"]
    q = np.array([e["q"]], np.int8)
    d = np.array([e["dWhat"]], np.float64)
    assert V.group_code_dot(q, d, 4)[0, 0] == e["dalpha"]
    assert BR.group_code_dot(q.tolist(), d.tolist(), 4) == [[e["dalpha"]]]


def _check_twin(g, eps):
    rng = np.random.default_rng(g)
    W = (rng.standard_normal((6, 2 * g)) * 0.02).astype(np.float32)
    W[0, :7] = 0.0
    s32 = T.group_scales_f32(W, g)
    mult = np.array([0.8, 1.0, 0.5, 1.25, 0.8, 3.0], np.float32)
    q = V.ternary_codes_thresh(W, s32, g, eps, mult)
    assert q.tolist() == BR.codes_thresh(W.tolist(), s32.tolist(), g, eps, mult.tolist())


@pytest.mark.parametrize("g", [32, 128])
@pytest.mark.parametrize("eps", [0.0, 1e-5, 5e-3])
def test_threshold_codes_against_twin(g, eps):
    _check_twin(g, eps)


def test_unit_multiplier_is_the_standard_code():
    rng = np.random.default_rng(3)
    W = (rng.standard_normal((40, 512)) * 0.02).astype(np.float32)
    for g in (32, 128, 512):
        s32 = T.group_scales_f32(W, g)
        q = V.ternary_codes_thresh(W, s32, g, 1e-5, np.ones(40, np.float32))
        assert np.array_equal(q, T.ternary_codes(W, s32, g, 1e-5))


def test_zeros_grow_with_the_multiplier():
    rng = np.random.default_rng(4)
    W = (rng.standard_normal((64, 1024)) * 0.02).astype(np.float32)
    s32 = T.group_scales_f32(W, 128)
    zeros = [T.zero_count(V.ternary_codes_thresh(W, s32, 128, 1e-5, np.full(64, m, np.float32)))
             for m in (0.5, 0.8, 1.0, 1.2, 2.0)]
    assert zeros == sorted(zeros) and zeros[0] < zeros[-1]
    # the gate setting of the paper (0.8 x absmean) lowers the zero ratio of
    # Gaussian weights from about 0.31 to about 0.25 (2 Phi(0.4 sqrt(2/pi)) - 1)
    from scipy.stats import norm
    closed = 2 * norm.cdf(0.4 * np.sqrt(2 / np.pi)) - 1
    assert abs(zeros[1] / W.size - closed) < 0.01


def test_group_dot_is_the_autograd_gradient_of_the_magnitude():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    N, K, g = 12, 256, 64
    q = rng.integers(-1, 2, (N, K)).astype(np.int8)
    G = rng.standard_normal((N, K))
    alpha = torch.tensor(rng.random((N, K // g)) + 0.1, dtype=torch.float64, requires_grad=True)
    What = alpha.repeat_interleave(g, dim=1) * torch.from_numpy(q.astype(np.float64))
    (What * torch.from_numpy(G)).sum().backward()
    assert np.allclose(alpha.grad.numpy(), V.group_code_dot(q, G, g), rtol=1e-12, atol=1e-12)
    assert np.allclose(V.group_code_dot(q, G, g),
                       np.array(BR.group_code_dot(q.tolist(), G.tolist(), g)), rtol=1e-12)


@pytest.mark.parametrize("mutant", ["abs_codes", "drop_neg", "mult_after_eps"])
def test_planted_variant_mistakes_are_caught(ex, mutant, monkeypatch):
    e = ex
    if mutant == "abs_codes":
        monkeypatch.setattr(V, "group_code_dot", lambda q, d, g: (
            np.abs(np.asarray(q, np.float64)) * np.asarray(d, np.float64)
        ).reshape(np.asarray(q).shape[0], -1, g).sum(2))
        with pytest.raises(AssertionError):
            test_hand_group_dot(e)
    elif mutant == "drop_neg":
        orig = V.group_code_dot
        monkeypatch.setattr(V, "group_code_dot",
                            lambda q, d, g: orig(np.maximum(np.asarray(q), 0), d, g))
        with pytest.raises(AssertionError):
            test_hand_group_dot(e)
    else:
        # multiplying s + eps instead of s changes decisions once eps matters
        orig = T.ternary_codes

        def wrong(W, s32, g, eps, row_mult):
            N = np.asarray(W).shape[0]
            m = np.asarray(row_mult, np.float32).reshape(N, 1)
            d = (m * (np.asarray(s32, np.float32) + np.float32(eps))).astype(np.float32)
            return orig(W, d, g, 0.0)
        monkeypatch.setattr(V, "ternary_codes_thresh", wrong)
        with pytest.raises(AssertionError):
            _check_twin(32, 5e-3)  # an eps comparable to the scales


# --------------------------------------------------------------------------
# Learnable scale with the straight-through rounding (scale_ste_grad)
# --------------------------------------------------------------------------

def _ste_case(ex, case):
    e = ex["scale_ste_grad"]
    W = np.array([e["W"]], np.float32)
    s = np.array([[case["s"]]], np.float32)
    q = T.ternary_codes(W, s, 4, case["eps"])
    return W, s, q, np.array([e["dWhat"]])


def test_hand_scale_ste_grad(ex):
    for case in ex["scale_ste_grad"]["cases"]:
        W, s, q, dwh = _ste_case(ex, case)
        assert q[0].tolist() == case["q"], case["why"]
        ds, dw = V.scale_ste_grad(W, q, s, dwh, 4, case["eps"])
        assert ds[0, 0] == case["ds"], case["why"]
        assert dw[0].tolist() == case["dw"], case["why"]


@pytest.mark.parametrize("g,eps", [(32, 0.0), (128, 1e-5), (64, 3e-3)])
def test_scale_ste_grad_is_pytorch_autograd(g, eps):
    """CPU autograd of the layer written the usual PyTorch way, in float64:
    x = clamp(w / (s + eps), -1, 1); q = x + (round(x) - x).detach();
    What = s * q.  Weights and scales are drawn so that no quotient lies
    within 1e-9 of a rounding or clip boundary, where float32 and float64
    decisions could differ."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(60 + g)
    N, K = 6, 512
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    s32 = (np.abs(W).reshape(N, K // g, g).mean(axis=2) * rng.uniform(0.6, 1.6, (N, K // g))
           ).astype(np.float32)
    d = np.repeat((s32 + np.float32(eps)).astype(np.float64), g, axis=1)
    x = np.abs(W.astype(np.float64)) / d
    assert np.min(np.abs(x - 0.5)) > 1e-9 and np.min(np.abs(x - 1.0)) > 1e-9
    G = rng.standard_normal((N, K))
    wt = torch.tensor(W.astype(np.float64), requires_grad=True)
    st = torch.tensor(s32.astype(np.float64), requires_grad=True)
    sf = st.repeat_interleave(g, dim=1)
    # s + eps as the float32 layer forms it: the float32 rounding of the sum is
    # added as a constant, so d(s + eps)/ds stays exactly 1 in float64
    d32 = (s32 + np.float32(eps)).astype(np.float32).astype(np.float64)
    delta = torch.from_numpy(np.repeat(d32 - s32.astype(np.float64), g, axis=1))
    dt = sf + delta
    xt = torch.clamp(wt / dt, -1.0, 1.0)
    qt = xt + (torch.round(xt) - xt).detach()
    (sf * qt * torch.from_numpy(G)).sum().backward()
    q = T.ternary_codes(W, s32, g, eps)
    assert np.array_equal(q, torch.round(xt).detach().numpy().astype(np.int8))
    ds, dw = V.scale_ste_grad(W, q, s32, G, g, eps)
    np.testing.assert_allclose(ds, st.grad.numpy(), rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-9, atol=1e-15)
    # the magnitude-only reading differs by the threshold term
    assert not np.allclose(V.group_code_dot(q, G, g), ds, rtol=1e-3)


_ORIG_STE = V.scale_ste_grad


@pytest.mark.parametrize("mutant", ["magnitude_only", "threshold_sign", "no_mask",
                                    "strict_mask", "no_eps_in_factor", "unmasked_dw"])
def test_planted_scale_ste_mistakes_are_caught(ex, mutant, monkeypatch):
    def mutated(W, q, s32, dWhat, g, eps):
        ds, dw = _ORIG_STE(W, q, s32, dWhat, g, eps)
        N, K = np.asarray(W).shape
        s64 = np.repeat(np.asarray(s32, np.float64).reshape(N, K // g), g, axis=1)
        d64 = np.repeat((np.asarray(s32, np.float32) + np.float32(eps)).astype(np.float64)
                        .reshape(N, K // g), g, axis=1)
        w = np.asarray(W, np.float64)
        m = (np.abs(np.asarray(W, np.float32)) / d64.astype(np.float32) <= 1).astype(float)
        dwh = np.asarray(dWhat, np.float64)
        qf = np.asarray(q, np.float64)
        if mutant == "magnitude_only":
            return V.group_code_dot(q, dWhat, g), dw
        if mutant == "threshold_sign":
            t = dwh * (qf + m * s64 * w / d64 ** 2)
        elif mutant == "no_mask":
            t = dwh * (qf - s64 * w / d64 ** 2)
        elif mutant == "strict_mask":
            ms = (np.abs(np.asarray(W, np.float32)) / d64.astype(np.float32) < 1).astype(float)
            t = dwh * (qf - ms * s64 * w / d64 ** 2)
            return t.reshape(N, K // g, g).sum(axis=2), dwh * ms * s64 / d64
        elif mutant == "no_eps_in_factor":
            t = dwh * (qf - m * w / s64)
            return t.reshape(N, K // g, g).sum(axis=2), dwh * m
        elif mutant == "unmasked_dw":
            return ds, dwh * s64 / d64
        return t.reshape(N, K // g, g).sum(axis=2), dw

    monkeypatch.setattr(V, "scale_ste_grad", mutated)
    with pytest.raises(AssertionError):
        test_hand_scale_ste_grad(ex)
