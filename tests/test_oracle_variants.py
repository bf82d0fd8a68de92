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
