"""Pins of the CPU oracle against things other than itself.

Hand-worked dyadic examples (tests/golden/hand_examples.json), the
pure-Python twin (a different formulation of every step), exhaustive small
grids, closed forms for Gaussian weights, invariants, special cases that
reduce to exact arithmetic, and the paper's printed storage numbers.  The
last block plants plausible mistakes in copies of the oracle and checks that
a pin catches each one.
"""

import json
import math
import os

import numpy as np
import pytest
from scipy import integrate
from scipy.stats import norm

from oracle import brute
from oracle import ternary as O
from paper_2606_18114_amd import synth


@pytest.fixture(scope="module")
def hand(golden_dir):
    with open(os.path.join(golden_dir, "hand_examples.json")) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# Hand-worked examples
# --------------------------------------------------------------------------

def test_hand_examples_quantizer(hand):
    for ex in hand["examples"]:
        W = np.array(ex["W"], dtype=np.float32)
        g, eps = ex["g"], ex["eps"]
        s64, s32, q, z = O.ternarize(W, g, eps)
        np.testing.assert_array_equal(s64, np.array(ex["scales"]), err_msg=ex["name"])
        np.testing.assert_array_equal(s32, np.array(ex["scales"], np.float32))
        np.testing.assert_array_equal(q, np.array(ex["codes"]), err_msg=ex["name"])
        np.testing.assert_array_equal(O.dequantize(q, s32, g), np.array(ex["What"]))
        assert z == ex["zero_count"], ex["name"]
        if "nrmse_squared" in ex:
            num, den = ex["nrmse_squared"]
            assert O.nrmse(W, q, s32, g) == pytest.approx(math.sqrt(num / den), rel=1e-15)
        if "Y" in ex:
            X = np.array(ex["X"])
            np.testing.assert_array_equal(O.gemm_fwd(X, q, s32, g), np.array(ex["Y"]))


def test_hand_examples_twin(hand):
    for ex in hand["examples"]:
        s = brute.scales(ex["W"], ex["g"])
        assert s == ex["scales"], ex["name"]
        assert brute.codes(ex["W"], s, ex["g"], ex["eps"]) == ex["codes"], ex["name"]


def test_hand_linear_maps(hand):
    lm = hand["linear_maps"]
    W = np.array(lm["W"], dtype=np.float32)
    _, s32, q, _ = O.ternarize(W, lm["g"], lm["eps"])
    X, dY = np.array(lm["X"]), np.array(lm["dY"])
    np.testing.assert_array_equal(O.gemm_fwd(X, q, s32, lm["g"]), np.array(lm["Y"]))
    np.testing.assert_array_equal(O.gemm_bwd_dx(dY, q, s32, lm["g"]), np.array(lm["dX"]))
    np.testing.assert_array_equal(O.gemm_bwd_dw(dY, X), np.array(lm["dW"]))
    # the twin's loops agree
    s = s32.tolist()
    ql = q.tolist()
    assert brute.gemm(lm["X"], ql, s, lm["g"]) == lm["Y"]
    assert brute.gemm_dx(lm["dY"], ql, s, lm["g"]) == lm["dX"]
    assert brute.gemm_dw(lm["dY"], lm["X"]) == lm["dW"]


def test_hand_packing(hand):
    p = hand["packing"]
    q = np.array([p["codes"]], dtype=np.int8)
    assert O.pack(q).tolist() == [p["bytes"]]
    assert brute.pack_row(p["codes"]) == p["bytes"]
    np.testing.assert_array_equal(O.unpack(O.pack(q), 16), q)


def test_unpack_rejects_unused_code():
    bad = np.zeros((1, 4), dtype=np.uint8)
    bad[0, 0] = 0b10
    with pytest.raises(ValueError):
        O.unpack(bad, 16)


# --------------------------------------------------------------------------
# Vectorized oracle vs pure-Python twin
# --------------------------------------------------------------------------

@pytest.mark.parametrize("eps", [0.0, 0.25])
def test_exhaustive_four_element_groups(eps):
    """Every group of four values from {-2, -1.75, ..., 2}: 17^4 = 83521 groups,
    dense with exact ties at eps = 0."""
    grid = np.arange(-8, 9, dtype=np.float32) * np.float32(0.25)
    W = np.stack(np.meshgrid(grid, grid, grid, grid, indexing="ij"), -1).reshape(-1, 4)
    s64, s32, q, _ = O.ternarize(W, 4, eps)
    s_twin = brute.scales(W.tolist(), 4)
    np.testing.assert_array_equal(s32, np.array(s_twin, np.float32))
    q_twin = np.array(brute.codes(W.tolist(), s_twin, 4, eps), dtype=np.int8)
    np.testing.assert_array_equal(q, q_twin)


@pytest.mark.parametrize("g", synth.C5_GROUPS)
def test_random_rows_against_twin(g):
    rng = np.random.default_rng(100 + g)
    W = synth.weights(rng, 3, 1024, outliers=True)
    s64, s32, q, z = O.ternarize(W, g, 1e-5)
    s_twin = brute.scales(W.tolist(), g)
    np.testing.assert_array_equal(s32, np.array(s_twin, np.float32))
    q_twin = brute.codes(W.tolist(), s_twin, g, 1e-5)
    np.testing.assert_array_equal(q, np.array(q_twin, np.int8))
    packed = O.pack(q)
    for n in range(3):
        assert packed[n].tolist() == brute.pack_row(q_twin[n])


def test_gemm_triple_loop_small():
    """A C1-shaped slice: 3 tokens x 256 inputs -> 8 outputs, fsum loops."""
    rng = np.random.default_rng(7)
    W = synth.weights(rng, 8, 256)
    X = synth.activations(rng, 3, 256)
    dY = synth.activations(rng, 3, 8, std=0.01)
    _, s32, q, _ = O.ternarize(W, 32, 1e-5)
    Xf = synth.bf16_bits_to_f32(X).astype(float)
    dYf = synth.bf16_bits_to_f32(dY).astype(float)
    ql, sl = q.tolist(), s32.astype(float).tolist()
    np.testing.assert_allclose(O.gemm_fwd(X, q, s32, 32),
                               np.array(brute.gemm(Xf.tolist(), ql, sl, 32)), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(O.gemm_bwd_dx(dY, q, s32, 32),
                               np.array(brute.gemm_dx(dYf.tolist(), ql, sl, 32)), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(O.gemm_bwd_dw(dY, X),
                               np.array(brute.gemm_dw(dYf.tolist(), Xf.tolist())), rtol=1e-12, atol=1e-15)


# --------------------------------------------------------------------------
# Invariants (Sec. 3.1 definitions)
# --------------------------------------------------------------------------

@pytest.fixture(scope="module")
def rand_w():
    return synth.weights(np.random.default_rng(11), 64, 512, outliers=True)


@pytest.mark.parametrize("g", [32, 128, 512])
def test_invariants(rand_w, g):
    W, eps = rand_w, 1e-5
    s64, s32, q, z = O.ternarize(W, g, eps)
    assert set(np.unique(q)) <= {-1, 0, 1}
    N, K = W.shape
    s_full = np.repeat(s32.astype(np.float64), g, axis=1)
    d_full = np.repeat((s32 + np.float32(eps)).astype(np.float64), g, axis=1)
    a = np.abs(W.astype(np.float64))
    # zero ratio identity with the same divisor as the rounding
    assert z == int(np.count_nonzero(a / d_full <= 0.5 * (1 + 2.0 ** -24)))
    # error bound |W - q s| <= s/2 + eps wherever |W/s| <= 1.5 (a few ulps slack)
    err = np.abs(W - q * s_full)
    dom = a / s_full <= 1.5
    assert np.all(err[dom] <= (s_full / 2 + eps)[dom] * (1 + 1e-6))
    # sign symmetry
    _, s2, q2, _ = O.ternarize(-W, g, eps)
    np.testing.assert_array_equal(s2, s32)
    np.testing.assert_array_equal(q2, -q)
    # groups are independent: shuffling whole groups permutes scales and codes
    perm = np.random.default_rng(3).permutation(K // g)
    Wp = W.reshape(N, K // g, g)[:, perm].reshape(N, K)
    _, sp, qp, _ = O.ternarize(Wp, g, eps)
    np.testing.assert_array_equal(sp, s32[:, perm])
    np.testing.assert_array_equal(qp, q.reshape(N, K // g, g)[:, perm].reshape(N, K))
    # a permutation inside each group permutes the codes
    ip = np.random.default_rng(4).permutation(g)
    Wi = W.reshape(N, K // g, g)[:, :, ip].reshape(N, K)
    _, si, qi, _ = O.ternarize(Wi, g, eps)
    np.testing.assert_allclose(si, s32, rtol=2 ** -23)   # sum order changes
    np.testing.assert_array_equal(qi, q.reshape(N, K // g, g)[:, :, ip].reshape(N, K))
    # pack / unpack round trip
    np.testing.assert_array_equal(O.unpack(O.pack(q), K), q)


def test_power_of_two_equivariance(rand_w):
    W = rand_w
    _, s, q, _ = O.ternarize(W, 128, 0.0)
    for k in (-3, 5):
        _, sk, qk, _ = O.ternarize(W * np.float32(2.0 ** k), 128, 0.0)
        np.testing.assert_array_equal(sk, s * np.float32(2.0 ** k))
        np.testing.assert_array_equal(qk, q)


def test_boundary_mask_flags_exact_ties():
    W = np.array([[1.5, -0.5, 0.25, -1.75]], np.float32)
    s64 = O.group_scales_f64(W, 4)
    np.testing.assert_array_equal(O.boundary_mask(W, s64, 4, 0.0), [[False, True, False, False]])


# --------------------------------------------------------------------------
# Special cases
# --------------------------------------------------------------------------

@pytest.mark.parametrize("eps", [0.0, 1e-5])
def test_special_groups(eps):
    g = 32
    W = np.zeros((4, 2 * g), np.float32)
    W[1, :g] = 0.03                       # constant group
    W[2, 5] = -0.7                        # single nonzero in group 0
    W[3, g:] = np.float32(2.0 ** -140)    # subnormal constant group
    s64, s, q, _ = O.ternarize(W, g, eps)
    assert s[0].tolist() == [0.0, 0.0] and not q[0].any()      # all-zero group
    assert s[1, 0] == np.float32(0.03) and np.all(q[1, :g] == 1)
    np.testing.assert_array_equal(O.dequantize(q[1:2], s[1:2], g)[0, :g], W[1, :g])
    assert s[2, 0] == np.float32(np.float64(np.float32(0.7)) / g)
    assert q[2, 5] == -1 and np.count_nonzero(q[2]) == 1
    # the all-zero rows give exactly zero outputs
    X = synth.activations(np.random.default_rng(0), 3, 2 * g)
    assert not O.gemm_fwd(X, q[:1], s[:1], g).any()


def test_one_hot_and_integer_inputs():
    rng = np.random.default_rng(5)
    N, K, g = 16, 64, 32
    q = rng.integers(-1, 2, (N, K)).astype(np.int8)
    s = np.ones((N, K // g), np.float32)
    # one-hot token rows select columns of What
    X = np.zeros((K, K)); X[np.arange(K), np.arange(K)] = 1
    np.testing.assert_array_equal(O.gemm_fwd(X, q, s, g), q.T.astype(float))
    # small integer activations give exact integers
    Xi = rng.integers(-8, 9, (5, K)).astype(float)
    Y = O.gemm_fwd(Xi, q, s, g)
    np.testing.assert_array_equal(Y, Xi @ q.T.astype(float))
    # one-hot token rows in dW copy dY columns
    dY = rng.standard_normal((K, N))
    np.testing.assert_array_equal(O.gemm_bwd_dw(dY, X), dY.T)


# --------------------------------------------------------------------------
# Closed forms for Gaussian weights
# --------------------------------------------------------------------------

def _gaussian_closed_forms():
    """Zero ratio and NRMSE of absmean ternarization of N(0,1) weights when
    the group mean equals its expectation sqrt(2/pi) (g -> infinity)."""
    s = math.sqrt(2 / math.pi)
    t = s / 2
    zr = 2 * norm.cdf(t) - 1
    e_in = 2 * integrate.quad(lambda w: w * w * norm.pdf(w), 0, t)[0]
    e_out = 2 * integrate.quad(lambda w: (w - s) ** 2 * norm.pdf(w), t, np.inf)[0]
    return zr, math.sqrt(e_in + e_out)


def test_gaussian_closed_forms():
    zr, e = _gaussian_closed_forms()
    W = np.random.default_rng(21).standard_normal((512, 4096), dtype=np.float32)
    _, s, q, z = O.ternarize(W, 512, 0.0)
    assert z / W.size == pytest.approx(zr, abs=1.5e-3)          # 0.31006
    assert O.nrmse(W, q, s, 512) == pytest.approx(e, abs=2e-3)  # 0.51321
    # smaller groups: noisier scales, slightly fewer zeros
    _, s32_, q32_, z32 = O.ternarize(W, 32, 0.0)
    assert zr - 0.01 < z32 / W.size < zr


# --------------------------------------------------------------------------
# Storage arithmetic against the paper's printed numbers
# --------------------------------------------------------------------------

def test_storage_size_against_paper(golden_dir):
    with open(os.path.join(golden_dir, "paper_numbers.json")) as f:
        p = json.load(f)
    quant = p["params_M"]["in_proj_x48"] + p["params_M"]["out_proj_x48"]
    assert quant == p["params_M"]["total_quantized"]
    rest = p["params_M"]["embedding_lm_head"] + p["params_M"]["ssm_norms_conv"]
    g = p["memory_MB"]["group_size"]
    # the oracle's format: K/4 bytes of codes per row, one float16 per group
    q = np.zeros((1, 1024), np.int8)
    code_bytes_per_w = O.pack(q).nbytes / q.size
    s16_bytes_per_w = O.scales_f16(np.zeros(1024 // g, np.float32)).nbytes / q.size
    ours = quant * (code_bytes_per_w + s16_bytes_per_w) + rest * 2
    fp32_scales = quant * (code_bytes_per_w + 4 / g) + rest * 2
    paper = p["memory_MB"]["ternary_packed_projected"]
    assert abs(ours - paper) / paper < 0.01
    assert abs(ours - paper) < abs(fp32_scales - paper)
    assert p["memory_MB"]["fp16_abstract"] / paper == pytest.approx(
        p["memory_MB"]["compression_ratio"], abs=0.005)


# --------------------------------------------------------------------------
# Planted mistakes: each must be caught by a pin above
# --------------------------------------------------------------------------

def _codes_half_away(W, s32, g, eps):
    N, K = W.shape
    d = (np.asarray(s32, np.float32) + np.float32(eps)).astype(np.float32)
    x = np.clip(W.reshape(N, K // g, g) / d[:, :, None], -1, 1)
    return (np.sign(x) * np.floor(np.abs(x) + 0.5)).reshape(N, K).astype(np.int8)


_ORIG_CODES = O.ternary_codes
_ORIG_SCALES = O.group_scales_f64


def _codes_no_eps(W, s32, g, eps):
    return _ORIG_CODES(W, s32, g, 0.0)


def _scales_sum_not_mean(W, g):
    return _ORIG_SCALES(W, g) * g


@pytest.mark.parametrize("mutant", ["half_away", "no_eps", "sum_not_mean", "sign_flip_pack"])
def test_planted_mistakes_are_caught(hand, mutant, monkeypatch):
    def quant_pins_pass():
        try:
            test_hand_examples_quantizer(hand)
            test_hand_packing(hand)
            test_exhaustive_four_element_groups(0.0)
            return True
        except AssertionError:
            return False

    if mutant == "half_away":
        monkeypatch.setattr(O, "ternary_codes", _codes_half_away)
    elif mutant == "no_eps":
        monkeypatch.setattr(O, "ternary_codes", _codes_no_eps)
    elif mutant == "sum_not_mean":
        monkeypatch.setattr(O, "group_scales_f64", _scales_sum_not_mean)
    elif mutant == "sign_flip_pack":
        orig = O.pack
        monkeypatch.setattr(O, "pack", lambda q: orig(-np.asarray(q)))
    assert not quant_pins_pass(), f"mutant {mutant} escaped the pins"


@pytest.mark.parametrize("mutant", ["fwd_no_scale", "dx_no_scale", "dw_swapped", "dx_rows_reversed"])
def test_planted_linear_map_mistakes_are_caught(hand, mutant, monkeypatch):
    orig_fwd, orig_dx, orig_dw = O.gemm_fwd, O.gemm_bwd_dx, O.gemm_bwd_dw
    if mutant == "fwd_no_scale":
        monkeypatch.setattr(O, "gemm_fwd", lambda X, q, s, g: orig_fwd(X, q, np.ones_like(s), g))
    elif mutant == "dx_no_scale":
        monkeypatch.setattr(O, "gemm_bwd_dx", lambda dY, q, s, g: orig_dx(dY, q, np.ones_like(s), g))
    elif mutant == "dw_swapped":
        monkeypatch.setattr(O, "gemm_bwd_dw", lambda dY, X: orig_dw(X, dY))
    elif mutant == "dx_rows_reversed":
        monkeypatch.setattr(O, "gemm_bwd_dx", lambda dY, q, s, g: orig_dx(dY, q[::-1], s[::-1], g))
    with pytest.raises(AssertionError):
        test_hand_linear_maps(hand)
