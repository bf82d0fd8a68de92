"""Pins of the Mamba-2 mixer decode-step oracle (oracle/mamba.py): a
hand-worked step whose output has a closed form, special cases (identity and
oldest-tap convolutions, a decay of zero, a vanishing step size), scale
invariance of the gated normalization, a pure-Python loop twin, and planted
mistakes that a pin must catch."""

import math

import numpy as np
import pytest

from oracle import brute
from oracle import mamba as MB

L3, LN2 = math.log(3.0), math.log(2.0)


def hand_case():
    """B = 1, one head of 2 channels, d_state 2, d_conv 4.  Every conv channel
    has taps [0, 0, 0, 1] (the newest input only) and no bias; dt = dt_bias =
    0 gives dt' = ln 2, A_log = 0 gives A = -1, so the decay is exactly 1/2."""
    xbc = [L3, -L3, L3, 0.0, L3, L3]              # x (2), B (2), C (2)
    zxbcdt = np.array([[0.0, L3] + xbc + [0.0]])  # z = [0, ln 3], dt = 0
    conv_state = np.array([[[c, c + 0.5, c + 0.25, c + 0.125] for c in range(6)]],
                          np.float16)
    ssm_state = np.array([[[[1.0, 2.0], [-1.0, 0.5]]]], np.float16)
    conv_w = np.tile(np.array([0.0, 0.0, 0.0, 1.0], np.float32), (6, 1))
    conv_b = np.zeros(6, np.float32)
    return dict(zxbcdt=zxbcdt, conv_state=conv_state, ssm_state=ssm_state, conv_w=conv_w,
                conv_b=conv_b, dt_bias=np.zeros(1, np.float32), A_log=np.zeros(1, np.float32),
                D=np.ones(1, np.float32), norm_w=np.ones(2, np.float32), eps=0.0, headdim=2,
                d_state=2)


def test_hand_step():
    """By hand: SiLU(ln 3) = 3/4 ln 3 and SiLU(-ln 3) = -1/4 ln 3, so
    x = [3L/4, -L/4], B = [3L/4, 0], C = [3L/4, 3L/4] (L = ln 3).  New state
    = 1/2 old + ln2 x B^T; y = state C + x; z = [0, ln 3] gates y[0] to 0, so
    the normalized output is [0, sign(y1) sqrt(2)] = [0, -sqrt 2]."""
    c = hand_case()
    out, conv_new, ssm_new = MB.mixer_step(**c)
    x0, x1, b0, cc = 0.75 * L3, -0.25 * L3, 0.75 * L3, 0.75 * L3
    s = np.array([[0.5 + LN2 * x0 * b0, 1.0], [-0.5 + LN2 * x1 * b0, 0.25]])
    assert np.array_equal(ssm_new[0, 0], s.astype(np.float16))
    y1 = cc * (s[1, 0] + s[1, 1]) + x1
    assert y1 < 0
    np.testing.assert_allclose(out, [[0.0, -math.sqrt(2.0)]], rtol=1e-14, atol=1e-15)
    # the conv window moved by one and took the new input (rounded to float16)
    for ch in range(6):
        assert conv_new[0, ch, :3].tolist() == [ch + 0.5, ch + 0.25, ch + 0.125]
        assert conv_new[0, ch, 3] == np.float16(c["zxbcdt"][0, 2 + ch])
    # the intermediate readout by hand, too
    z, xBC, dt = MB.split_in_proj(c["zxbcdt"], 2, 2, 1)
    u, _ = MB.conv_step(c["conv_state"], xBC, c["conv_w"], c["conv_b"])
    np.testing.assert_allclose(u[0], [0.75 * L3, -0.25 * L3, 0.75 * L3, 0.0, 0.75 * L3,
                                      0.75 * L3], rtol=1e-15)
    y, _ = MB.ssm_step(c["ssm_state"], u[:, :2].reshape(1, 1, 2), u[:, 2:4], u[:, 4:], dt,
                       c["dt_bias"], c["A_log"], c["D"])
    s16 = c["ssm_state"][0, 0].astype(np.float64)
    ref = [cc * ((0.5 * s16[p] + LN2 * [x0, x1][p] * np.array([b0, 0.0])).sum()) + [x0, x1][p]
           for p in range(2)]
    np.testing.assert_allclose(y[0, 0], ref, rtol=1e-14)


def test_closed_forms_of_the_scalar_functions():
    assert MB.softplus(np.array(0.0)) == pytest.approx(LN2, rel=1e-15)
    assert MB.softplus(np.array(40.0)) == 40.0
    assert MB.softplus(np.array(-30.0)) == pytest.approx(math.exp(-30.0), rel=1e-12)
    assert MB.silu(np.array(L3)) == pytest.approx(0.75 * L3, rel=1e-15)
    assert MB.silu(np.array(-L3)) == pytest.approx(-0.25 * L3, rel=1e-15)
    assert MB.silu(np.array(0.0)) == 0.0


def _random_case(rng, B=2, nheads=3, headdim=4, d_state=5, eps=1e-5):
    d_inner = nheads * headdim
    conv_dim = d_inner + 2 * d_state
    return dict(
        zxbcdt=rng.standard_normal((B, d_inner + conv_dim + nheads)),
        conv_state=rng.standard_normal((B, conv_dim, 4)).astype(np.float16),
        ssm_state=(rng.standard_normal((B, nheads, headdim, d_state)) * 0.5).astype(np.float16),
        conv_w=(rng.standard_normal((conv_dim, 4)) * 0.5).astype(np.float32),
        conv_b=(rng.standard_normal(conv_dim) * 0.1).astype(np.float32),
        dt_bias=rng.uniform(-4, -1, nheads).astype(np.float32),
        A_log=np.log(rng.uniform(1, 16, nheads)).astype(np.float32),
        D=rng.uniform(0.5, 1.5, nheads).astype(np.float32),
        norm_w=rng.uniform(0.5, 1.5, d_inner).astype(np.float32),
        eps=eps, headdim=headdim, d_state=d_state)


def test_special_cases():
    rng = np.random.default_rng(3)
    c = _random_case(rng)
    d_inner, conv_dim = 12, 22
    # oldest-tap convolution: the output is SiLU of the window's first entry
    c1 = dict(c, conv_w=np.tile(np.array([1, 0, 0, 0], np.float32), (conv_dim, 1)),
              conv_b=np.zeros(conv_dim, np.float32))
    _, xBC, _ = MB.split_in_proj(c1["zxbcdt"], d_inner, 5, 3)
    u, _ = MB.conv_step(c1["conv_state"], xBC, c1["conv_w"], c1["conv_b"])
    np.testing.assert_array_equal(u, MB.silu(c1["conv_state"][..., 1].astype(np.float64)))
    # a decay of zero (A = -e^40): the new state forgets the old one
    x = rng.standard_normal((2, 3, 4))
    Bv, Cv = rng.standard_normal((2, 5)), rng.standard_normal((2, 5))
    dt = rng.standard_normal((2, 3))
    y, st = MB.ssm_step(c["ssm_state"], x, Bv, Cv, dt, c["dt_bias"], np.full(3, 40.0), c["D"])
    dtp = MB.softplus(dt + c["dt_bias"])
    fresh = (dtp[:, :, None] * x)[..., None] * Bv[:, None, None, :]
    np.testing.assert_allclose(st.astype(np.float64), fresh.astype(np.float16), rtol=0, atol=0)
    # a vanishing step (dt' ~ e^-60): the state and the readout stay put
    y, st = MB.ssm_step(c["ssm_state"], x, Bv, Cv, np.full((2, 3), -60.0), c["dt_bias"],
                        c["A_log"], c["D"])
    np.testing.assert_array_equal(st, c["ssm_state"])
    old = c["ssm_state"].astype(np.float64)
    np.testing.assert_allclose(y, (old * Cv[:, None, None, :]).sum(-1)
                               + c["D"][None, :, None] * x, rtol=1e-12)


def test_gated_norm_scale_invariance():
    rng = np.random.default_rng(4)
    y, z, w = rng.standard_normal((3, 64)), rng.standard_normal((3, 64)), rng.uniform(0.5, 2, 64)
    a = MB.gated_rmsnorm(y, z, w, 0.0)
    np.testing.assert_allclose(MB.gated_rmsnorm(1024.0 * y, z, w, 0.0), a, rtol=1e-13)
    np.testing.assert_allclose(np.sqrt(((a / w) ** 2).mean(-1)), 1.0, rtol=1e-13)


@pytest.mark.parametrize("seed", [0, 1])
def test_against_loop_twin(seed):
    c = _random_case(np.random.default_rng(seed))
    out, conv_new, ssm_new = MB.mixer_step(**c)
    lists = {k: (v.astype(np.float64).tolist() if isinstance(v, np.ndarray) else v)
             for k, v in c.items()}
    t_out, t_conv, t_ssm = brute.mixer_step(**lists)
    np.testing.assert_allclose(out, np.array(t_out), rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(conv_new, np.array(t_conv).astype(np.float16))
    twin16 = np.array(t_ssm).astype(np.float16)
    # the same float64 values up to summation order: identical float16 except
    # at a rounding midpoint
    assert np.count_nonzero(ssm_new != twin16) <= 1


_ORIG = {n: getattr(MB, n) for n in ("conv_step", "ssm_step", "gated_rmsnorm", "silu")}


@pytest.mark.parametrize("mutant", ["no_shift", "no_conv_silu", "no_dt_bias", "growing_decay",
                                    "no_skip", "norm_then_gate", "sum_not_mean", "b_c_swapped"])
def test_planted_mixer_mistakes_are_caught(mutant, monkeypatch):
    if mutant == "no_shift":
        def conv(st, xBC, w, b):
            win = np.asarray(st, np.float16).astype(np.float64)
            out = (win * np.asarray(w, np.float64)[None]).sum(-1) + np.asarray(b, np.float64)
            return MB.silu(out), win.astype(np.float16)
        monkeypatch.setattr(MB, "conv_step", conv)
    elif mutant == "no_conv_silu":
        def conv(st, xBC, w, b):
            u, new = _ORIG["conv_step"](st, xBC, w, b)
            win = new.astype(np.float64)
            win[..., -1] = np.asarray(xBC, np.float64)
            return (win * np.asarray(w, np.float64)[None]).sum(-1) + np.asarray(b), new
        monkeypatch.setattr(MB, "conv_step", conv)
    elif mutant == "no_dt_bias":
        monkeypatch.setattr(MB, "ssm_step", lambda s, x, B, C, dt, dtb, A, D:
                            _ORIG["ssm_step"](s, x, B, C, dt, np.zeros_like(dtb), A, D))
    elif mutant == "growing_decay":
        def grow(st, x, Bv, Cv, dt, dtb, A_log, D):
            s64 = np.asarray(st, np.float16).astype(np.float64)
            dtp = MB.softplus(np.asarray(dt, np.float64) + np.asarray(dtb, np.float64)[None])
            a = np.exp(dtp * np.exp(np.asarray(A_log, np.float64))[None])   # A = +e^A_log
            x = np.asarray(x, np.float64)
            new = s64 * a[:, :, None, None] + (dtp[:, :, None] * x)[..., None] * \
                np.asarray(Bv, np.float64)[:, None, None, :]
            y = (new * np.asarray(Cv, np.float64)[:, None, None, :]).sum(-1) + \
                np.asarray(D, np.float64)[None, :, None] * x
            return y, new.astype(np.float16)
        monkeypatch.setattr(MB, "ssm_step", grow)
    elif mutant == "no_skip":
        monkeypatch.setattr(MB, "ssm_step", lambda s, x, B, C, dt, dtb, A, D:
                            _ORIG["ssm_step"](s, x, B, C, dt, dtb, A, np.zeros_like(D)))
    elif mutant == "norm_then_gate":
        def gn(y, z, w, eps):
            y = np.asarray(y, np.float64)
            r = 1.0 / np.sqrt((y * y).mean(-1, keepdims=True) + eps)
            return y * r * np.asarray(w)[None] * MB.silu(z)
        monkeypatch.setattr(MB, "gated_rmsnorm", gn)
    elif mutant == "sum_not_mean":
        def gn(y, z, w, eps):
            g = np.asarray(y, np.float64) * MB.silu(z)
            return g / np.sqrt((g * g).sum(-1, keepdims=True) + eps) * np.asarray(w)[None]
        monkeypatch.setattr(MB, "gated_rmsnorm", gn)
    elif mutant == "b_c_swapped":
        monkeypatch.setattr(MB, "ssm_step", lambda s, x, B, C, dt, dtb, A, D:
                            _ORIG["ssm_step"](s, x, C, B, dt, dtb, A, D))
    pins = [test_hand_step, lambda: test_against_loop_twin(0)]
    caught = False
    for p in pins:
        try:
            p()
        except AssertionError:
            caught = True
    assert caught, f"mutant {mutant} escaped the pins"


def test_rmsnorm_closed_forms():
    # a constant row c: every output is sign(c) * w (eps = 0)
    w = np.array([0.5, 2.0, -1.0, 3.0])
    np.testing.assert_allclose(MB.rmsnorm(np.full((1, 4), -7.5), w, 0.0), [-w], rtol=1e-15)
    # [3, 4, 0, 0]: mean square 25/4, scale 2/5
    np.testing.assert_allclose(MB.rmsnorm(np.array([[3.0, 4.0, 0.0, 0.0]]), np.ones(4), 0.0),
                               [[1.2, 1.6, 0.0, 0.0]], rtol=1e-15)
    # eps enters under the root: [1, 1] with eps 3 -> 1/2
    np.testing.assert_allclose(MB.rmsnorm(np.ones((1, 2)), np.ones(2), 3.0), [[0.5, 0.5]],
                               rtol=1e-15)
