"""GPU parity of the fused decode block (tm_tgemv_rms, tm_dgemv_rms,
tm_mixer_gate) against the oracle.

The fused projections normalize a float32 row (RMSNorm with a weight),
round it to bfloat16 and multiply.  The reference is the oracle's float64
normalization times the oracle's weights, without the rounding, so each
output may differ by the rounding of its activations: at most 2^-8 of
sum_k |x_k w_nk| (half a bfloat16 step of every x_k), plus float32
arithmetic.  The codes and scales come from the oracle's ternarizer on the
CPU; no reference value is derived from a GPU result.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import mamba as MB  # noqa: E402
from oracle import ternary as O  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402
from mixer_bounds import StateBound, oracle_gate  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()


def _d(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _oracle_packed(W, g, eps=1e-5):
    """Codes (packed), float16 scales and the dequantized matrix, all by the oracle."""
    _, s32, q, _ = O.ternarize(W, g, eps)
    s16 = O.scales_f16(s32)
    return O.pack(q), s16, q, O.dequantize(q, s16.astype(np.float64), g)


def _check_rms_product(y, src, w, eps, Wd, y0=None):
    """y (float32 [B, N]) against (y0 +) rmsnorm(src) * w . Wd^T within the
    activations' bfloat16 rounding."""
    x = MB.rmsnorm(src.astype(np.float64), w, eps)
    ref = x @ Wd.T
    bound = 2.0 ** -8 * (np.abs(x) @ np.abs(Wd).T) * (1 + 1e-4)
    if y0 is not None:
        ref = ref + y0
        bound = bound + 2.0 ** -23 * np.abs(ref)
    bound = bound + 1e-6 * np.abs(ref).max()
    err = np.abs(y.astype(np.float64) - ref)
    assert np.all(err <= bound), f"max err / bound {float((err / bound).max()):.3f}"
    return float((err / bound).max())


def _src(rng, B, K, outliers=False):
    src = rng.standard_normal((B, K)).astype(np.float32)
    if outliers:   # a residual stream with a few large channels
        src[:, rng.choice(K, 4, replace=False)] *= 64.0
    return src


@pytest.mark.parametrize("N,K,g,B,acc", [
    (8512, 2048, 128, 1, False),   # in_proj of Mamba-2 1.3B
    (8512, 2048, 128, 4, False),
    (2048, 4096, 128, 1, True),    # out_proj, added into the residual
    (2048, 4096, 128, 4, True),
    (300, 384, 64, 2, True),       # ragged rows, K of three 128-column chunks
    (96, 256, 32, 1, False),       # K of one slot (no split across waves)
    (130, 1536, 256, 3, False),
    (64, 1024, 512, 2, True),
])
def test_tgemv_rms_against_oracle(N, K, g, B, acc):
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(N + K + g + B)
    print(f"[tgemv_rms] N={N} K={K} g={g} B={B} acc={acc}", flush=True)
    W = synth.weights(rng, N, K, outliers=True)
    codes, s16, q, Wd = _oracle_packed(W, g)
    src = _src(rng, B, K, outliers=True)
    w = (1 + 0.1 * rng.standard_normal(K)).astype(np.float32)
    y0 = rng.standard_normal((B, N)).astype(np.float32) if acc else None
    y = _d(y0) if acc else None
    y = ops.tgemv_rms(_d(src), _d(codes), _d(s16.view(np.int16)).view(torch.float16), g, _d(w),
                      1e-5, y=y, accumulate=acc)
    torch.cuda.synchronize()
    r = _check_rms_product(y.cpu().numpy(), src, w, 1e-5, Wd, y0)
    print(f"  max error / bound {r:.3f}", flush=True)


def test_tgemv_rms_is_deterministic_and_scale_free():
    """Two calls give the same bits; scaling src by 2^k changes nothing
    (the normalization removes it exactly) unless eps matters."""
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(3)
    N, K, g = 8512, 2048, 128
    codes, s16, _, _ = _oracle_packed(synth.weights(rng, N, K), g)
    c, s = _d(codes), _d(s16.view(np.int16)).view(torch.float16)
    src = _src(rng, 2, K)
    w = _d((1 + 0.1 * rng.standard_normal(K)).astype(np.float32))
    a = ops.tgemv_rms(_d(src), c, s, g, w, 0.0)
    b = ops.tgemv_rms(_d(src), c, s, g, w, 0.0)
    d = ops.tgemv_rms(_d(src * np.float32(8.0)), c, s, g, w, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(a, d)


@pytest.mark.parametrize("N,K,B,acc", [(8512, 2048, 1, False), (2048, 4096, 4, True),
                                       (100, 192, 3, True)])
def test_dgemv_rms_against_oracle(N, K, B, acc):
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(N + K + B)
    print(f"[dgemv_rms] N={N} K={K} B={B} acc={acc}", flush=True)
    W16 = synth.weights(rng, N, K, outliers=True).astype(np.float16)
    src = _src(rng, B, K, outliers=True)
    w = (1 + 0.1 * rng.standard_normal(K)).astype(np.float32)
    y0 = rng.standard_normal((B, N)).astype(np.float32) if acc else None
    y = ops.dgemv_rms(_d(src), _d(W16.view(np.int16)).view(torch.float16), _d(w), 1e-5,
                      y=_d(y0) if acc else None, accumulate=acc)
    torch.cuda.synchronize()
    r = _check_rms_product(y.cpu().numpy(), src, w, 1e-5, W16.astype(np.float64), y0)
    print(f"  max error / bound {r:.3f}", flush=True)


@pytest.mark.parametrize("B,H,steps", [(1, 64, 3), (4, 64, 2), (2, 5, 6)])
def test_mixer_gate_against_oracle(B, H, steps):
    """The gated values per step against the oracle's, each side carrying its
    own states on; the ring position advances once per call, and a
    tm_mixer_step after the gated steps continues the same ring."""
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(100 + B + H)
    print(f"[mixer_gate] B={B} H={H} steps={steps}", flush=True)
    prm = synth.mixer_params(rng, H)
    conv0, ssm0 = synth.mixer_states(rng, B, H)
    dp = {k: _d(v) for k, v in prm.items()}
    conv_t = _d(conv0.view(np.int16)).view(torch.float16)
    ssm_t = _d(ssm0.view(np.int16)).view(torch.float16)
    pos_t = torch.zeros((1,), dtype=torch.int32, device="cuda")
    conv_ref, ssm_ref = conv0, ssm0
    sb = StateBound(ssm0)
    for step in range(steps):
        z = synth.in_proj_out(rng, B, H)
        g = ops.mixer_gate(_d(z), conv_t, pos_t, ssm_t, dp["conv_w"], dp["conv_b"],
                           dp["dt_bias"], dp["A_log"], dp["D"])
        gref, conv_ref, ssm_ref, C, sz, dx = oracle_gate(z, conv_ref, ssm_ref, prm)
        sb.step(ssm_ref)
        torch.cuda.synchronize()
        pos = int(pos_t.cpu()[0])
        assert pos == (step + 1) % 4, "position word after the call"
        ring = conv_t.cpu().numpy()
        win = np.stack([ring[..., (pos + j) % 4] for j in range(4)], axis=-1)
        assert np.array_equal(win, conv_ref), "convolution ring"
        sb.check(ssm_t.cpu().numpy(), ssm_ref)
        got = g.cpu().numpy().astype(np.float64)
        bar = sb.gate_bar(ssm_ref, C, sz, dx, gref)
        err = np.abs(got - gref)
        assert np.all(err <= bar), f"step {step}: max err / bar {float((err / bar).max()):.3f}"
    # the unfused step continues the ring from the gated steps' position
    z = synth.in_proj_out(rng, B, H)
    ops.mixer_step(_d(z), conv_t, pos_t, ssm_t, dp["conv_w"], dp["conv_b"], dp["dt_bias"],
                   dp["A_log"], dp["D"], dp["norm_w"], 1e-5)
    conv_ref = oracle_gate(z, conv_ref, ssm_ref, prm)[1]
    torch.cuda.synchronize()
    pos = int(pos_t.cpu()[0])
    assert pos == (steps + 1) % 4
    ring = conv_t.cpu().numpy()
    assert np.array_equal(np.stack([ring[..., (pos + j) % 4] for j in range(4)], axis=-1),
                          conv_ref)
