"""GPU parity of the Mamba-2 mixer decode step (tm_mixer_step) against the
oracle (oracle/mamba.py).

Bars: the convolution ring takes the new inputs rounded to float16, bit for
bit; the float16 SSM state matches the oracle's float16 rounding except
where the float32 and float64 results straddle a float16 rounding midpoint
(at most one float16 step apart, on a tiny fraction of elements); the
bfloat16 output is within one bfloat16 rounding (2^-8 relative) plus float32
arithmetic error of the oracle's float64 value.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import mamba as MB  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()


def _d(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def ring_to_window(ring, pos):
    """float16 ring [B, C, 4] at position pos -> window oldest first."""
    return np.stack([ring[..., (pos + j) % 4] for j in range(4)], axis=-1)


def check_ssm_state(s_gpu, ssm_ref):
    """float16 states: equal except at float16 rounding midpoints, where the
    float32 and float64 results may round to neighbours (one float16 step,
    on a tiny fraction of the elements)."""
    diff = s_gpu != ssm_ref
    if diff.any():
        a, b = s_gpu[diff].astype(np.float64), ssm_ref[diff].astype(np.float64)
        step16 = np.abs(np.nextafter(ssm_ref[diff], np.float16(np.inf)).astype(np.float64) - b)
        assert np.all(np.abs(a - b) <= step16 * 1.001)
        assert diff.sum() <= 1e-4 * diff.size + 2, int(diff.sum())


def run_steps(B, nheads, steps, seed, eps=1e-5):
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(seed)
    prm = synth.mixer_params(rng, nheads)
    conv0, ssm0 = synth.mixer_states(rng, B, nheads)
    print(f"[mixer] B={B} nheads={nheads} steps={steps} seed={seed}", flush=True)
    dp = {k: _d(v) for k, v in prm.items()}
    conv_t = _d(conv0.view(np.int16)).view(torch.float16)
    ssm_t = _d(ssm0.view(np.int16)).view(torch.float16)
    pos_t = torch.zeros((1,), dtype=torch.int32, device="cuda")
    conv_ref, ssm_ref = conv0, ssm0
    worst = 0.0
    for step in range(steps):
        z = synth.in_proj_out(rng, B, nheads)
        out = ops.mixer_step(_d(z), conv_t, pos_t, ssm_t, dp["conv_w"], dp["conv_b"],
                             dp["dt_bias"], dp["A_log"], dp["D"], dp["norm_w"], eps)
        ref, conv_ref, ssm_ref = MB.mixer_step(z, conv_ref, ssm_ref, prm["conv_w"], prm["conv_b"],
                                               prm["dt_bias"], prm["A_log"], prm["D"],
                                               prm["norm_w"], eps, synth.HEADDIM, synth.D_STATE)
        torch.cuda.synchronize()
        got = (out.cpu().view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16
               ).view(np.float32).astype(np.float64)
        pos = int(pos_t.cpu()[0])
        assert pos == (step + 1) % 4
        win = ring_to_window(conv_t.cpu().numpy(), pos)
        assert np.array_equal(win, conv_ref), "convolution ring"
        s_gpu = ssm_t.cpu().numpy()
        check_ssm_state(s_gpu, ssm_ref)
        err = np.abs(got - ref) / (2.0 ** -8 * np.abs(ref) + 1e-6 * np.abs(ref).max())
        worst = max(worst, float(err.max()))
        assert np.all(err <= 1.0), f"step {step}: max err / bar {err.max():.3f}"
        # carry the GPU's own state on (the oracle continues from its own)
        conv_ref, ssm_ref = win, s_gpu
    print(f"  max error / bar {worst:.3f}", flush=True)


@pytest.mark.parametrize("B", [1, 4])
def test_mixer_step_full_layer(B):
    """The Mamba-2 1.3B layer: 64 heads, d_inner 4096, conv_dim 4352."""
    run_steps(B, 64, steps=3, seed=B)


def test_mixer_step_ring_wraps():
    """Six steps: the convolution ring position wraps past 3."""
    run_steps(2, 5, steps=6, seed=11)


def test_mixer_step_zero_input_keeps_decaying_state():
    """dt large and negative (no update): the state stays, the window shifts."""
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(4)
    H, B = 2, 1
    prm = synth.mixer_params(rng, H)
    prm["dt_bias"][:] = -60.0
    conv0, ssm0 = synth.mixer_states(rng, B, H)
    ssm_t = _d(ssm0.view(np.int16)).view(torch.float16)
    conv_t = _d(conv0.view(np.int16)).view(torch.float16)
    pos_t = torch.zeros((1,), dtype=torch.int32, device="cuda")
    z = synth.in_proj_out(rng, B, H)
    ops.mixer_step(_d(z), conv_t, pos_t, ssm_t, *[_d(prm[k]) for k in
                   ("conv_w", "conv_b", "dt_bias", "A_log", "D", "norm_w")], 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(ssm_t.cpu().numpy(), ssm0)


def _bf16_to_f64(t):
    return (t.cpu().view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16
            ).view(np.float32).astype(np.float64)


def test_residual_rmsnorm():
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(21)
    B, D = 3, 2048
    r0 = rng.standard_normal((B, D)).astype(np.float32)
    y = (rng.standard_normal((B, D)) * 0.5).astype(np.float32)
    w = (1 + 0.1 * rng.standard_normal(D)).astype(np.float32)
    r = _d(r0)
    x = ops.residual_rmsnorm(r, _d(y), _d(w), 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(r.cpu().numpy(), r0 + y)         # float32 add, exact rounding
    ref = MB.rmsnorm((r0 + y).astype(np.float64), w, 1e-5)
    got = _bf16_to_f64(x)
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-7 * np.abs(ref).max())
    # without y: the residual stays
    x2 = ops.residual_rmsnorm(r, None, _d(w), 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(r.cpu().numpy(), r0 + y)
    assert np.array_equal(_bf16_to_f64(x2), got)


def _small_decoder(seed, keep=(2,), B=1, L=3):
    from paper_2606_18114_amd.stack import Mamba2Decoder
    rng = np.random.default_rng(seed)
    d_model, H = 256, 2
    Z = 2 * 128 + 256 + H
    Ws = {("in", l): synth.weights(rng, Z, d_model, outliers=True) for l in range(L)}
    Ws.update({("out", l): synth.weights(rng, d_model, H * 64) for l in range(L)})
    mix = [synth.mixer_params(rng, H) for _ in range(L)]
    pre = [(1 + 0.1 * rng.standard_normal(d_model)).astype(np.float32) for _ in range(L)]
    dec = Mamba2Decoder(lambda k, l: _d(Ws[(k, l)]), lambda l: mix[l],
                        lambda l: torch.from_numpy(pre[l]), L, d_model, H, keep=keep,
                        g=128, batch=B)
    for l in range(L):
        conv, ssm = synth.mixer_states(rng, B, H)
        dec.set_states(l, _d(conv.view(np.int16)).view(torch.float16),
                       _d(ssm.view(np.int16)).view(torch.float16))
    dec.emb.copy_(_d(rng.standard_normal((B, d_model)).astype(np.float32)))
    return dec, Ws, mix, pre


@pytest.mark.parametrize("B", [1, 2])
def test_decoder_layers_against_oracle(B):
    """Three layers (the last kept in float16), checked stage by stage with
    the GPU's own inputs to each stage: the pre-norm, in_proj, the mixer
    step (with the layer's states) and out_proj."""
    from oracle import ternary as O
    dec, Ws, mix, pre = _small_decoder(7 + B, B=B)
    y_prev = None
    res_prev = dec.emb.cpu().numpy().astype(np.float64)
    for l in range(dec.L):
        lay = dec.layers[l]
        conv0 = ring_to_window(lay["conv"].cpu().numpy(), int(lay["pos"].cpu()[0]))
        ssm0 = lay["ssm"].cpu().numpy()
        dec.layer_step(l)
        torch.cuda.synchronize()
        res = dec.residual.cpu().numpy()
        if y_prev is not None:
            assert np.array_equal(res, (res_prev + y_prev).astype(np.float32))
        x = _bf16_to_f64(dec.x[0])
        ref = MB.rmsnorm(res.astype(np.float64), pre[l], dec.eps)
        assert np.all(np.abs(x - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-7 * np.abs(ref).max())
        xb = dec.x[0].cpu().view(torch.int16).numpy().view(np.uint16)
        zx = dec.zx[0].cpu().numpy()
        if l in dec.keep:
            zref = O.dense_gemv(xb, Ws[("in", l)].astype(np.float16))
        else:
            q = O.unpack(lay["in"][1][0].cpu().numpy(), 256)
            zref = O.gemv(xb, q, lay["in"][2][0].cpu().numpy(), 128)
        assert O.rel_fro_error(zx, zref) <= 1e-6
        mref, conv1, ssm1 = MB.mixer_step(zx.astype(np.float64), conv0, ssm0, mix[l]["conv_w"],
                                          mix[l]["conv_b"], mix[l]["dt_bias"], mix[l]["A_log"],
                                          mix[l]["D"], mix[l]["norm_w"], dec.eps, 64, 128)
        m = _bf16_to_f64(dec.m[0])
        assert np.all(np.abs(m - mref) <= 2.0 ** -8 * np.abs(mref) + 1e-6 * np.abs(mref).max())
        win = ring_to_window(lay["conv"].cpu().numpy(), int(lay["pos"].cpu()[0]))
        assert np.array_equal(win, conv1)
        check_ssm_state(lay["ssm"].cpu().numpy(), ssm1)
        mb = dec.m[0].cpu().view(torch.int16).numpy().view(np.uint16)
        y = dec.y[0].cpu().numpy()
        if l in dec.keep:
            yref = O.dense_gemv(mb, Ws[("out", l)].astype(np.float16))
        else:
            q = O.unpack(lay["out"][1][0].cpu().numpy(), 128)
            yref = O.gemv(mb, q, lay["out"][2][0].cpu().numpy(), 128)
        assert O.rel_fro_error(y, yref) <= 1e-6
        res_prev, y_prev = res.astype(np.float32), y.astype(np.float32)
    print(f"[decoder] B={B} layers {dec.L} (kept {sorted(dec.keep)}) match stage by stage",
          flush=True)


def test_decoder_graph_replays_match_eager():
    """Three tokens eagerly, then the same three from the same states as
    replays of one captured graph (with other GPU work and host syncs in
    between): outputs, residual and every layer's states agree bit for bit."""
    dec, _, _, _ = _small_decoder(5, B=2)
    init = [(l["conv"].clone(), l["ssm"].clone(), l["pos"].clone()) for l in dec.layers]
    emb = [torch.randn_like(dec.emb) for _ in range(3)]
    eager = []
    for e in emb:
        dec.emb.copy_(e)
        eager.append(dec.token().clone())
    final_eager = [(l["conv"].clone(), l["ssm"].clone(), l["pos"].clone()) for l in dec.layers]
    for lay, (c, s, p) in zip(dec.layers, init):
        lay["conv"].copy_(c)
        lay["ssm"].copy_(s)
        lay["pos"].copy_(p)
    dec.capture()
    # capture does not execute: the states are still the initial ones
    for lay, (c, s, p) in zip(dec.layers, init):
        assert torch.equal(lay["ssm"], s) and torch.equal(lay["pos"], p)
    for t, e in enumerate(emb):
        dec.emb.copy_(e)
        out = dec.replay()
        torch.cuda.synchronize()
        _ = torch.randn(1000, device="cuda").sum().item()   # unrelated work in between
        assert torch.equal(out, eager[t]), f"token {t}"
    for lay, (c, s, p) in zip(dec.layers, final_eager):
        assert torch.equal(lay["conv"], c) and torch.equal(lay["ssm"], s)
        assert torch.equal(lay["pos"], p)
