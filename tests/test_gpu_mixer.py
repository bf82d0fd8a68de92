"""GPU parity of the Mamba-2 mixer decode step (tm_mixer_step) and of the
layer-ordered decoder built on it, against the oracle (oracle/mamba.py).

The GPU and the oracle each carry their own states from step to step (no
reference value comes from a GPU result).  Bars: the convolution ring takes
the new inputs rounded to float16, bit for bit; the float16 SSM states stay
within the running bound of tests/mixer_bounds.py; the bfloat16 output is
within one bfloat16 rounding (2^-8 relative) of the oracle's float64 value
plus what the states' difference can move it.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import mamba as MB  # noqa: E402
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


def ring_to_window(ring, pos):
    """float16 ring [B, C, 4] at position pos -> window oldest first."""
    return np.stack([ring[..., (pos + j) % 4] for j in range(4)], axis=-1)


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
    sb = StateBound(ssm0)
    worst = 0.0
    for step in range(steps):
        z = synth.in_proj_out(rng, B, nheads)
        out = ops.mixer_step(_d(z), conv_t, pos_t, ssm_t, dp["conv_w"], dp["conv_b"],
                             dp["dt_bias"], dp["A_log"], dp["D"], dp["norm_w"], eps)
        g, _, _, C, sz, dx = oracle_gate(z, conv_ref, ssm_ref, prm)
        ref, conv_ref, ssm_ref = MB.mixer_step(z, conv_ref, ssm_ref, prm["conv_w"], prm["conv_b"],
                                               prm["dt_bias"], prm["A_log"], prm["D"],
                                               prm["norm_w"], eps, synth.HEADDIM, synth.D_STATE)
        torch.cuda.synchronize()
        got = _bf16_to_f64(out)
        pos = int(pos_t.cpu()[0])
        assert pos == (step + 1) % 4
        win = ring_to_window(conv_t.cpu().numpy(), pos)
        assert np.array_equal(win, conv_ref), "convolution ring"
        sb.step(ssm_ref)
        sb.check(ssm_t.cpu().numpy(), ssm_ref)
        # g may differ by bar_g (the states' difference); the normalization
        # moves with it by at most |bar_g| / |g| relative
        bar_g = sb.gate_bar(ssm_ref, C, sz, dx, g)
        r = 1.0 / np.sqrt((g * g).mean(-1, keepdims=True) + eps)
        rel = np.linalg.norm(bar_g, axis=-1, keepdims=True) / np.linalg.norm(g, axis=-1,
                                                                           keepdims=True)
        bar = (2.0 ** -8 * np.abs(ref) + r * np.abs(prm["norm_w"])[None] * bar_g
               + 1.01 * rel * np.abs(ref) + 1e-6 * np.abs(ref).max())
        err = np.abs(got - ref) / bar
        worst = max(worst, float(err.max()))
        assert np.all(err <= 1.0), f"step {step}: max err / bar {err.max():.3f}"
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


def _small_decoder(seed, keep=(2,), B=1, L=3, fused=None, stack=False):
    # layer-by-layer forms (the one-launch form has tests of its own)
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
                        g=128, batch=B, fused=fused, stack=stack)
    states = []
    for l in range(L):
        conv, ssm = synth.mixer_states(rng, B, H)
        states.append((conv, ssm))
        dec.set_states(l, _d(conv.view(np.int16)).view(torch.float16),
                       _d(ssm.view(np.int16)).view(torch.float16))
    dec.emb.copy_(_d(rng.standard_normal((B, d_model)).astype(np.float32)))
    return dec, Ws, mix, pre, states


class OracleDecoder:
    """The same blocks on the oracle: weights ternarized by the oracle (kept
    layers rounded to float16), activations rounded to bfloat16 where the
    layer hands them to a projection, states carried in float16."""

    def __init__(self, Ws, mix, pre, states, keep, g, eps):
        from oracle import ternary as O
        self.O, self.mix, self.pre, self.keep, self.g, self.eps = O, mix, pre, keep, g, eps
        self.states = [(c.copy(), s.copy()) for c, s in states]
        self.W = {}
        for (kind, l), W in Ws.items():
            if l in keep:
                self.W[(kind, l)] = ("dense", W.astype(np.float16))
            else:
                _, s32, q, _ = O.ternarize(W, g, eps)
                self.W[(kind, l)] = ("ternary", q, O.scales_f16(s32))

    def _proj(self, kind, l, x64):
        xb = synth.f32_to_bf16_bits(x64.astype(np.float32))
        w = self.W[(kind, l)]
        if w[0] == "dense":
            return self.O.dense_gemv(xb, w[1])
        return self.O.gemv(xb, w[1], w[2], self.g)

    def token(self, emb):
        res = emb.astype(np.float64)
        for l, m in enumerate(self.mix):
            zx = self._proj("in", l, MB.rmsnorm(res, self.pre[l], self.eps))
            conv, ssm = self.states[l]
            out, conv, ssm = MB.mixer_step(zx, conv, ssm, m["conv_w"], m["conv_b"], m["dt_bias"],
                                           m["A_log"], m["D"], m["norm_w"], self.eps, 64, 128)
            self.states[l] = (conv, ssm)
            res = res + self._proj("out", l, out)
        return MB.rmsnorm(res, np.ones(res.shape[-1]), self.eps)


@pytest.mark.parametrize("B,fused", [(1, True), (2, True), (2, False), (16, False)])
def test_decoder_tokens_against_oracle(B, fused):
    """Three tokens through three blocks (the last kept in float16), fused or
    not, against the oracle's own decode from the same weights, states and
    embeddings.  The two sides round the activations handed to a projection
    to bfloat16 from float32 and float64 values, so an element may land one
    bfloat16 step apart; the output stays within two bfloat16 steps plus
    1e-3 of its largest element, and the states within 1e-3 (Frobenius)."""
    # (blocks kept in FP16 decode at batch up to 8: the batch-16 stack is all ternary)
    dec, Ws, mix, pre, states = _small_decoder(7 + B, keep=(2,) if B <= 8 else (), B=B,
                                               fused=fused)
    assert dec.fused == fused
    ref_dec = OracleDecoder(Ws, mix, pre, states, dec.keep, dec.g, dec.eps)
    rng = np.random.default_rng(40 + B)
    print(f"[decoder] B={B} fused={fused} launches/token {dec.launches_per_token()}", flush=True)
    for t in range(3):
        emb = rng.standard_normal((B, dec.d_model)).astype(np.float32)
        dec.emb.copy_(_d(emb))
        got = _bf16_to_f64(dec.token())
        ref = ref_dec.token(emb)
        torch.cuda.synchronize()
        bar = 2.0 ** -7 * np.abs(ref) + 1e-3 * np.abs(ref).max()
        err = np.abs(got - ref)
        assert np.all(err <= bar), f"token {t}: max err / bar {float((err / bar).max()):.3f}"
    from oracle import ternary as O
    for l, lay in enumerate(dec.layers):
        conv_ref, ssm_ref = ref_dec.states[l]
        win = ring_to_window(lay["conv"].cpu().numpy(), int(lay["pos"].cpu()[0]))
        assert int(lay["pos"].cpu()[0]) == 3
        assert O.rel_fro_error(win.astype(np.float64), conv_ref.astype(np.float64)) <= 1e-3
        assert O.rel_fro_error(lay["ssm"].cpu().numpy().astype(np.float64),
                               ssm_ref.astype(np.float64)) <= 1e-3


def test_fused_and_unfused_decoders_agree():
    """The fused decode (3 launches per block) and the unfused one (5) on the
    same inputs: the same result up to bfloat16 rounding of the activations."""
    a, *_ = _small_decoder(11, B=2, fused=True)
    b, *_ = _small_decoder(11, B=2, fused=False)
    assert a.launches_per_token() == 3 * a.L + 2 and b.launches_per_token() == 5 * b.L + 2
    for t in range(3):
        e = torch.randn_like(a.emb)
        a.emb.copy_(e)
        b.emb.copy_(e)
        xa = _bf16_to_f64(a.token())
        xb = _bf16_to_f64(b.token())
        torch.cuda.synchronize()
        assert np.all(np.abs(xa - xb) <= 2.0 ** -7 * np.abs(xb) + 1e-3 * np.abs(xb).max()), t


@pytest.mark.parametrize("fused", [True, False])
def test_decoder_graph_replays_match_eager(fused):
    """Three tokens eagerly, then the same three from the same states as
    replays of one captured graph (with other GPU work and host syncs in
    between): outputs, residual and every layer's states agree bit for bit."""
    dec, *_ = _small_decoder(5, B=2, fused=fused)
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
