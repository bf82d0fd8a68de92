"""GPU parity of the one-launch stack decode (tm_mamba2_decode_token): a
token per batch row (batch 1 .. 4) through every Mamba-2 block with grid
barriers between the phases, against the oracle's own decode (oracle
ternarization, float16 states carried by each side), and against the
layer-by-layer fused decode on the same states.

Bars as for the layer-by-layer decoder: the two sides round the activations
handed to a projection to bfloat16 from float32 and float64 values (and the
stack kernel sums its normalizations in another order than the fused
launches), so an element may land one bfloat16 step apart; outputs stay
within two bfloat16 steps plus 1e-3 of their largest element, states within
1e-3 (Frobenius).
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_18114_amd import synth  # noqa: E402
from test_gpu_mixer import OracleDecoder, _bf16_to_f64, _d, ring_to_window  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()


def _decoder(seed, L, d_model, H, g=128, stack=None, outliers=True, keep=(), batch=1):
    from paper_2606_18114_amd.stack import Mamba2Decoder
    rng = np.random.default_rng(seed)
    Z = 2 * 64 * H + 256 + H
    Ws = {("in", l): synth.weights(rng, Z, d_model, outliers=outliers) for l in range(L)}
    Ws.update({("out", l): synth.weights(rng, d_model, H * 64) for l in range(L)})
    mix = [synth.mixer_params(rng, H) for _ in range(L)]
    pre = [(1 + 0.1 * rng.standard_normal(d_model)).astype(np.float32) for _ in range(L)]
    dec = Mamba2Decoder(lambda k, l: _d(Ws[(k, l)]), lambda l: mix[l],
                        lambda l: torch.from_numpy(pre[l]), L, d_model, H, keep=keep, g=g,
                        batch=batch, stack=stack)
    states = []
    for l in range(L):
        conv, ssm = synth.mixer_states(rng, batch, H)
        states.append((conv, ssm))
        dec.set_states(l, _d(conv.view(np.int16)).view(torch.float16),
                       _d(ssm.view(np.int16)).view(torch.float16))
    return dec, Ws, mix, pre, states


def _need_cus(n):
    cus = torch.cuda.get_device_properties(torch.cuda.current_device()).multi_processor_count
    if cus < n:
        pytest.skip(f"the mixer phase needs {n} workgroups resident at once; {cus} CUs")


def _timeout_flag(dec):
    torch.cuda.synchronize()
    return int(dec.stack_ws[24576:24580].view(torch.int32).cpu()[0])   # word 6144


@pytest.mark.parametrize("L,d_model,H,g", [(3, 256, 2, 128), (2, 512, 8, 64), (2, 1024, 4, 256)])
def test_stack_decode_against_oracle(L, d_model, H, g):
    dec, Ws, mix, pre, states = _decoder(17 + L + H, L, d_model, H, g)
    assert dec.stack and dec.launches_per_token() == 2
    ref_dec = OracleDecoder(Ws, mix, pre, states, (), g, dec.eps)
    rng = np.random.default_rng(50 + H)
    print(f"[stack decode] L={L} d_model={d_model} nheads={H} g={g}", flush=True)
    for t in range(3):
        emb = rng.standard_normal((1, d_model)).astype(np.float32)
        dec.emb.copy_(_d(emb))
        got = _bf16_to_f64(dec.token())
        ref = ref_dec.token(emb)
        torch.cuda.synchronize()
        bar = 2.0 ** -7 * np.abs(ref) + 1e-3 * np.abs(ref).max()
        err = np.abs(got - ref)
        assert np.all(err <= bar), f"token {t}: max err / bar {float((err / bar).max()):.3f}"
    assert _timeout_flag(dec) == 0
    from oracle import ternary as O
    for l, lay in enumerate(dec.layers):
        conv_ref, ssm_ref = ref_dec.states[l]
        pos = int(lay["pos"].cpu()[0])
        assert pos == 3
        win = ring_to_window(lay["conv"].cpu().numpy(), pos)
        assert O.rel_fro_error(win.astype(np.float64), conv_ref.astype(np.float64)) <= 1e-3
        assert O.rel_fro_error(lay["ssm"].cpu().numpy().astype(np.float64),
                               ssm_ref.astype(np.float64)) <= 1e-3


@pytest.mark.parametrize("L,d_model,H,g,keep", [(4, 256, 2, 128, (0, 3)),
                                                (3, 512, 4, 64, (1,)),
                                                (5, 1024, 8, 256, (0, 1, 4))])
def test_stack_decode_kept_fp16_layers(L, d_model, H, g, keep):
    """Blocks kept in FP16 (Sec. 7) inside the one-launch decode: their
    projections from float16 weights, the rest ternary, against the oracle's
    decode of the same mixed stack, next to the layer-by-layer fused decode
    from the same weights and states.  Outputs within the bars above.  The
    states drift from the oracle's as the activations handed to each
    projection (bfloat16 of float32 against bfloat16 of float64 values) land
    a bfloat16 step apart here and there, more with every block: each state
    stays within 1e-3 of the oracle's, or within twice the fused decode's
    own distance to it (and 4e-3)."""
    a, Ws, mix, pre, states = _decoder(40 + L + H, L, d_model, H, g, stack=True, keep=keep)
    b, *_ = _decoder(40 + L + H, L, d_model, H, g, stack=False, keep=keep)
    assert a.stack and a.kept == sorted(keep) and not b.stack
    ref_dec = OracleDecoder(Ws, mix, pre, states, keep, g, a.eps)
    rng = np.random.default_rng(60 + H)
    print(f"[stack decode] kept {keep} L={L} d_model={d_model} nheads={H} g={g}", flush=True)
    for t in range(3):
        emb = rng.standard_normal((1, d_model)).astype(np.float32)
        a.emb.copy_(_d(emb))
        b.emb.copy_(_d(emb))
        xa = _bf16_to_f64(a.token())
        xb = _bf16_to_f64(b.token())
        ref = ref_dec.token(emb)
        torch.cuda.synchronize()
        bar = 2.0 ** -7 * np.abs(ref) + 1e-3 * np.abs(ref).max()
        ra = float((np.abs(xa - ref) / bar).max())
        rb = float((np.abs(xb - ref) / bar).max())
        print(f"  token {t}: err/bar one launch {ra:.3f}, layer by layer {rb:.3f}", flush=True)
        assert ra <= 1.0 and rb <= 1.0
    assert _timeout_flag(a) == 0
    from oracle import ternary as O
    for l in range(L):
        conv_ref, ssm_ref = ref_dec.states[l]
        e = {}
        for name, dec in (("a", a), ("b", b)):
            lay = dec.layers[l]
            win = ring_to_window(lay["conv"].cpu().numpy(), int(lay["pos"].cpu()[0]))
            e[name] = (O.rel_fro_error(win.astype(np.float64), conv_ref.astype(np.float64)),
                       O.rel_fro_error(lay["ssm"].cpu().numpy().astype(np.float64),
                                       ssm_ref.astype(np.float64)))
        print(f"  block {l}: conv/ssm state err one launch {e['a'][0]:.2e}/{e['a'][1]:.2e}, "
              f"layer by layer {e['b'][0]:.2e}/{e['b'][1]:.2e}", flush=True)
        for i in range(2):
            assert e["a"][i] <= max(1e-3, min(2 * e["b"][i], 4e-3)), (l, i, e)


@pytest.mark.parametrize("B", [1, 4])
def test_stack_decode_full_size_against_oracle(B):
    """Two blocks of the Mamba-2 1.3B shapes (d_model 2048, 64 heads,
    in_proj 8512 x 2048, out_proj 2048 x 4096), three tokens per batch row
    (batch 4: 256 mixer workgroups), against the oracle's decode; then the
    layer-by-layer fused decode from the same weights and states stays
    within twice the bar of the one-launch decode (each is within the bar of
    the exact result)."""
    _need_cus(64 * B)
    a, Ws, mix, pre, states = _decoder(3, 2, synth.D_MODEL, 64, stack=True, batch=B)
    b, *_ = _decoder(3, 2, synth.D_MODEL, 64, stack=False, batch=B)
    assert a.stack and not b.stack and b.fused
    ref_dec = OracleDecoder(Ws, mix, pre, states, (), a.g, a.eps)
    rng = np.random.default_rng(77)
    for t in range(3):
        emb = rng.standard_normal((B, synth.D_MODEL)).astype(np.float32)
        a.emb.copy_(_d(emb))
        b.emb.copy_(_d(emb))
        xa = _bf16_to_f64(a.token())
        xb = _bf16_to_f64(b.token())
        ref = ref_dec.token(emb)
        torch.cuda.synchronize()
        bar = 2.0 ** -7 * np.abs(ref) + 1e-3 * np.abs(ref).max(axis=1, keepdims=True)
        ra = float((np.abs(xa - ref) / bar).max())
        rb = float((np.abs(xb - ref) / bar).max())
        rab = float((np.abs(xa - xb) / (2 * bar)).max())
        print(f"[stack decode] full size B={B} token {t}: err/bar stack {ra:.3f} fused {rb:.3f} "
              f"stack-vs-fused/2bar {rab:.3f}", flush=True)
        assert ra <= 1.0 and rab <= 1.0
    assert _timeout_flag(a) == 0
    from oracle import ternary as O
    for l, lay in enumerate(a.layers):
        conv_ref, ssm_ref = ref_dec.states[l]
        pos = int(lay["pos"].cpu()[0])
        win = ring_to_window(lay["conv"].cpu().numpy(), pos)
        assert O.rel_fro_error(win.astype(np.float64), conv_ref.astype(np.float64)) <= 1e-3
        assert O.rel_fro_error(lay["ssm"].cpu().numpy().astype(np.float64),
                               ssm_ref.astype(np.float64)) <= 1e-3


@pytest.mark.parametrize("L,d_model,H,g,B,keep", [(3, 256, 2, 128, 4, ()),
                                                  (2, 512, 8, 64, 2, (1,)),
                                                  (3, 1024, 4, 256, 3, (0,)),
                                                  (2, 256, 64, 128, 4, (1,))])
def test_stack_decode_batches(L, d_model, H, g, B, keep):
    """B tokens at once (one per batch row; the mixer's workgroups one per
    head and row, 256 of them at 64 heads and B = 4), blocks kept in FP16
    among them, against the oracle's decode of the same batch and next to
    the layer-by-layer fused decode: outputs of every row within the bars
    above, states as in the kept-block test."""
    _need_cus(H * B)
    a, Ws, mix, pre, states = _decoder(90 + L + H + B, L, d_model, H, g, stack=True, keep=keep,
                                       batch=B)
    b, *_ = _decoder(90 + L + H + B, L, d_model, H, g, stack=False, keep=keep, batch=B)
    assert a.stack and a.B == B and not b.stack and a.launches_per_token() == 2
    ref_dec = OracleDecoder(Ws, mix, pre, states, keep, g, a.eps)
    rng = np.random.default_rng(70 + B)
    print(f"[stack decode] batch {B} kept {keep} L={L} d_model={d_model} nheads={H} g={g}",
          flush=True)
    for t in range(3):
        emb = rng.standard_normal((B, d_model)).astype(np.float32)
        a.emb.copy_(_d(emb))
        b.emb.copy_(_d(emb))
        xa = _bf16_to_f64(a.token())
        xb = _bf16_to_f64(b.token())
        ref = ref_dec.token(emb)
        torch.cuda.synchronize()
        assert xa.shape == ref.shape == (B, d_model)
        bar = 2.0 ** -7 * np.abs(ref) + 1e-3 * np.abs(ref).max(axis=1, keepdims=True)
        ra = (np.abs(xa - ref) / bar).max(axis=1)
        rb = (np.abs(xb - ref) / bar).max(axis=1)
        print(f"  token {t}: err/bar per row one launch {np.round(ra, 3).tolist()}, "
              f"layer by layer {np.round(rb, 3).tolist()}", flush=True)
        assert np.all(ra <= 1.0) and np.all(rb <= 1.0)
    assert _timeout_flag(a) == 0
    from oracle import ternary as O
    for l in range(L):
        conv_ref, ssm_ref = ref_dec.states[l]
        assert int(a.layers[l]["pos"].cpu()[0]) == 3
        for r in range(B):
            e = {}
            for name, dec in (("a", a), ("b", b)):
                lay = dec.layers[l]
                win = ring_to_window(lay["conv"].cpu().numpy(), int(lay["pos"].cpu()[0]))
                e[name] = (O.rel_fro_error(win[r].astype(np.float64),
                                           conv_ref[r].astype(np.float64)),
                           O.rel_fro_error(lay["ssm"].cpu().numpy()[r].astype(np.float64),
                                           ssm_ref[r].astype(np.float64)))
            for i in range(2):
                assert e["a"][i] <= max(1e-3, min(2 * e["b"][i], 4e-3)), (l, r, i, e)


def test_stack_decode_batch_rows_match_batch_one():
    """Each row of a batch-4 one-launch decode against batch-1 one-launch
    decodes of that row alone (same weights, states and embeddings): the two
    forms sum in different orders (the batched rows reduce through one
    four-way butterfly), so rows agree to the bars of the oracle test, and
    the row's states to 1e-3."""
    B, L, d_model, H = 4, 2, 512, 4
    a, Ws, mix, pre, states = _decoder(123, L, d_model, H, stack=True, batch=B)
    singles = []
    for r in range(B):
        d1, *_ = _decoder(123, L, d_model, H, stack=True, batch=1)
        for l in range(L):
            conv, ssm = states[l]
            d1.set_states(l, _d(conv[r:r + 1].view(np.int16)).view(torch.float16),
                          _d(ssm[r:r + 1].view(np.int16)).view(torch.float16))
        singles.append(d1)
    rng = np.random.default_rng(321)
    for t in range(2):
        emb = rng.standard_normal((B, d_model)).astype(np.float32)
        a.emb.copy_(_d(emb))
        xa = _bf16_to_f64(a.token())
        for r, d1 in enumerate(singles):
            d1.emb.copy_(_d(emb[r:r + 1]))
            x1 = _bf16_to_f64(d1.token())[0]
            bar = 2.0 ** -7 * np.abs(x1) + 1e-3 * np.abs(x1).max()
            assert np.all(np.abs(xa[r] - x1) <= 2 * bar), (t, r)
    assert _timeout_flag(a) == 0
    from oracle import ternary as O
    for l in range(L):
        for r, d1 in enumerate(singles):
            sa = a.layers[l]["ssm"].cpu().numpy()[r].astype(np.float64)
            s1 = d1.layers[l]["ssm"].cpu().numpy()[0].astype(np.float64)
            assert O.rel_fro_error(sa, s1) <= 1e-3, (l, r)


@pytest.mark.parametrize("B", [1, 4])
def test_stack_decode_graph_replays_match_eager(B):
    """The one-launch decode captured as a HIP graph (its barrier words are
    cleared by a fill kernel inside the graph): three tokens eagerly, then the
    same three from the same states as replays of one captured graph, with
    other GPU work and host syncs in between; outputs and every block's
    states agree bit for bit (the kernel sums in a fixed order)."""
    _need_cus(2 * B)
    dec, *_ = _decoder(31 + B, 3, 256, 2, stack=True, keep=(1,), batch=B)
    assert dec.stack and dec.B == B
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
    for lay, (c, s, p) in zip(dec.layers, init):   # capturing runs nothing
        assert torch.equal(lay["ssm"], s) and torch.equal(lay["pos"], p)
    for t, e in enumerate(emb):
        dec.emb.copy_(e)
        out = dec.replay()
        torch.cuda.synchronize()
        _ = torch.randn(1000, device="cuda").sum().item()   # unrelated work in between
        assert torch.equal(out, eager[t]), f"token {t}"
    assert _timeout_flag(dec) == 0
    for lay, (c, s, p) in zip(dec.layers, final_eager):
        assert torch.equal(lay["conv"], c) and torch.equal(lay["ssm"], s)
        assert torch.equal(lay["pos"], p)
