"""Layer-selective quantization (Sec. 7): the kept-block selection, the QAT
wiring (CPU), and a decode token over a mixed ternary / FP16 stack against
the oracle (GPU)."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import ternary as O  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402


def test_keep_first_last():
    from paper_2606_18114_amd.stack import keep_first_last
    assert keep_first_last(48, 2) == [0, 1, 46, 47]
    assert keep_first_last(48, 0) == []
    assert keep_first_last(4, 2) == [0, 1, 2, 3]
    with pytest.raises(ValueError):
        keep_first_last(3, 2)


class _Block(torch.nn.Module):
    def __init__(self, d, e):
        super().__init__()
        self.in_proj = torch.nn.Linear(d, 2 * e, bias=False)
        self.out_proj = torch.nn.Linear(e, d, bias=False)


def test_quantize_projections_keeps_the_selected_blocks():
    from paper_2606_18114_amd.qat import TernaryLinear
    from paper_2606_18114_amd.stack import keep_first_last, quantize_projections
    torch.manual_seed(0)
    blocks = torch.nn.ModuleList([_Block(128, 256) for _ in range(6)])
    ref = [(b.in_proj.weight.detach().clone(), b.out_proj.weight.detach().clone())
           for b in blocks]
    done = quantize_projections(blocks, keep_first_last(6, 1), g=64)
    assert done == [1, 2, 3, 4]
    for i, b in enumerate(blocks):
        kind = torch.nn.Linear if i in (0, 5) else TernaryLinear
        assert isinstance(b.in_proj, kind) and isinstance(b.out_proj, kind)
        assert torch.equal(b.in_proj.weight, ref[i][0])
        assert torch.equal(b.out_proj.weight, ref[i][1])
    assert blocks[2].in_proj.g == 64
    with pytest.raises(ValueError):
        quantize_projections(blocks, keep=[7])
    biased = torch.nn.ModuleList([_Block(128, 256)])
    biased[0].in_proj = torch.nn.Linear(128, 512, bias=True)
    with pytest.raises(TypeError):
        quantize_projections(biased)


@pytest.mark.gpu
@pytest.mark.parametrize("B", [1, 4])
def test_mixed_stack_decode_token(B):
    """Six layers, the first and last kept in FP16: every layer's in_proj and
    out_proj output against the oracle (ternary layers ternarized by the
    oracle, kept layers with their float16 weights).  The stack's codes equal
    the oracle's off the rounding-boundary band; a band element whose code
    differs widens that output's bar by its own product."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd.stack import DecodeStack, keep_first_last
    L, shapes, g = 6, {"in": (520, 256), "out": (256, 512)}, 128
    rng = np.random.default_rng(31 + B)
    Ws = {(k, l): synth.weights(rng, *shapes[k], outliers=(k == "in"))
          for k in shapes for l in range(L)}
    st = DecodeStack(lambda k, l: torch.from_numpy(Ws[(k, l)]).cuda(), L, shapes,
                     keep=keep_first_last(L, 1), g=g, batch=B)
    xs = {k: synth.activations(rng, L * B, shapes[k][1]).reshape(L, B, shapes[k][1])
          for k in shapes}
    for k in shapes:
        st.set_inputs(k, torch.from_numpy(xs[k].view(np.int16)).cuda().view(torch.bfloat16))
    st.token()
    torch.cuda.synchronize()
    for k, (N, K) in shapes.items():
        y = st.outputs(k).cpu().numpy()
        for l in range(L):
            if l in st.keep:
                W16 = Ws[(k, l)].astype(np.float16)
                assert np.array_equal(st.w16[k][st.keep.index(l)].cpu().numpy(), W16)
                ref = O.dense_gemv(xs[k][l], W16)
                err = O.rel_fro_error(y[l], ref)
                assert err <= 1e-6, (k, l, err)
            else:
                s64, s32, q, _ = O.ternarize(Ws[(k, l)], g, 1e-5)
                s16 = O.scales_f16(s32)
                t = st.tern.index(l)
                q_gpu = O.unpack(st.codes[k][t].cpu().numpy(), K)
                band = O.boundary_mask(Ws[(k, l)], s64, g, 1e-5)
                assert np.array_equal(q_gpu[~band], q[~band]), (k, l)
                s16_gpu = st.s16[k][t].cpu().numpy()
                ds = np.abs(s16_gpu.astype(np.float64) - s16.astype(np.float64))
                assert np.all(ds <= np.spacing(s16).astype(np.float64)), (k, l)
                ref = O.gemv(xs[k][l], q, s16, g)
                xa = np.abs(synth.bf16_bits_to_f32(xs[k][l]).astype(np.float64))
                sw = np.abs(O.dequantize(np.ones_like(q), s16.astype(np.float64), g))
                # a code off by up to 2 (band elements), a scale off by one step
                moved = (q_gpu != q) * 2 * (sw + O.dequantize(np.ones_like(q), ds, g)) \
                    + np.abs(O.dequantize(q, ds, g))
                bar = 1e-6 * (xa @ np.abs(O.dequantize(q, s16.astype(np.float64), g)).T) \
                    + xa @ moved.T + 1e-30
                assert np.all(np.abs(y[l] - ref) <= bar), (k, l)
    # bytes: 4 ternary layers of codes + scales, 2 kept layers in float16
    exp = sum(4 * (N * K / 4 + 2 * N * K / g) + 2 * 2 * N * K + L * (2 * B * K + 4 * B * N)
              for N, K in shapes.values())
    assert st.bytes_per_token() == exp


def test_decoder_refuses_kept_blocks_past_batch_8():
    """Blocks kept in FP16 decode through tm_dgemv, which takes batches up to
    8: the decoder says so when it is built, before touching any device."""
    torch = pytest.importorskip("torch")
    from paper_2606_18114_amd.stack import Mamba2Decoder

    def never(*a):
        raise AssertionError("no weight is read before the check")

    with pytest.raises(ValueError, match="batch 1 .. 8"):
        Mamba2Decoder(never, never, never, 3, 256, 2, keep=(1,), batch=16,
                      device=torch.device("cpu"))
