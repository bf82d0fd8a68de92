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
    out_proj output against the oracle (ternary layers with the stack's own
    codes and float16 scales, kept layers with their float16 weights)."""
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
            else:
                t = st.tern.index(l)
                q = O.unpack(st.codes[k][t].cpu().numpy(), K)
                s16 = st.s16[k][t].cpu().numpy()
                ref = O.gemv(xs[k][l], q, s16, g)
            err = O.rel_fro_error(y[l], ref)
            assert err <= 1e-6, (k, l, err)
    # bytes: 4 ternary layers of codes + scales, 2 kept layers in float16
    exp = sum(4 * (N * K / 4 + 2 * N * K / g) + 2 * 2 * N * K + L * (2 * B * K + 4 * B * N)
              for N, K in shapes.values())
    assert st.bytes_per_token() == exp
