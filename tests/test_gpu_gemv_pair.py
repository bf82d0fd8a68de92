"""GPU parity of ``tm_tgemv_pair``: two strided stacks of decode GEMVs in one
launch, each against the oracle's float64 product (codes and float16 scales
from the oracle's ternarizer), and bit for bit against ``tm_tgemv`` where
that call takes the same one-workgroup-per-128-rows form."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import ternary as O  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

REL_DESIGN = 1e-4


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()
    return ops


def _ops():
    from paper_2606_18114_amd import ops
    return ops


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).cuda().view(
        torch.bfloat16)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def oracle_stack(rng, count, B, N, K, g, outliers):
    codes, s16s, qs, s16h = [], [], [], []
    for _ in range(count):
        W = synth.weights(rng, N, K, outliers)
        _, s32, q, _ = O.ternarize(W, g, 1e-5)
        s16 = O.scales_f16(s32)
        codes.append(torch.from_numpy(O.pack(q)).cuda())
        s16s.append(torch.from_numpy(s16.view(np.int16)).cuda().view(torch.float16))
        qs.append(q)
        s16h.append(s16)
    x = synth.activations(rng, count * B, K).reshape(count, B, K)
    return dev_bf16(x), torch.stack(codes), torch.stack(s16s), x, qs, s16h


@pytest.mark.parametrize("B,g,K1", [(1, 128, 4096), (4, 128, 4096), (2, 64, 1536),
                                    (1, 64, 192)])
def test_pair_against_oracle(B, g, K1):
    # in_proj- and out_proj-like stacks (ragged N); K1 = 192 at g = 64 gives
    # an odd number of groups per row, so the scales load differently from
    # the first stack and the call runs as two launches
    ops = _ops()
    rng = np.random.default_rng(B * 100 + g + K1)
    print(f"[gemv pair] B={B} g={g} stacks 3 x 520x2048, 2 x 264x{K1}", flush=True)
    a = oracle_stack(rng, 3, B, 520, 2048, g, True)
    b = oracle_stack(rng, 2, B, 264, K1, g, False)
    y0, y1 = ops.tgemv_pair(a[0], a[1], a[2], b[0], b[1], b[2], g)
    y0, y1 = host(y0), host(y1)
    errs = [O.rel_fro_error(y0[i], O.gemv(a[3][i], a[4][i], a[5][i], g)) for i in range(3)]
    errs += [O.rel_fro_error(y1[i], O.gemv(b[3][i], b[4][i], b[5][i], g)) for i in range(2)]
    print(f"  max rel fro err {max(errs):.3e}", flush=True)
    assert max(errs) <= REL_DESIGN


@pytest.mark.parametrize("B", [1, 4])
def test_pair_matches_two_calls_on_decode_stacks(B):
    """Stacks of the decode shapes large enough that tm_tgemv takes the same
    form (8 in_proj layers, 32 out_proj layers): the paired launch gives the
    same bits as two tm_tgemv calls.  Codes and scales are random bytes and
    float16 values here (no oracle: this compares two launch forms)."""
    ops = _ops()
    gen = torch.Generator(device="cuda").manual_seed(5 + B)
    shapes = [(8, synth.IN_PROJ_N, synth.D_MODEL), (32, synth.D_MODEL, synth.D_INNER)]
    st = []
    for count, N, K in shapes:
        c = torch.randint(0, 256, (count, N, K // 4), dtype=torch.uint8, device="cuda",
                          generator=gen)
        s = (torch.rand((count, N, K // 128), device="cuda", generator=gen) * 0.02 + 0.01
             ).to(torch.float16)
        x = torch.randn((count, B, K), device="cuda", generator=gen).to(torch.bfloat16)
        st.append((x, c, s))
    y0, y1 = ops.tgemv_pair(*st[0], *st[1], 128)
    r0 = ops.tgemv(*st[0], 128)
    r1 = ops.tgemv(*st[1], 128)
    torch.cuda.synchronize()
    assert torch.equal(y0, r0) and torch.equal(y1, r1)
