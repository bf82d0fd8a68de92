"""TernaryLinear: the QAT layer built on the library's entry points.

GPU tests check one forward + straight-through backward against the float64
oracle (with the layer's own codes and scales), a few optimizer steps, the
zero-ratio readout and the decode packing.  The CPU tests check the argument
errors, which are raised before any library call.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import ternary as O  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402

REL_BAR = 2e-3
REL_DESIGN = 1e-4


def test_layer_rejects_bad_shapes_and_cpu_tensors():
    from paper_2606_18114_amd.qat import TernaryLinear
    with pytest.raises(ValueError):
        TernaryLinear(500, 64, g=128)  # in_features not a multiple of g
    layer = TernaryLinear(256, 64, g=128)
    with pytest.raises(ValueError, match="GPU"):
        layer(torch.zeros((4, 256), dtype=torch.bfloat16))  # no CPU fallback


@pytest.mark.parametrize("mode", ["decoupled", "learnable"])
def test_loaded_scale_is_not_reset(mode):
    """A learned scale restored with load_state_dict (a checkpoint or a resumed
    run) marks the layer initialised, so the first forward keeps it instead of
    resetting it to the absmean; a fresh layer still starts uninitialised."""
    from paper_2606_18114_amd.qat import TernaryLinear
    trained = TernaryLinear(256, 64, g=128, scale_mode=mode)
    with torch.no_grad():
        trained.scale.copy_(torch.linspace(0.01, 0.05, trained.scale.numel()).view_as(
            trained.scale))
    trained._scale_ready = True
    fresh = TernaryLinear(256, 64, g=128, scale_mode=mode)
    assert not fresh._scale_ready
    fresh.load_state_dict(trained.state_dict())
    assert fresh._scale_ready
    assert torch.equal(fresh.scale, trained.scale)
    # nested under a prefix (a model holding the layer)
    outer = torch.nn.Sequential(TernaryLinear(256, 64, g=128, scale_mode=mode))
    outer.load_state_dict(torch.nn.Sequential(trained).state_dict())
    assert outer[0]._scale_ready and torch.equal(outer[0].scale, trained.scale)


def _bf16(a):
    return torch.from_numpy(np.ascontiguousarray(synth.f32_to_bf16_bits(a)).view(np.int16)).cuda() \
        .view(torch.bfloat16)


def _bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def _oracle_codes(W, g, eps=1e-5):
    """The oracle's codes and float32 scales of the layer's weight (the
    layer's own may differ on rounding-boundary elements only)."""
    _, s32, q, _ = O.ternarize(W, g, eps)
    return q, s32


@pytest.mark.gpu
@pytest.mark.parametrize("g,dx_precision", [(64, "f16"), (128, "f16"), (128, "exact")])
def test_forward_backward_against_oracle(g, dx_precision):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(31 + g)
    N, K = 200, 512
    W = synth.weights(rng, N, K, outliers=True)
    layer = TernaryLinear.from_weight(torch.from_numpy(W).cuda(), g=g, dx_precision=dx_precision)
    xf = rng.standard_normal((3, 40, K), dtype=np.float32)
    x = _bf16(xf).requires_grad_(True)
    r = torch.from_numpy(rng.standard_normal((3, 40, N), dtype=np.float32)).cuda()
    y = layer(x)
    assert y.shape == (3, 40, N) and y.dtype == torch.float32
    (y * r).sum().backward()
    torch.cuda.synchronize()

    q, s = _oracle_codes(W, g)
    xb = _bits(x).reshape(-1, K)
    rb = synth.f32_to_bf16_bits(r.cpu().numpy().reshape(-1, N))  # the gradient is taken in bf16
    e_y = O.rel_fro_error(y.detach().cpu().numpy().reshape(-1, N), O.gemm_fwd(xb, q, s, g))
    e_dx = O.rel_fro_error(x.grad.float().cpu().numpy().reshape(-1, K), O.gemm_bwd_dx(rb, q, s, g))
    e_dw = O.rel_fro_error(layer.weight.grad.cpu().numpy(), O.gemm_bwd_dw(rb, xb))
    print(f"[qat] g={g} {dx_precision} y {e_y:.2e} dX (bf16) {e_dx:.2e} dW {e_dw:.2e}", flush=True)
    assert e_y <= REL_DESIGN
    assert e_dx <= REL_BAR  # dX is returned in the activations' dtype (bf16)
    assert e_dw <= REL_DESIGN
    # the scale is recomputed, never learned: no gradient reaches anything but W and x
    assert [n for n, _ in layer.named_parameters()] == ["weight"]


@pytest.mark.gpu
def test_sgd_steps_follow_the_straight_through_gradient():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(5)
    N, K, M, lr = 128, 256, 512, 2.0
    target_w = synth.weights(rng, N, K) * 4.0
    layer = TernaryLinear.from_weight(torch.from_numpy(synth.weights(rng, N, K)).cuda())
    x = _bf16(rng.standard_normal((M, K), dtype=np.float32))
    t = x.float() @ torch.from_numpy(target_w).cuda().t()
    opt = torch.optim.SGD(layer.parameters(), lr=lr)
    losses = []
    for step in range(30):
        opt.zero_grad()
        y = layer(x)
        loss = ((y - t) ** 2).mean()
        loss.backward()
        if step == 0:
            # one update is exactly W - lr * dY^T X with dY = bf16(2 (y - t) / (M N))
            w0 = layer.weight.detach().cpu().numpy().copy()
            dy = synth.f32_to_bf16_bits((2.0 * (y - t) / (M * N)).detach().cpu().numpy())
            dw_ref = O.gemm_bwd_dw(dy, _bits(x))
            opt.step()
            w1 = layer.weight.detach().cpu().numpy()
            upd = (w0 - w1) / lr
            err = O.rel_fro_error(upd, dw_ref)
            print(f"[qat] first update vs oracle dW: rel err {err:.2e}", flush=True)
            assert err <= 1e-3  # float32 subtraction of small updates from the weights
        else:
            opt.step()
        losses.append(float(loss.detach()))
    print(f"[qat] loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
    assert losses[-1] < 0.5 * losses[0]


@pytest.mark.gpu
def test_zero_ratio_and_decode_packing():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(8)
    N, K, g = 192, 1024, 128
    W = synth.weights(rng, N, K, outliers=True)
    layer = TernaryLinear.from_weight(torch.from_numpy(W).cuda(), g=g)
    x = _bf16(rng.standard_normal((4, K), dtype=np.float32))
    layer(x)
    s64, _, q_ref, z_ref = O.ternarize(W, g, 1e-5)
    z = layer.zero_ratio() * N * K
    assert abs(z - z_ref) <= int(O.boundary_mask(W, s64, g, 1e-5).sum())
    codes, s16 = layer.pack_for_decode()
    y = ops.tgemv(x[None], codes[None], s16[None], g)[0]
    torch.cuda.synchronize()
    band = O.boundary_mask(W, s64, g, 1e-5)
    assert np.array_equal(O.unpack(codes.cpu().numpy(), K)[~band], q_ref[~band])
    ref = O.gemv(_bits(x), q_ref, O.scales_f16(s64.astype(np.float32)), g)
    assert O.rel_fro_error(y.cpu().numpy(), ref) <= REL_DESIGN


@pytest.mark.gpu
def test_bf16_output_layer():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(77)
    N, K, g = 256, 512, 128
    W = synth.weights(rng, N, K, outliers=True)
    layer = TernaryLinear.from_weight(torch.from_numpy(W).cuda(), g=g, out_dtype=torch.bfloat16)
    x = _bf16(rng.standard_normal((64, K), dtype=np.float32)).requires_grad_(True)
    y = layer(x)
    assert y.dtype == torch.bfloat16
    r = _bf16(rng.standard_normal((64, N), dtype=np.float32) * 0.01)
    y.backward(r)
    torch.cuda.synchronize()
    q, s = _oracle_codes(W, g)
    xb, rb = _bits(x), _bits(r)
    e_y = O.rel_fro_error(y.detach().float().cpu().numpy(), O.gemm_fwd(xb, q, s, g))
    e_dx = O.rel_fro_error(x.grad.float().cpu().numpy(), O.gemm_bwd_dx(rb, q, s, g))
    e_dw = O.rel_fro_error(layer.weight.grad.cpu().numpy(), O.gemm_bwd_dw(rb, xb))
    print(f"[qat bf16 out] y {e_y:.2e} dX {e_dx:.2e} dW {e_dw:.2e}", flush=True)
    assert e_y <= REL_BAR and e_dx <= REL_BAR and e_dw <= REL_DESIGN


@pytest.mark.gpu
@pytest.mark.parametrize("mode", ["decoupled", "learnable"])
def test_reloaded_learned_layer_gives_the_same_outputs(mode):
    from paper_2606_18114_amd.qat import TernaryLinear
    torch.manual_seed(3)
    layer = TernaryLinear(512, 256, g=128, scale_mode=mode, device="cuda")
    x = _bf16(np.random.default_rng(3).standard_normal((32, 512)).astype(np.float32))
    layer(x)                                   # initialises the scale from the absmean
    with torch.no_grad():
        layer.scale.mul_(1.37)                 # a "trained" scale, away from the absmean
    y0 = layer(x).detach().clone()
    fresh = TernaryLinear(512, 256, g=128, scale_mode=mode, device="cuda")
    fresh.load_state_dict(layer.state_dict())
    y1 = fresh(x).detach()
    torch.cuda.synchronize()
    assert torch.equal(fresh.scale, layer.scale)
    assert torch.equal(y0, y1)
