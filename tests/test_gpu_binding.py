"""The Python binding rejects tensors whose shape, dtype or device does not
match what the kernels assume, before anything is launched (the C ABI sees
only pointers and sizes, so it cannot check allocation sizes itself)."""

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()
    return ops


def _e(shape, dtype=torch.float32):
    return torch.zeros(shape, dtype=dtype, device="cuda")


def test_ternarize_outputs_checked(ops):
    W = _e((64, 256))
    bad = [dict(codes=_e((64, 32), torch.uint8)),
           dict(codes=_e((64, 64), torch.int8)),
           dict(scales=_e((64, 4))),
           dict(scales=_e((64, 2), torch.float16)),
           dict(scales_f16=_e((64, 4), torch.float16)),
           dict(zero_count=_e((1,), torch.int32)),
           dict(zero_count=_e((2,), torch.int64)),
           dict(zero_count=torch.zeros((1,), dtype=torch.int64))]
    for kw in bad:
        with pytest.raises((ValueError, TypeError)):
            ops.ternarize_pack(W, 128, 1e-5, **kw)
    with pytest.raises(ValueError):
        ops.ternarize_pack(W, 128, 1e-5, row_mult=_e((63,)))
    with pytest.raises((ValueError, TypeError)):
        ops.ternarize_codes(W, _e((64, 2)), 128, codes=_e((64, 63), torch.uint8))
    with pytest.raises((ValueError, TypeError)):
        ops.group_code_dot(_e((64, 64), torch.uint8), W, 128, out=_e((64, 3)))
    torch.cuda.synchronize()


def test_products_checked(ops):
    X = _e((32, 256), torch.bfloat16)
    codes, scales = _e((64, 64), torch.uint8), _e((64, 2))
    with pytest.raises(ValueError):
        ops.tgemm_fwd(X, _e((64, 32), torch.uint8), scales, 128)
    with pytest.raises(ValueError):
        ops.tgemm_fwd(X, codes, _e((64, 4)), 128)
    with pytest.raises(ValueError):
        ops.tgemm_fwd(X, codes, scales, 128, Y=_e((32, 63)))
    with pytest.raises(TypeError):
        ops.tgemm_fwd(X, codes, scales, 128, Y=_e((32, 64), torch.float16))
    dY = _e((32, 64), torch.bfloat16)
    with pytest.raises(ValueError):
        ops.tgemm_bwd_dx(_e((32, 65), torch.bfloat16), codes, scales, 128)
    with pytest.raises(ValueError):
        ops.tgemm_bwd_dx(dY, codes, scales, 128, dX=_e((32, 255)))
    with pytest.raises(ValueError):
        ops.tgemm_bwd_dw_ste(dY, _e((31, 256), torch.bfloat16))
    with pytest.raises(ValueError):
        ops.tgemm_bwd_dw_ste(dY, X, dW=_e((64, 255)))
    x = _e((3, 1, 256), torch.bfloat16)
    c3, s3 = _e((3, 64, 64), torch.uint8), _e((3, 64, 2), torch.float16)
    with pytest.raises(ValueError):
        ops.tgemv(x, _e((2, 64, 64), torch.uint8), s3, 128)
    with pytest.raises(ValueError):
        ops.tgemv(x, c3, _e((3, 64, 1), torch.float16), 128)
    with pytest.raises(ValueError):
        ops.tgemv(x, c3, s3, 128, y=_e((3, 2, 64)))
    torch.cuda.synchronize()


def test_stack_decode_checked(ops):
    """tm_mamba2_decode_token's arrays: the state arrays carry the batch
    dimension whenever the embedding is [B, d_model], x_out matches emb, and
    batches above 4 are refused (no case here reaches a launch)."""
    L, D, H, g = 2, 256, 2, 128
    di, cd = 64 * H, 64 * H + 256
    Z = 2 * di + 256 + H
    f16, u8 = torch.float16, torch.uint8

    def arrays(lead):
        return {"in_codes": _e((L, Z, D // 4), u8), "in_scales": _e((L, Z, D // g), f16),
                "out_codes": _e((L, D, di // 4), u8), "out_scales": _e((L, D, di // g), f16),
                "pre_w": _e((L, D)), "conv_w": _e((L, cd, 4)), "conv_b": _e((L, cd)),
                "dt_bias": _e((L, H)), "A_log": _e((L, H)), "D": _e((L, H)),
                "norm_w": _e((L, di)), "final_w": _e((D,)),
                "conv_state": _e(lead + (cd, 4), f16),
                "conv_pos": _e((L,), torch.int32), "ssm_state": _e(lead + (H, 64, 128), f16)}

    with pytest.raises(ValueError):   # three dims
        ops.mamba2_decode_token(arrays((L, 2)), g, 1e-5, _e((1, 2, D)))
    with pytest.raises(ValueError):   # batch-1 states for a batch of 2
        ops.mamba2_decode_token(arrays((L,)), g, 1e-5, _e((2, D)))
    with pytest.raises(ValueError):   # x_out not [B, d_model]
        ops.mamba2_decode_token(arrays((L, 2)), g, 1e-5, _e((2, D)),
                                x_out=_e((D,), torch.bfloat16))
    with pytest.raises((ValueError, RuntimeError)):   # batch 5
        ops.mamba2_decode_token(arrays((L, 5)), g, 1e-5, _e((5, D)))
    torch.cuda.synchronize()
