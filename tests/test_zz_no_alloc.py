"""tm_mixer_step_noalloc (the allocation-free variant of tm_mixer_step,
whose workspace is the library's own device array) against tm_mixer_step
through the C ABI: two calls in a row, the second smaller, each checked bit
for bit against the workspace call on the same inputs and states."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_18114_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


def _d(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(rng, B, H):
    prm = {k: _d(v) for k, v in synth.mixer_params(rng, H).items()}
    conv, ssm = synth.mixer_states(rng, B, H)
    z = _d(synth.in_proj_out(rng, B, H))
    return prm, conv, ssm, z


def _run(ops, prm, conv, ssm, z, noalloc):
    conv_t = _d(conv.view(np.int16)).view(torch.float16)
    ssm_t = _d(ssm.view(np.int16)).view(torch.float16)
    pos = torch.zeros((1,), dtype=torch.int32, device="cuda")
    out = ops.mixer_step(z, conv_t, pos, ssm_t, prm["conv_w"], prm["conv_b"], prm["dt_bias"],
                         prm["A_log"], prm["D"], prm["norm_w"], 1e-5, noalloc=noalloc)
    torch.cuda.synchronize()
    return [t.cpu() for t in (out, conv_t, ssm_t, pos)]


def test_noalloc_matches_the_workspace_call():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()
    rng = np.random.default_rng(77)
    # first a full layer at batch 4, then a smaller call (batch 1, 5 heads):
    # the shared array keeps the first call's contents, which must not leak
    for B, H in ((4, 64), (1, 5)):
        prm, conv, ssm, z = _case(rng, B, H)
        print(f"[noalloc] B={B} nheads={H}", flush=True)
        ref = _run(ops, prm, conv, ssm, z, noalloc=False)
        got = _run(ops, prm, conv, ssm, z, noalloc=True)
        for a, b in zip(ref, got):
            assert torch.equal(a, b)
