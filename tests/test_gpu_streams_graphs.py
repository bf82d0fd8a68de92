"""Stream semantics and graph capture of the C ABI.

Every entry point enqueues its kernels on the stream it is given and allocates
nothing; the clears it needs (zero count, dW, the forward's cut-tile rows) are
fill kernels, not memset nodes.  So the calls run on any stream and can be
captured into a HIP graph.  These tests run the whole in_proj-shaped step
(ternarize -> forward -> dX -> dW -> decode GEMV) on a side stream and as a
captured graph, replayed several times with other work in between and with
new inputs, and compare every result with the eager run on the default
stream.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2606_18114_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()  # raises if the library is missing: no fallback


def _bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).cuda().view(
        torch.bfloat16)


class Step:
    """Static buffers of one step; run() enqueues it on the current stream."""

    def __init__(self, M=700, N=600, K=512, g=128, seed=0):
        from paper_2606_18114_amd import ops
        self.ops, self.g = ops, g
        rng = np.random.default_rng(seed)
        self.W = torch.from_numpy(synth.weights(rng, N, K, outliers=True)).cuda()
        self.X = _bf16(synth.activations(rng, M, K))
        self.dY = _bf16(synth.activations(rng, M, N, std=0.01))
        self.x = _bf16(synth.activations(rng, 3 * 2, K)).view(3, 2, K)
        self.codes = torch.empty((N, K // 4), dtype=torch.uint8, device="cuda")
        self.s = torch.empty((N, K // g), dtype=torch.float32, device="cuda")
        self.s16 = torch.empty((N, K // g), dtype=torch.float16, device="cuda")
        self.zc = torch.empty((1,), dtype=torch.int64, device="cuda")
        self.Y = torch.empty((M, N), device="cuda")
        self.dX = torch.empty((M, K), device="cuda")
        self.dX2 = torch.empty((M, K), device="cuda")
        self.ws = torch.empty(ops.dx_f16_workspace_bytes(M, N), dtype=torch.uint8, device="cuda")
        self.dW = torch.empty((N, K), device="cuda")
        self.y = torch.empty((3, 2, N), device="cuda")

    def run(self):
        o, g = self.ops, self.g
        o.ternarize_pack(self.W, g, 1e-5, codes=self.codes, scales=self.s, scales_f16=self.s16,
                         zero_count=self.zc)
        o.tgemm_fwd(self.X, self.codes, self.s, g, Y=self.Y)
        o.tgemm_bwd_dx(self.dY, self.codes, self.s, g, dX=self.dX, workspace=self.ws)
        o.tgemm_bwd_dx(self.dY, self.codes, self.s, g, dX=self.dX2, precision="exact")
        o.tgemm_bwd_dw_ste(self.dY, self.X, dW=self.dW)
        # the same packed matrix three times over (count = 3, stride 0 is not
        # allowed, so the GEMV reads a stacked copy made by a kernel of torch)
        o.tgemv(self.x, self.codes.unsqueeze(0).expand(3, -1, -1).contiguous(),
                self.s16.unsqueeze(0).expand(3, -1, -1).contiguous(), g, y=self.y)

    def outputs(self):
        torch.cuda.synchronize()
        return {k: getattr(self, k).detach().cpu().clone()
                for k in ("codes", "s", "s16", "zc", "Y", "dX", "dX2", "dW", "y")}


# bit-exact: codes, scales, counts, the GEMV, and Y (its tiles are cut into
# two parts at most here, and two float32 partial sums add exactly in either
# order onto the cleared rows); dX and dW add many parts with atomics
EXACT = ("codes", "s", "s16", "zc", "Y", "y")


def _compare(got, ref, label):
    for k in ref:
        a, b = got[k], ref[k]
        if k in EXACT:
            assert torch.equal(a, b), f"{label}: {k} differs"
        else:  # dX (both forms), dW: float32 atomics over the cut contraction
            rel = float((a.double() - b.double()).norm() / b.double().norm())
            assert rel <= 1e-6, f"{label}: {k} rel {rel:.2e}"


def test_side_stream_matches_default_stream():
    st = Step()
    st.run()
    ref = st.outputs()
    side = torch.cuda.Stream()
    st.Y.fill_(float("nan"))
    st.dX.fill_(float("nan"))
    st.dX2.fill_(float("nan"))
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        st.run()
    side.synchronize()
    _compare(st.outputs(), ref, "side stream")


def test_graph_capture_and_replays():
    st = Step(seed=1)
    st.run()
    ref = st.outputs()
    graph = torch.cuda.CUDAGraph()
    # the GEMV's stacked copies are made inside run(); warm up the caching
    # allocator on a side stream before capture, as torch's graph rules ask
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        st.run()
    for rep in range(3):
        for t in (st.Y, st.dX, st.dX2, st.dW, st.y):
            t.fill_(float("nan"))   # eager work between replays
        st.ws.fill_(255)            # the dX workspace is scratch: garbage in it is fine
        st.zc.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        _compare(st.outputs(), ref, f"replay {rep}")
    # new inputs in the captured buffers: the replay recomputes everything
    st2 = Step(seed=2)
    st2.run()
    ref2 = st2.outputs()
    for a, b in ((st.W, st2.W), (st.X, st2.X), (st.dY, st2.dY), (st.x, st2.x)):
        a.copy_(b)
    torch.cuda.synchronize()
    graph.replay()
    _compare(st.outputs(), ref2, "replay with new inputs")


def test_graph_of_single_matrix_gemvs_in_layer_order():
    # decode as a model runs it: one launch per matrix, layer by layer; these
    # launches take the split-K form (partial sums added in LDS in a fixed
    # order), so a captured graph must reproduce the eager outputs bit for bit
    from paper_2606_18114_amd import ops
    rng = np.random.default_rng(7)
    layers = []
    for N, K in ((1200, 2048), (640, 4096), (1200, 2048), (640, 4096)):
        W = torch.from_numpy(synth.weights(rng, N, K, outliers=True)).cuda()
        c, _, s16, _ = ops.ternarize_pack(W, 128, 1e-5)
        x = _bf16(synth.activations(rng, 1, K)).view(1, 1, K)
        layers.append((x, c.unsqueeze(0), s16.unsqueeze(0), torch.empty((1, 1, N), device="cuda")))

    def run():
        for x, c, s, y in layers:
            ops.tgemv(x, c, s, 128, y=y)

    run()
    torch.cuda.synchronize()
    ref = [y.clone() for *_, y in layers]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    for rep in range(3):
        for *_, y in layers:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (*_, y) in enumerate(layers):
            assert torch.equal(y, ref[i]), f"replay {rep}: layer {i} differs"
