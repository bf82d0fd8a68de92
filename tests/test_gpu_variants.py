"""GPU parity of the scale-variant entry points against the CPU oracle.

* tm_ternarize_pack_thresh: per-row threshold multipliers (the appendix's
  0.8 x absmean on the gate rows of in_proj);
* tm_ternarize_codes: codes against caller-given thresholds (the learned
  scale of Sec. 4);
* tm_group_code_dot: the gradient of a per-group magnitude, sum q * dWhat;
* tm_scale_ste_grad: a learnable scale's gradient with the rounding
  straight-through (threshold term, clip-masked weight gradient);
* TernaryLinear in its decoupled and learnable modes and with threshold
  multipliers, forward and backward.

Bars: given the GPU's own float32 scales, the oracle takes the same float32
decision, so codes and zero counts must match bit for bit; against the
oracle's own float64 scales they may differ only on elements flagged as
within 1e-6 of the rounding boundary.  Group dots are float64 sums rounded
once, held to one float32 rounding plus float64 summation error.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import ternary as O  # noqa: E402
from oracle import variants as V  # noqa: E402
from paper_2606_18114_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

REL_DESIGN = 1e-4
REL_BAR = 2e-3


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_18114_amd import ops
    ops.lib()  # raises if the library is missing: no fallback


def _ops():
    from paper_2606_18114_amd import ops
    return ops


def dev(a, dtype=np.float32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def dev_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).cuda().view(
        torch.bfloat16)


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def gate_mult(N, gate_rows=4096, m=0.8):
    mult = np.ones(N, np.float32)
    mult[:min(gate_rows, N)] = m
    return mult


def check_thresh(W, g, eps, mult, label):
    ops = _ops()
    N, K = W.shape
    print(f"[thresh] {label} N={N} K={K} g={g} eps={eps}", flush=True)
    c, s, s16, z = ops.ternarize_pack(dev(W), g, eps, row_mult=dev(mult))
    q = O.unpack(host(c), K)
    s_gpu, z_gpu = host(s), int(host(z)[0])
    # the stored scales are the plain absmean, whatever the multipliers
    s64 = O.group_scales_f64(W, g)
    s32 = s64.astype(np.float32)
    assert np.array_equal(s_gpu, s32) or \
        np.max(np.abs(s_gpu - s64) / np.maximum(s64, 1e-300)) <= 1e-6
    same = s_gpu == s32
    ref16 = O.scales_f16(s32)
    assert np.array_equal(host(s16).view(np.uint16)[same], ref16.view(np.uint16)[same])
    assert z_gpu == O.zero_count(q)
    # against the oracle's own decisions only boundary elements may differ
    q_orc = V.ternary_codes_thresh(W, s32, g, eps, mult)
    band = V.boundary_mask_thresh(W, s64, g, eps, mult)
    assert not np.any((q != q_orc) & ~band), f"{int(((q != q_orc) & ~band).sum())} codes differ"
    print(f"  zero ratio {z_gpu / W.size:.4f}, boundary elements {int(band.sum())}", flush=True)
    return q, s_gpu


def test_thresh_gate_rows_of_in_proj():
    W = synth.layer_weight(synth.C3, synth.SEED_W)
    mult = gate_mult(W.shape[0])
    q, _ = check_thresh(W, 128, 1e-5, mult, "in_proj 8512x2048, 0.8 on rows 0-4095")
    gate = float(np.mean(q[:4096] == 0))
    rest = float(np.mean(q[4096:] == 0))
    print(f"  gate-row zeros {gate:.4f}, other rows {rest:.4f}", flush=True)
    assert gate < rest  # a lower threshold keeps more weights


@pytest.mark.parametrize("g", synth.C5_GROUPS)
def test_thresh_ragged_rows_random_multipliers(g):
    rng = np.random.default_rng(100 + g)
    W = synth.weights(rng, 301, 1024, outliers=True)
    mult = rng.uniform(0.5, 2.0, 301).astype(np.float32)
    for eps in (0.0, 1e-5):
        check_thresh(W, g, eps, mult, "301x1024 random multipliers")


def test_thresh_unit_multipliers_are_the_standard_call():
    ops = _ops()
    W = dev(synth.weights(np.random.default_rng(7), 257, 2048, outliers=True))
    a = [host(t) for t in ops.ternarize_pack(W, 64, 1e-5)]
    b = [host(t) for t in ops.ternarize_pack(W, 64, 1e-5, row_mult=dev(np.ones(257)))]
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


# --------------------------------------------------------------------------
# codes against given thresholds
# --------------------------------------------------------------------------

def check_given(W, tau, g, eps, label):
    ops = _ops()
    N, K = W.shape
    print(f"[given] {label} N={N} K={K} g={g} eps={eps}", flush=True)
    c, z = ops.ternarize_codes(dev(W), dev(tau), g, eps)
    q = O.unpack(host(c), K)
    q_ref = O.ternary_codes(W, tau, g, eps)
    assert np.array_equal(q, q_ref), f"{int((q != q_ref).sum())} codes differ"
    assert int(host(z)[0]) == O.zero_count(q_ref)
    return q


@pytest.mark.parametrize("g", synth.C5_GROUPS)
def test_given_thresholds_ragged(g):
    rng = np.random.default_rng(200 + g)
    W = synth.weights(rng, 301, 1024, outliers=True)
    tau = (O.group_scales_f32(W, g) * rng.uniform(0.25, 4.0, (301, 1024 // g))).astype(np.float32)
    for eps in (0.0, 1e-5):
        check_given(W, tau, g, eps, "301x1024, thresholds 0.25-4 x absmean")


def test_given_thresholds_in_proj_and_ties():
    W = synth.layer_weight(synth.C3, synth.SEED_W)
    tau = (O.group_scales_f32(W, 128) * np.float32(1.3)).astype(np.float32)
    check_given(W, tau, 128, 1e-5, "in_proj 8512x2048, 1.3 x absmean")
    # exact ties |w| = tau / 2 at eps = 0 round to zero; just above does not
    T = np.zeros((2, 64), np.float32)
    T[0, :4] = [0.5, -0.5, np.nextafter(np.float32(0.5), np.float32(1)), -0.75]
    T[1, :] = 3.0
    q = check_given(T, np.array([[1.0], [2.0]], np.float32), 64, 0.0, "ties")
    assert q[0, :4].tolist() == [0, 0, 1, -1] and np.all(q[1] == 1)


def test_given_thresholds_tiny_and_huge():
    # The kernel tests |w| > d/2 in float32, halving d exactly, or truncating
    # its bits when d/2 falls below the normal range.  Thresholds across that
    # edge (subnormal, the two smallest normal binades), ordinary and huge
    # ones, each against the float32 neighbours of d/2: the float32 quotient
    # of the definition decides.
    f32 = np.float32
    ds = [2.0**-149, 3 * 2.0**-149, 2.0**-140 + 2.0**-149, 2.0**-126, 1.5 * 2.0**-126,
          2.0**-126 + 2.0**-149, 2.0**-125, 3 * 2.0**-125 + 2.0**-147, 0.3, 1.0, 3.0e38]
    rows, taus = [], []
    for d in ds:
        d32 = f32(d)
        assert float(d32) == d or d == 0.3 or d == 3.0e38
        h = float(d32) / 2.0                          # exact in float64
        lo = f32(h) if float(f32(h)) <= h else np.nextafter(f32(h), f32(0))
        cand = [lo, np.nextafter(lo, f32(np.inf)), np.nextafter(lo, f32(0)),
                np.nextafter(np.nextafter(lo, f32(np.inf)), f32(np.inf)), d32, f32(0)]
        row = np.zeros(64, np.float32)  # K = 64: two groups of 32, the same threshold
        vals = np.array(cand, np.float32)
        row[:len(vals)] = vals
        row[8:8 + len(vals)] = -vals
        row[32:] = row[:32]
        rows.append(row)
        taus.append([d32, d32])
    W = np.stack(rows)
    tau = np.array(taus, np.float32)
    q = check_given(W, tau, 32, 0.0, "tiny and huge thresholds")
    # sanity: the definition gives both codes on every row
    assert all(np.any(q[r] != 0) and np.any(q[r] == 0) for r in range(len(ds)))


def test_given_thresholds_equal_the_absmean_call():
    # the absmean itself as the given threshold reproduces tm_ternarize_pack
    ops = _ops()
    W = dev(synth.weights(np.random.default_rng(11), 333, 1024, outliers=True))
    c0, s, _, z0 = ops.ternarize_pack(W, 128, 1e-5)
    c1, z1 = ops.ternarize_codes(W, s, 128, 1e-5)
    assert np.array_equal(host(c0), host(c1)) and host(z0)[0] == host(z1)[0]


# --------------------------------------------------------------------------
# group code dot
# --------------------------------------------------------------------------

def check_gcd(q, dW, g, label):
    ops = _ops()
    N, K = dW.shape
    print(f"[group dot] {label} N={N} K={K} g={g}", flush=True)
    codes = dev(O.pack(q), np.uint8)
    out = host(ops.group_code_dot(codes, dev(dW), g))
    ref = V.group_code_dot(q, dW, g)
    mag = (np.abs(q.astype(np.float64)) * np.abs(dW.astype(np.float64))).reshape(
        N, K // g, g).sum(2)
    bound = 2.0 ** -24 * np.abs(ref) + 2.0 * g * 2.0 ** -53 * mag + 1e-300
    err = np.abs(out.astype(np.float64) - ref)
    assert np.all(err <= bound), f"max err / bound {np.max(err / bound):.3f}"
    return out


@pytest.mark.parametrize("g", synth.C5_GROUPS)
def test_group_dot_ragged(g):
    rng = np.random.default_rng(300 + g)
    N, K = 301, 1024
    q = rng.integers(-1, 2, (N, K)).astype(np.int8)
    dW = (rng.standard_normal((N, K)) * np.exp(rng.uniform(-8, 8, (N, 1)))).astype(np.float32)
    check_gcd(q, dW, g, "301x1024, row magnitudes e^-8..e^8")


def test_group_dot_in_proj_full():
    rng = np.random.default_rng(42)
    W = synth.layer_weight(synth.C3, synth.SEED_W)
    _, _, q, _ = O.ternarize(W, 128, 1e-5)
    dW = rng.standard_normal(W.shape, dtype=np.float32) * np.float32(1e-3)
    check_gcd(q, dW, 128, "in_proj 8512x2048 codes")


def test_group_dot_special_cases():
    g = 32
    q = np.zeros((4, 128), np.int8)
    dW = np.ones((4, 128), np.float32)
    q[1] = 1                              # every code +1: the group sum
    q[2] = -1                             # every code -1
    q[3, ::2], q[3, 1::2] = 1, -1         # cancelling pairs: exactly zero
    dW[3] = 0.375
    out = check_gcd(q, dW, g, "special cases")
    assert out[0].tolist() == [0.0] * 4
    assert out[1].tolist() == [32.0] * 4 and out[2].tolist() == [-32.0] * 4
    assert out[3].tolist() == [0.0] * 4


# --------------------------------------------------------------------------
# learnable scale with the rounding straight-through
# --------------------------------------------------------------------------

def check_ssg(W, s, dWhat, g, eps, label):
    ops = _ops()
    N, K = W.shape
    print(f"[scale ste grad] {label} N={N} K={K} g={g} eps={eps}", flush=True)
    Wd, sd, gd = dev(W), dev(s), dev(dWhat)
    codes, _ = ops.ternarize_codes(Wd, sd, g, eps)
    q = O.ternary_codes(W, s, g, eps)
    assert np.array_equal(O.unpack(host(codes), K), q)   # same float32 decisions
    ds, dw = ops.scale_ste_grad(Wd, codes, sd, gd, g, eps)
    ds, dw = host(ds), host(dw)
    ds_ref, dw_ref = V.scale_ste_grad(W, q, s, dWhat, g, eps)
    d = np.repeat((s + np.float32(eps)).astype(np.float32).astype(np.float64), g, axis=1)
    sf = np.repeat(s.astype(np.float64), g, axis=1)
    mag = (np.abs(dWhat.astype(np.float64)) * (np.abs(q) + np.abs(W) * sf / d ** 2)).reshape(
        N, K // g, g).sum(2)
    bound = 2.0 ** -24 * np.abs(ds_ref) + 4.0 * g * 2.0 ** -53 * mag + 1e-300
    err = np.abs(ds.astype(np.float64) - ds_ref)
    assert np.all(err <= bound), f"ds: max err / bound {np.max(err / bound):.3f}"
    # dw: one float32 rounding of a float64 product
    assert np.all(np.abs(dw.astype(np.float64) - dw_ref) <= 2.0 ** -24 * np.abs(dw_ref))
    # in place over dWhat gives the same bits
    gi = gd.clone()
    ds2, dw2 = ops.scale_ste_grad(Wd, codes, sd, gi, g, eps, in_place=True)
    assert dw2.data_ptr() == gi.data_ptr()
    assert np.array_equal(host(ds2), ds) and np.array_equal(host(gi), dw)
    # scale only
    ds3, none = ops.scale_ste_grad(Wd, codes, sd, gd, g, eps, want_dW=False)
    assert none is None and np.array_equal(host(ds3), ds)
    masked = int((dw_ref == 0).sum() - (dWhat == 0).sum())
    print(f"  clip-masked elements {masked}, max ds err / bound {np.max(err / bound):.3f}",
          flush=True)
    return q, ds, dw


@pytest.mark.parametrize("g", synth.C5_GROUPS)
@pytest.mark.parametrize("eps", [0.0, 1e-5])
def test_scale_ste_grad_ragged(g, eps):
    rng = np.random.default_rng(700 + g)
    N, K = 301, 1024
    W = synth.weights(rng, N, K, outliers=True)
    s = (O.group_scales_f32(W, g) * rng.uniform(0.6, 1.6, (N, K // g))).astype(np.float32)
    dWhat = (rng.standard_normal((N, K)) * np.exp(rng.uniform(-6, 6, (N, 1)))).astype(np.float32)
    check_ssg(W, s, dWhat, g, eps, "301x1024 outliers, scales 0.6..1.6 x absmean")


def test_scale_ste_grad_in_proj_full():
    rng = np.random.default_rng(43)
    W = synth.layer_weight(synth.C3, synth.SEED_W)
    s = O.group_scales_f32(W, 128) * np.float32(1.2)
    dWhat = rng.standard_normal(W.shape, dtype=np.float32) * np.float32(1e-3)
    check_ssg(W, s.astype(np.float32), dWhat, 128, 1e-5, "in_proj 8512x2048")


def test_scale_ste_grad_bounds_and_ties():
    """Weights exactly on the clip bound (|w| = s, eps = 0: m = 1), one float32
    step above it (m = 0), exact rounding ties (|w| = s/2: code 0) and zeros."""
    g = 32
    N, K = 4, 128
    s = np.full((N, K // g), 0.75, np.float32)
    W = np.zeros((N, K), np.float32)
    W[0, :] = 0.75
    W[1, :] = np.nextafter(np.float32(0.75), np.float32(1))
    W[2, ::2], W[2, 1::2] = 0.375, -0.375
    dWhat = np.linspace(-1, 1, N * K).astype(np.float32).reshape(N, K)
    q, ds, dw = check_ssg(W, s, dWhat, g, 0.0, "bounds and ties")
    assert np.all(q[0] == 1) and np.all(q[1] == 1) and np.all(q[2] == 0) and np.all(q[3] == 0)
    assert np.array_equal(dw[0], dWhat[0]) and not dw[1].any()   # closed clip range
    assert np.array_equal(dw[2], dWhat[2]) and np.array_equal(dw[3], dWhat[3])


# --------------------------------------------------------------------------
# TernaryLinear variants
# --------------------------------------------------------------------------

def _bits(t):
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("mode,mult", [("absmean", True), ("decoupled", False),
                                       ("decoupled", True), ("learnable", False),
                                       ("learnable_ste", False)])
def test_layer_variants_forward_backward(mode, mult):
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(51)
    N, K, g, eps = 200, 512, 64, 1e-5
    W = synth.weights(rng, N, K, outliers=True)
    m = gate_mult(N, gate_rows=96) if mult else None
    layer = TernaryLinear.from_weight(dev(W), g=g, eps=eps, scale_mode=mode,
                                      threshold_mult=None if m is None else dev(m))
    if layer.scale is not None:
        # move the learned scale off the absmean so that the magnitude matters
        with torch.no_grad():
            layer.scale.mul_(dev(rng.uniform(0.7, 1.4, layer.scale.shape)))
    print(f"[layer] mode={mode} threshold_mult={mult}", flush=True)
    x = dev_bf16(synth.f32_to_bf16_bits(rng.standard_normal((2, 40, K), dtype=np.float32)))
    x.requires_grad_(True)
    r = dev(rng.standard_normal((2, 40, N), dtype=np.float32))
    y = layer(x)
    (y * r).sum().backward()
    torch.cuda.synchronize()

    if mode in ("learnable", "learnable_ste"):
        mag = host(layer.scale)
        q = O.ternary_codes(W, mag, g, eps)
    else:
        # the layer's absmean thresholds: the oracle's float32 scales (the
        # library's agree to 1e-6, so decisions differ on the band only)
        s64 = O.group_scales_f64(W, g)
        s32 = s64.astype(np.float32)
        mag = s32 if mode == "absmean" else host(layer.scale)
        mm = m if mult else np.ones(N, np.float32)
        q = V.ternary_codes_thresh(W, s32, g, eps, mm)
        band = V.boundary_mask_thresh(W, s64, g, eps, mm)
    codes, _ = layer.pack_for_decode()
    q_gpu = O.unpack(host(codes), K)
    if mode in ("learnable", "learnable_ste"):
        assert np.array_equal(q_gpu, q)
        assert layer.zero_ratio() == O.zero_count(q) / q.size
    else:
        assert not np.any((q_gpu != q) & ~band)
        assert abs(layer.zero_ratio() * q.size - O.zero_count(q)) <= int(band.sum())

    xb = _bits(x).reshape(-1, K)
    rb = synth.f32_to_bf16_bits(host(r).reshape(-1, N))
    e_y = O.rel_fro_error(host(y).reshape(-1, N), O.gemm_fwd(xb, q, mag, g))
    e_dx = O.rel_fro_error(host(x.grad.float()).reshape(-1, K), O.gemm_bwd_dx(rb, q, mag, g))
    dw_ref = O.gemm_bwd_dw(rb, xb)
    dw_hat = dw_ref
    if mode == "learnable_ste":
        ds_ste, dw_ref = V.scale_ste_grad(W, q, mag, dw_hat, g, eps)
    e_dw = O.rel_fro_error(host(layer.weight.grad), dw_ref)
    print(f"  y {e_y:.2e} dX {e_dx:.2e} dW {e_dw:.2e}", flush=True)
    assert e_y <= REL_DESIGN and e_dx <= REL_BAR and e_dw <= REL_DESIGN
    if layer.scale is None:
        assert [n for n, _ in layer.named_parameters()] == ["weight"]
    else:
        ds = host(layer.scale.grad)
        ds_ref = ds_ste if mode == "learnable_ste" else V.group_code_dot(q, dw_hat, g)
        e_ds = O.rel_fro_error(ds, ds_ref)
        print(f"  d scale {e_ds:.2e}", flush=True)
        assert e_ds <= REL_DESIGN


def test_layer_learned_scales_move_under_sgd():
    from paper_2606_18114_amd.qat import TernaryLinear
    rng = np.random.default_rng(6)
    N, K, M = 128, 256, 512
    x = dev_bf16(synth.f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32)))
    t = x.float() @ dev(synth.weights(rng, N, K) * 3.0).t()
    W0 = synth.weights(rng, N, K)
    for mode in ("decoupled", "learnable"):
        layer = TernaryLinear.from_weight(dev(W0), scale_mode=mode)
        s0 = host(layer.scale).copy()
        opt = torch.optim.SGD(layer.parameters(), lr=0.5)
        losses = []
        for _ in range(20):
            opt.zero_grad()
            loss = ((layer(x) - t) ** 2).mean()
            loss.backward()
            opt.step()
            losses.append(float(loss.detach()))
        moved = float(np.abs(host(layer.scale) - s0).max() / np.abs(s0).max())
        print(f"[layer sgd] {mode}: loss {losses[0]:.4f} -> {losses[-1]:.4f}, "
              f"scale moved {moved:.3f}", flush=True)
        assert min(losses[1:]) < losses[0] and moved > 0.01
