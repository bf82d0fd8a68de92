"""One-GPU benchmark of the ternary linear hot path on MI355X.

A step is one pass of the whole path on synthetic Mamba-2 1.3B-shaped data:
  * in_proj QAT step (8512 x 2048 weights, 16384 tokens, g = 128):
    ternarize_pack -> tgemm_fwd -> tgemm_bwd_dx (one float16 pass, its
    prepass included) -> tgemm_bwd_dw_ste;
  * one decode token over all 48 layers: the GEMV over the 48 packed in_proj
    matrices and the 48 packed out_proj matrices (batch 1), both stacks in
    one launch (tm_tgemv_pair).
All inputs are resident in HBM before the timed region.  Per-kernel times
come from HIP events recorded on the stream the kernels run on.

The headline `value` is the in_proj forward ternary GEMM in TFLOP/s
(2*M*N*K algorithmic flops over the kernel's mean duration); every other
kernel is reported beside it.  The decode GEMV is also timed the way a server
runs it, tokens back to back (batch 1 and 4), after the step loop, warm (one
weight arena) and cold (tokens cycling over copies of the arenas, >= 1.1 GiB
in all, so nothing is left in the 256 MB memory-side cache); the cold batch-1
figure is `roofline_tgemv`.  The HBM-bound ternarizers are reported cold and
warm the same way (`cold_vs_warm`).  `small_configs` has the single linear
layer's latency and the out_proj forward, `group_sweep` the group sizes 32 ..
512 on in_proj with 2048 tokens, `codes_vs_oracle` the in_proj codes against
the oracle's (boundary-band elements and mismatches on and off the band).

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
    python bench.py --sweep-g     # group-size workload: one JSON line per g
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0     # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true")
    ap.add_argument("--decode-batch", type=int, default=1)
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--sweep-g", action="store_true",
                    help="group-size workload (in_proj W, X 2048 x 2048, g = 32 .. 512)")
    ap.add_argument("--micro", action="store_true",
                    help="measured roofline denominators instead of the step: an MFMA loop "
                         "(random and zero operands), a 1 GiB HBM read stream, a 1 GiB device "
                         "copy, and torch.mm bf16 on the in_proj shape as context")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="leave out the measured MFMA-loop and read-stream ceilings")
    ap.add_argument("--skip", default="",
                    help="comma list of optional sections to leave out: qat, variants, "
                         "per_layer, small, sweep, mixed, blocks, cold, dx_exact (keeps a profiler trace to the "
                         "kernels of interest)")
    args = ap.parse_args()
    args.skip = {x for x in args.skip.split(",") if x}
    bad = args.skip - {"qat", "variants", "per_layer", "small", "sweep", "mixed", "blocks", "cold",
                       "dx_exact"}
    if bad:
        ap.error(f"unknown --skip sections: {sorted(bad)}")
    return args


def log(msg):
    print(msg, file=sys.stderr, flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
KERNEL_SOURCES = {"tgemm_fwd": "tgemm_fwd.hip", "tgemv_pair": "tgemv.hip"}


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE counters (scaled by a plain-copy calibration), or None when
    there are none or the kernel source has changed since they were taken."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)["kernels"][kernel]
    except (OSError, KeyError, ValueError):
        return None
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_18114_amd", "csrc")
    for name in (KERNEL_SOURCES[kernel], "common.hpp"):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != rec.get("source_sha256"):
        return None
    return int(rec["read_bytes"]) + int(rec["write_bytes"])


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path is built for one GPU; sharding across GPUs is not)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_18114_amd import ops, synth

    if args.sweep_g:
        return sweep_g(args)
    if args.micro:
        return micro(args)
    if not os.path.exists(ops.lib_path()):
        from paper_2606_18114_amd import build
        build.build()
    ops.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def bf16(bits):
        return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)

    # ---------------- in_proj QAT step inputs ----------------
    cfg = synth.C3
    M, N, K, g, eps = cfg.M, cfg.N, cfg.K, cfg.g, cfg.eps
    t0 = time.time()
    W_h = synth.layer_weight(cfg, synth.SEED_W)
    X_h = synth.layer_acts(M, K, synth.SEED_X)
    dY_h = synth.layer_acts(M, N, synth.SEED_DY, std=synth.DY_STD)
    W = torch.from_numpy(W_h).to(dev)
    X = bf16(X_h)
    dY = bf16(dY_h)
    codes = torch.empty((N, K // 4), dtype=torch.uint8, device=dev)
    scales = torch.empty((N, K // g), dtype=torch.float32, device=dev)
    s16 = torch.empty((N, K // g), dtype=torch.float16, device=dev)
    zc = torch.empty((1,), dtype=torch.int64, device=dev)
    Y = torch.empty((M, N), dtype=torch.float32, device=dev)
    dX = torch.empty((M, K), dtype=torch.float32, device=dev)
    dW = torch.empty((N, K), dtype=torch.float32, device=dev)
    dx_ws = torch.empty(ops.dx_f16_workspace_bytes(M, N), dtype=torch.uint8, device=dev)
    log(f"in_proj inputs ready in {time.time() - t0:.1f}s")

    # ---------------- decode: 48 layers of packed weights ----------------
    t0 = time.time()
    L = synth.N_LAYERS
    B = args.decode_batch
    dec = {}
    for kind, dcfg in (("in", synth.DECODE_IN), ("out", synth.DECODE_OUT)):
        n, k = dcfg.N, dcfg.K
        arena_c = torch.empty((L, n, k // 4), dtype=torch.uint8, device=dev)
        arena_s = torch.empty((L, n, k // dcfg.g), dtype=torch.float16, device=dev)
        tmp_s = torch.empty((n, k // dcfg.g), dtype=torch.float32, device=dev)
        for layer in range(L):
            Wl = torch.from_numpy(synth.layer_weight(dcfg, synth.decode_seed(f"{kind}_w", layer)))
            ops.ternarize_pack(Wl.to(dev), dcfg.g, dcfg.eps, codes=arena_c[layer], scales=tmp_s,
                               scales_f16=arena_s[layer], want_zero_count=False)
        xs = np.stack([synth.layer_acts(B, k, synth.decode_seed(f"{kind}_x", layer))
                       for layer in range(L)])
        x4 = np.stack([synth.layer_acts(4, k, synth.decode_seed(f"{kind}_x", layer))
                       for layer in range(L)])
        dec[kind] = dict(cfg=dcfg, codes=arena_c, s16=arena_s, x=bf16(xs),
                         y=torch.empty((L, B, n), dtype=torch.float32, device=dev),
                         x4=bf16(x4), y4=torch.empty((L, 4, n), dtype=torch.float32, device=dev))
    torch.cuda.synchronize()
    log(f"decode arenas ready in {time.time() - t0:.1f}s")

    names = ["ternarize_pack", "tgemm_fwd", "tgemm_bwd_dx", "tgemm_bwd_dw_ste", "tgemv_pair"]

    def decode_token(xk, yk, arenas=None):
        """One decode token over the 48 in_proj and 48 out_proj matrices in
        one launch (tm_tgemv_pair); arenas: (in codes, in s16, out codes, out
        s16) to read instead of the resident ones."""
        a, b = dec["in"], dec["out"]
        ci, si, co, so = arenas or (a["codes"], a["s16"], b["codes"], b["s16"])
        ops.tgemv_pair(a[xk], ci, si, b[xk], co, so, a["cfg"].g, y0=a[yk], y1=b[yk])

    def step(ev):
        ev[0].record()
        ops.ternarize_pack(W, g, eps, codes=codes, scales=scales, scales_f16=s16, zero_count=zc)
        ev[1].record()
        ops.tgemm_fwd(X, codes, scales, g, Y=Y)
        ev[2].record()
        ops.tgemm_bwd_dx(dY, codes, scales, g, dX=dX, workspace=dx_ws)
        ev[3].record()
        ops.tgemm_bwd_dw_ste(dY, X, dW=dW)
        ev[4].record()
        decode_token("x", "y")
        ev[5].record()

    mk = lambda: [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for _ in range(args.warmup):
        step(mk())
    torch.cuda.synchronize()
    events = [mk() for _ in range(args.steps)]
    torch.cuda.synchronize()
    torch.cuda._sleep(2_000_000)  # the GPU spins while the host queues the first launches
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = wall * 1e3 / args.steps

    per = {n: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in events]))
           for i, n in enumerate(names)}

    # the two-pass dX (16 bits of every scale) on the same operands, for comparison
    dx_exact_ms = None
    if "dx_exact" not in args.skip:
        for _ in range(2):
            ops.tgemm_bwd_dx(dY, codes, scales, g, dX=dX, precision="exact")
        ex = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(max(args.steps // 2, 3))]
        for a, b in ex:
            a.record()
            ops.tgemm_bwd_dx(dY, codes, scales, g, dX=dX, precision="exact")
            b.record()
        torch.cuda.synchronize()
        dx_exact_ms = float(np.mean([a.elapsed_time(b) for a, b in ex]))

    # ---------------- decode as a server runs it: tokens back to back ----------------
    def serving(batch, tokens):
        """(in_proj ms, out_proj ms, two-launch token ms, one-launch token ms)"""
        xk, yk = ("x", "y") if batch == B else ("x4", "y4")
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(tokens)]
        for _ in range(3):
            for kind in ("in", "out"):
                d = dec[kind]
                ops.tgemv(d[xk], d["codes"], d["s16"], d["cfg"].g, y=d[yk])
        torch.cuda.synchronize()
        torch.cuda._sleep(2_000_000)
        for t in range(tokens):
            for i, kind in enumerate(("in", "out")):
                d = dec[kind]
                ev[t][i].record()
                ops.tgemv(d[xk], d["codes"], d["s16"], d["cfg"].g, y=d[yk])
            ev[t][2].record()
        torch.cuda.synchronize()
        # the same tokens with one event pair around the run: per-kernel events
        # add a few microseconds each, which a server does not pay
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(2_000_000)
        e0.record()
        for t in range(tokens):
            for kind in ("in", "out"):
                d = dec[kind]
                ops.tgemv(d[xk], d["codes"], d["s16"], d["cfg"].g, y=d[yk])
        e1.record()
        torch.cuda.synchronize()
        two = e0.elapsed_time(e1) / tokens
        # ... and in one launch per token
        for _ in range(3):
            decode_token(xk, yk)
        torch.cuda.synchronize()
        torch.cuda._sleep(2_000_000)
        e0.record()
        for t in range(tokens):
            decode_token(xk, yk)
        e1.record()
        torch.cuda.synchronize()
        return (float(np.mean([e[0].elapsed_time(e[1]) for e in ev])),
                float(np.mean([e[1].elapsed_time(e[2]) for e in ev])),
                two, e0.elapsed_time(e1) / tokens)
    serve = {b: serving(b, max(args.steps, 10)) for b in sorted({B, 4})}
    cold = ({} if "cold" in args.skip
            else cold_figures(ops, dec, W, dW, codes, scales, g, eps, max(args.steps // 4, 3),
                              decode_token))
    small = None if "small" in args.skip else small_configs(ops, dev, args.steps)
    sweep = None if "sweep" in args.skip else group_sweep(ops, dev, max(args.steps // 2, 5))

    # ---------------- decode in layer order: one launch per matrix ----------------
    per_layer = (None if "per_layer" in args.skip
                 else decode_per_layer(ops, dec, L, max(args.steps, 10)))
    mixed = None if "mixed" in args.skip else decode_mixed_stack(dev, max(args.steps // 4, 3))
    blocks = None
    if "blocks" not in args.skip:
        from paper_2606_18114_amd.stack import keep_first_last
        blocks = {"all_ternary_one_launch": decode_mamba2_blocks(dev, args.steps, stack=True),
                  "all_ternary": decode_mamba2_blocks(dev, args.steps),
                  "all_ternary_unfused": decode_mamba2_blocks(dev, args.steps, fused=False),
                  "first_last_2_fp16": decode_mamba2_blocks(
                      dev, args.steps, keep=keep_first_last(synth.N_LAYERS, 2)),
                  "first_last_2_fp16_one_launch": decode_mamba2_blocks(
                      dev, args.steps, keep=keep_first_last(synth.N_LAYERS, 2), stack=True),
                  "all_ternary_B4": decode_mamba2_blocks(dev, args.steps, batch=4),
                  "all_ternary_B4_one_launch": decode_mamba2_blocks(dev, args.steps, batch=4,
                                                                    stack=True),
                  "all_ternary_B16_unfused": decode_mamba2_blocks(dev, args.steps, batch=16,
                                                                  fused=False)}

    # ---------------- QAT block: both projections through autograd ----------------
    qat_block = None if "qat" in args.skip else qat_block_step(args, dev, X, synth)
    qat_block_bf16 = (None if "qat" in args.skip
                      else qat_block_step(args, dev, X, synth, out_dtype=torch.bfloat16))

    # ---------------- scale variants on the in_proj shapes ----------------
    variants = (None if "variants" in args.skip
                else variants_step(args, ops, W, scales, codes, dW, g, eps))

    # ---------------- algorithmic work per launch ----------------
    fl = 2.0 * M * N * K
    dcfg_in, dcfg_out = synth.DECODE_IN, synth.DECODE_OUT

    def gemv_bytes(c, batch=B):
        return L * (c.N * c.K / 4 + 2 * c.N * c.K / c.g + 2 * batch * c.K + 4 * batch * c.N)

    work = {
        "ternarize_pack": ("hbm", N * K * (4 + 0.25 + 4 / g + 2 / g)),
        "tgemm_fwd": ("mfma", fl),
        "tgemm_bwd_dx": ("mfma", fl),
        "tgemm_bwd_dw_ste": ("mfma", fl),
        "tgemv_pair": ("hbm", gemv_bytes(dcfg_in) + gemv_bytes(dcfg_out)),
    }
    kernels = {}
    for n in names:
        bound, amount = work[n]
        sec = per[n] * 1e-3
        if bound == "mfma":
            ach = amount / sec / 1e12
            kernels[n] = dict(ms=round(per[n], 4), bound="mfma", achieved=round(ach, 1),
                              unit="TFLOP/s", frac=round(ach / PEAK_BF16_TFLOPS, 4))
        else:
            ach = amount / sec / 1e9
            kernels[n] = dict(ms=round(per[n], 4), bound="hbm", achieved=round(ach, 1),
                              unit="GB/s", frac=round(ach / PEAK_HBM_GBPS, 4))
    if dx_exact_ms is not None:
        ach = fl / (dx_exact_ms * 1e-3) / 1e12
        kernels["tgemm_bwd_dx_exact"] = dict(
            ms=round(dx_exact_ms, 4), bound="mfma", achieved=round(ach, 1), unit="TFLOP/s",
            frac=round(ach / PEAK_BF16_TFLOPS, 4),
            what="two bfloat16 passes (16 bits of every scale); not part of the step")
    # in the step (after the training kernels) ...
    dec_ms = per["tgemv_pair"]
    dec_bytes = gemv_bytes(dcfg_in) + gemv_bytes(dcfg_out)
    dec_gbps = dec_bytes / (dec_ms * 1e-3) / 1e9
    # ... and tokens back to back (one launch per token; the two-launch form
    # and its per-projection events beside it)
    decode_serving = {}
    for b, (t_in_ms, t_out_ms, t_two_ms, t_tok_ms) in serve.items():
        nb = gemv_bytes(dcfg_in, b) + gemv_bytes(dcfg_out, b)
        gbps = nb / (t_tok_ms * 1e-3) / 1e9
        gbps2 = nb / (t_two_ms * 1e-3) / 1e9
        decode_serving[f"B{b}"] = {
            "us_per_token": round(t_tok_ms * 1e3, 2),
            "GBps": round(gbps, 1), "frac_hbm": round(gbps / PEAK_HBM_GBPS, 4),
            "bytes_per_token": nb,
            "two_launches": {"us_per_token": round(t_two_ms * 1e3, 2), "GBps": round(gbps2, 1),
                             "frac_hbm": round(gbps2 / PEAK_HBM_GBPS, 4),
                             "per_kernel_events": {"in_proj_us": round(t_in_ms * 1e3, 2),
                                                   "out_proj_us": round(t_out_ms * 1e3, 2)}}}
    for b in serve:
        ck = cold.get(f"decode_B{b}")
        if ck:
            decode_serving[f"B{b}"]["cold"] = ck
        ck2 = cold.get(f"decode_B{b}_two_launches")
        if ck2:
            decode_serving[f"B{b}"]["two_launches"]["cold"] = ck2
    srv = decode_serving[f"B{B}"]
    srv_cold = srv.get("cold", srv)

    fwd = kernels["tgemm_fwd"]
    dec_traffic = measured_traffic("tgemv_pair")
    out = {
        "metric": "ternary GEMM TFLOP/s (in_proj, 16k tokens) + batch-1 tgemv GB/s, % of roofline",
        "value": fwd["achieved"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded numpy; N(0,0.02) weights with 1% Laplace(0,0.2) outliers, "
                "N(0,1) activations, N(0,0.01) gradients)",
        "config": {
            "workload": "Mamba-2 1.3B in_proj QAT step (W 8512x2048 fp32, X bf16 16384x2048, "
                        "dY bf16 16384x8512, g=128) + batch-1 decode over 48 layers "
                        "(in_proj 8512x2048 + out_proj 2048x4096, 2-bit codes + fp16 scales)",
            "M": M, "N": N, "K": K, "g": g, "eps": eps, "decode_layers": L, "decode_batch": B,
        },
        "tgemv_GBps": srv_cold["GBps"],
        "tgemv_frac_hbm": srv_cold["frac_hbm"],
        "tgemv_us_per_token": srv_cold["us_per_token"],
        "tgemv_warm": {"GBps": srv["GBps"], "frac_hbm": srv["frac_hbm"],
                       "us_per_token": srv["us_per_token"]},
        "tgemv_in_step": {"GBps": round(dec_gbps, 1), "frac_hbm": round(dec_gbps / PEAK_HBM_GBPS, 4),
                          "us_per_token": round(dec_ms * 1e3, 2)},
        "decode_serving": decode_serving,
        "roofline": {"bound": "mfma", "achieved": fwd["achieved"], "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": fwd["frac"],
                     "traffic": measured_traffic("tgemm_fwd"),
                     "kernel": "tgemm_fwd (in_proj)", "algorithmic_per_launch": fl},
        "roofline_tgemv": {"bound": "hbm", "achieved": srv_cold["GBps"], "peak": PEAK_HBM_GBPS,
                           "unit": "GB/s", "frac": srv_cold["frac_hbm"],
                           "traffic": dec_traffic, "algorithmic_per_token": dec_bytes,
                           "kernel": "tgemv_pair, 48 in_proj + 48 out_proj layers in one launch, "
                                     "tokens back to back, "
                                     + ("weights rotated over >= 1.1 GiB of copies (cold)"
                                        if "cold" in srv else "one weight arena (warm)"),
                           "warm": {"achieved": srv["GBps"], "frac": srv["frac_hbm"]}},
        "kernels": kernels,
        "qat_block": qat_block,
        "decode_per_layer": per_layer,
        "decode_mixed_fp16_blocks": mixed,
        "decode_mamba2_blocks_layer_order": blocks,
        "qat_block_bf16_out": qat_block_bf16,
        "variants": variants,
        "cold_vs_warm": {k: v for k, v in cold.items() if not k.startswith("decode_")},
        "small_configs": small,
        "group_sweep": sweep,
        "zero_ratio": None,
    }
    out["zero_ratio"] = round(int(zc.item()) / (N * K), 5)

    if args.calib_copy:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # ---------------- measured ceilings (context for the fractions) ----------------
    if not args.no_ceilings:
        c = measure_ceilings()
        out["base3_packing_probe"] = c.pop("base3_packing_probe", None)
        out["measured_ceilings"] = dict(c, what=MICRO_WHAT)
        out["roofline"]["frac_of_measured"] = round(
            fwd["achieved"] / c["mfma_bf16_loop_random_TFLOPs"], 4)
        out["roofline_tgemv"]["frac_of_measured"] = round(
            srv_cold["GBps"] / c["hbm_read_stream_1GiB_GBps"], 4)
        out["roofline_tgemv"]["frac_of_measured_decode_pattern"] = round(
            srv_cold["GBps"] / c["hbm_read_stream_decode_pattern_GBps"], 4)

    # ---------------- CPU oracle baseline (bounded sample) ----------------
    # The oracle's outputs of that step are also the reference for a sampled
    # end-to-end parity check of this run's GPU outputs (the GPU codes may
    # differ from the oracle's on rounding-boundary elements only).
    if not args.no_cpu_baseline:
        gpu_out = None if args.no_parity else dict(Y=Y, dX=dX, dW=dW, codes=codes)
        out["cpu_baseline"], par, band = cpu_baseline(W_h, X_h, dY_h, g, eps, dec, gpu_out)
        if par is not None:
            out["parity_rel_fro"] = {k: float(f"{v:.3e}") for k, v in par.items()}
            out["codes_vs_oracle"] = band
            out["parity_ok"] = (max(par.values()) <= 2e-3 and band["mismatch_off_band"] == 0)
            if not out["parity_ok"]:
                log(f"PARITY FAILURE: {par}")

    print(json.dumps(out), flush=True)


ROTATE_BYTES = 1.1 * 2 ** 30   # cold figures rotate over this much distinct input


def cold_figures(ops, dec, W, dW, codes, scales, g, eps, reps, decode_token):
    """HBM-bound calls with their inputs rotated over >= 1.1 GiB of distinct
    copies, so no call finds its input in the 256 MB memory-side cache or the
    L2 (the "cold" figures; the warm ones repeat one input):
      * the decode token (48 in_proj + 48 out_proj matrices), B = 1 and 4,
        cycling over copies of both arenas, tokens back to back under one
        event pair, in one launch per token (tm_tgemv_pair) and in two;
      * ternarize_pack, the threshold-multiplier and given-threshold
        ternarizers, cycling over copies of the in_proj W;
      * the group-magnitude gradient, cycling over copies of dW.
    Returns per-call microseconds and GB/s."""
    import torch
    dev = W.device
    res = {}
    # decode arenas
    tok_bytes = sum(d["codes"].numel() + 2 * d["s16"].numel() for d in dec.values())
    nsets = int(np.ceil(ROTATE_BYTES / tok_bytes))
    sets = [{k: (d["codes"], d["s16"]) for k, d in dec.items()}]
    for _ in range(nsets - 1):
        sets.append({k: (d["codes"].clone(), d["s16"].clone()) for k, d in dec.items()})
    for batch, (xk, yk) in ((1, ("x", "y")), (4, ("x4", "y4"))):
        if dec["in"][xk].shape[1] != batch:
            continue

        def token_two(t):
            for kind in ("in", "out"):
                d = dec[kind]
                c, sc = sets[t % nsets][kind]
                ops.tgemv(d[xk], c, sc, d["cfg"].g, y=d[yk])

        def token_one(t):
            st = sets[t % nsets]
            decode_token(xk, yk, (st["in"][0], st["in"][1], st["out"][0], st["out"][1]))
        nb = sum(L * (c.N * c.K / 4 + 2 * c.N * c.K / c.g + 2 * batch * c.K + 4 * batch * c.N)
                 for c, L in ((dec[k]["cfg"], dec[k]["codes"].shape[0]) for k in ("in", "out")))
        for key, token in ((f"decode_B{batch}", token_one),
                           (f"decode_B{batch}_two_launches", token_two)):
            for t in range(2 * nsets):
                token(t)
            torch.cuda.synchronize()
            ntok = max(reps, 5) * nsets
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(2_000_000)
            e0.record()
            for t in range(ntok):
                token(t)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / ntok
            res[key] = {"us_per_token": round(us, 2), "GBps": round(nb / (us * 1e-6) / 1e9, 1),
                        "frac_hbm": round(nb / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
                        "copies": nsets}
    del sets
    # W and dW copies
    N, K = W.shape
    ncp = int(np.ceil(ROTATE_BYTES / (N * K * 4)))
    Ws = [W] + [W.clone() for _ in range(ncp - 1)]
    dWs = [dW] + [dW.clone() for _ in range(ncp - 1)]
    mult = torch.ones((N,), dtype=torch.float32, device=dev)
    mult[:4096] = 0.8
    c2, s2 = torch.empty_like(codes), torch.empty_like(scales)
    s16 = torch.empty(scales.shape, dtype=torch.float16, device=dev)
    zc = torch.empty((1,), dtype=torch.int64, device=dev)
    ds = torch.empty_like(scales)
    calls = {
        "ternarize_pack": (lambda i: ops.ternarize_pack(Ws[i], g, eps, codes=c2, scales=s2,
                                                        scales_f16=s16, zero_count=zc),
                           N * K * (4 + 0.25 + 4 / g + 2 / g)),
        "ternarize_pack_thresh": (lambda i: ops.ternarize_pack(Ws[i], g, eps, codes=c2, scales=s2,
                                                               zero_count=zc, want_f16=False,
                                                               row_mult=mult),
                                  N * K * (4 + 0.25) + N * K / g * 4 + N * 4),
        "ternarize_codes": (lambda i: ops.ternarize_codes(Ws[i], scales, g, eps, codes=c2,
                                                          zero_count=zc),
                            N * K * (4 + 0.25) + N * K / g * 4),
        "group_code_dot": (lambda i: ops.group_code_dot(codes, dWs[i], g, out=ds),
                           N * K * (4 + 0.25) + N * K / g * 4),
    }
    for name, (fn, nbytes) in calls.items():
        out = {}
        for mode, pick in (("cold", lambda i: i % ncp), ("warm", lambda i: 0)):
            for i in range(ncp):
                fn(pick(i))
            torch.cuda.synchronize()
            n = max(reps, 5) * ncp
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(2_000_000)
            e0.record()
            for i in range(n):
                fn(pick(i))
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / n
            out[mode] = {"us": round(us, 2), "GBps": round(nbytes / (us * 1e-6) / 1e9, 1),
                         "frac_hbm": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)}
        out["copies"] = ncp
        res[name] = out
    del Ws, dWs
    return res


def variants_step(args, ops, W, scales, codes, dW, g, eps):
    """The entry points of the scale variants, timed on the in_proj shapes:
    ternarize with 0.8 x absmean thresholds on rows 0-4095 (the appendix's
    gate setting), codes against given thresholds (a learned scale; the
    absmean is passed), the group-magnitude gradient sum q * dW over the
    step's dW, and the learnable-scale gradient with the rounding
    straight-through (the absmean as the learned scale).  All are single HBM
    passes."""
    import torch
    N, K = W.shape
    dev = W.device
    mult = torch.ones((N,), dtype=torch.float32, device=dev)
    mult[:4096] = 0.8
    c2 = torch.empty_like(codes)
    s2 = torch.empty_like(scales)
    zc = torch.empty((1,), dtype=torch.int64, device=dev)
    ds = torch.empty_like(scales)
    dWm = torch.empty_like(dW)
    calls = {
        "ternarize_pack_thresh": (
            lambda: ops.ternarize_pack(W, g, eps, codes=c2, scales=s2, zero_count=zc,
                                       want_f16=False, row_mult=mult),
            N * K * (4 + 0.25) + N * K / g * 4 + N * 4),
        "ternarize_codes": (
            lambda: ops.ternarize_codes(W, scales, g, eps, codes=c2, zero_count=zc),
            N * K * (4 + 0.25) + N * K / g * 4),
        "group_code_dot": (
            lambda: ops.group_code_dot(codes, dW, g, out=ds),
            N * K * (4 + 0.25) + N * K / g * 4),
        # learnable scale, rounding straight-through: reads W, the codes, s and
        # dWhat, writes ds and the clip-masked dW (here not in place, so that
        # the step's dW stays as it is)
        "scale_ste_grad": (
            lambda: ops.scale_ste_grad(W, codes, scales, dW, g, eps, ds=ds, dW=dWm),
            N * K * (4 + 4 + 0.25 + 4) + N * K / g * 8),
    }
    steps = max(args.steps, 10)
    res = {}
    for name, (fn, nbytes) in calls.items():
        for _ in range(3):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        torch.cuda._sleep(1_000_000)
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
        gbps = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"ms": round(ms, 4), "GBps": round(gbps, 1),
                     "frac_hbm": round(gbps / PEAK_HBM_GBPS, 4), "bytes": nbytes}
    # zero ratios of the two row ranges, counted by the kernel on each range
    zg = ops.ternarize_pack(W[:4096], g, eps, want_f16=False, row_mult=mult[:4096])[3]
    zr = ops.ternarize_pack(W[4096:], g, eps, want_f16=False)[3]
    res["zero_ratio_gate_rows_0.8"] = round(int(zg.item()) / (4096 * K), 5)
    res["zero_ratio_other_rows"] = round(int(zr.item()) / ((N - 4096) * K), 5)
    return res


def qat_block_step(args, dev, X_in, synth, out_dtype=None):
    """One QAT step of a Mamba-2 1.3B block's two ternary projections through
    the autograd layer (forward, straight-through backward, 16384 tokens):
    in_proj 2048 -> 8512 on the block input, out_proj 4096 -> 2048 on a
    synthetic SSM output.  The upstream gradients are given (in the layers'
    output dtype); the time covers the library calls plus, with float32
    outputs, the layer's gradient casts to bfloat16."""
    import torch
    from paper_2606_18114_amd.qat import TernaryLinear, flops_per_step

    torch.manual_seed(7)
    M = X_in.shape[0]
    od = out_dtype or torch.float32
    lin = TernaryLinear(synth.D_MODEL, synth.IN_PROJ_N, device=dev, out_dtype=od)
    lout = TernaryLinear(synth.D_INNER, synth.D_MODEL, device=dev, out_dtype=od)
    z = torch.randn((M, synth.D_INNER), device=dev).to(torch.bfloat16).requires_grad_(True)
    x = X_in.detach().requires_grad_(True)  # gradients flow on to the layers below
    g_in = (torch.randn((M, synth.IN_PROJ_N), device=dev) * synth.DY_STD).to(od)
    g_out = (torch.randn((M, synth.D_MODEL), device=dev) * synth.DY_STD).to(od)

    def step():
        lin.weight.grad = lout.weight.grad = x.grad = z.grad = None
        y1 = lin(x)
        y2 = lout(z)
        torch.autograd.backward([y1, y2], [g_in, g_out])

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    reps = max(args.steps // 2, 5)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(2_000_000)
    e0.record()
    for _ in range(reps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    fl = flops_per_step(M, lin) + flops_per_step(M, lout)
    return {"ms_per_step": round(ms, 4), "TFLOPs": round(fl / (ms * 1e-3) / 1e12, 1),
            "frac_mfma": round(fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "tokens": M, "zero_ratio_in_proj": round(lin.zero_ratio(), 5),
            "what": "TernaryLinear in_proj 2048->8512 + out_proj 4096->2048, forward + "
                    "straight-through backward (dX and dW), 16384 tokens, g=128, "
                    f"{str(od).replace('torch.', '')} outputs"}


def cpu_baseline(W_h, X_h, dY_h, g, eps, dec, gpu_out=None):
    """The oracle as it stands, timed on the host over one whole step of the
    same workload: the in_proj QAT step at full size (ternarize, float64
    forward, dX and dW GEMMs) and one batch-1 decode token over all 96 packed
    matrices (unpack + float64 GEMV per matrix; the packed arenas are copied
    to the host before timing).  `value` is the oracle's forward-GEMM TFLOP/s,
    the unit of the headline.

    Returns (baseline, parity, codes): after the timing, 64 sampled rows of
    the GPU's Y and dX, 64 rows of dW and the last in_proj decode output are
    compared with the oracle's (relative Frobenius errors), and the GPU's
    in_proj codes with the oracle's over the whole matrix: elements within
    1e-6 of the rounding boundary, and mismatches on and off that band
    (unless gpu_out is None)."""
    import torch
    from oracle import ternary as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    N, K = W_h.shape
    M = X_h.shape[0]
    host = {kind: (dec[kind]["cfg"], dec[kind]["codes"].cpu().numpy(), dec[kind]["s16"].cpu().numpy(),
                   dec[kind]["x"].cpu().view(torch.int16).numpy().view(np.uint16))
            for kind in ("in", "out")}
    t = {}
    t0 = time.perf_counter()
    s64, s32, q, z_orc = O.ternarize(W_h, g, eps)
    t["ternarize"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    Y_ref = O.gemm_fwd(X_h, q, s32, g)
    t["fwd"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    dX_ref = O.gemm_bwd_dx(dY_h, q, s32, g)
    t["dx"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    dW_ref = O.gemm_bwd_dw(dY_h, X_h)
    t["dw"] = time.perf_counter() - t0
    gemv_bytes, nmat, t0 = 0.0, 0, time.perf_counter()
    for kind in ("in", "out"):
        c, codes, s16, x = host[kind]
        for layer in range(codes.shape[0]):
            y_ref = O.gemv(x[layer], O.unpack(codes[layer], c.K), s16[layer], c.g)
            if kind == "in":
                y_in_last = y_ref
            gemv_bytes += c.N * c.K / 4 + 2 * c.N * c.K / c.g
            nmat += 1
    t["gemv"] = time.perf_counter() - t0
    par = codes_cmp = None
    if gpu_out is not None:
        dev = gpu_out["Y"].device
        rows = np.sort(np.random.default_rng(123).choice(M, 64, replace=False))
        cols = np.sort(np.random.default_rng(124).choice(N, 64, replace=False))
        ri, ci = torch.from_numpy(rows).to(dev), torch.from_numpy(cols).to(dev)
        par = {
            "fwd": O.rel_fro_error(gpu_out["Y"][ri].cpu().numpy(), Y_ref[rows]),
            "dx": O.rel_fro_error(gpu_out["dX"][ri].cpu().numpy(), dX_ref[rows]),
            "dw": O.rel_fro_error(gpu_out["dW"][ci].cpu().numpy(), dW_ref[cols]),
            "tgemv": O.rel_fro_error(dec["in"]["y"][-1].cpu().numpy(), y_in_last),
        }
        band = O.boundary_mask(W_h, s64, g, eps)
        diff = O.unpack(gpu_out["codes"].cpu().numpy(), K) != q
        codes_cmp = {"elements": int(q.size), "boundary_elements": int(band.sum()),
                     "mismatch_on_band": int((diff & band).sum()),
                     "mismatch_off_band": int((diff & ~band).sum()),
                     "zero_count_oracle": int(z_orc)}
    del Y_ref, dX_ref, dW_ref
    fl = 2.0 * M * N * K
    total = sum(t.values())
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f
                              if ln.startswith("model name")), None)
    except OSError:
        pass
    base = {"value": round(fl / t["fwd"] / 1e12, 4), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model,
            "cores_available": len(os.sched_getaffinity(0)),
            "sample": (f"one whole step on the host ({total:.1f}s): in_proj QAT step, ternarize "
                       f"{t['ternarize']:.2f}s ({N * K * 4 / t['ternarize'] / 1e9:.2f} GB/s of W), "
                       f"float64 fwd {t['fwd']:.2f}s, dX {t['dx']:.2f}s, dW {t['dw']:.2f}s "
                       f"({fl / 1e9:.0f} GFLOP each); batch-1 decode token over {nmat} matrices "
                       f"{t['gemv']:.2f}s ({gemv_bytes / t['gemv'] / 1e9:.3f} GB/s of packed weights)")}
    return base, par, codes_cmp


def decode_mamba2_blocks(dev, tokens, keep=(), batch=1, fused=True, stack=False):
    """Decode as a model runs it: 48 whole Mamba-2 blocks in layer order, each
    pre-norm -> in_proj -> mixer step (convolution, FP16 SSM state update,
    gated RMSNorm) -> out_proj, then the final norm.  Fused: 3 launches per
    layer (the norms inside the projections' staging, the residual add in
    out_proj's store); unfused: 5; stack: the whole token in one
    launch with grid barriers between the phases.  Timed eagerly (one Python
    call per launch) and as one captured HIP graph per token (where the
    launches can be captured); states persist from token to token."""
    import torch
    from paper_2606_18114_amd import synth
    from paper_2606_18114_amd.stack import Mamba2Decoder

    cfg = {"in": synth.DECODE_IN, "out": synth.DECODE_OUT}
    L, H = synth.N_LAYERS, synth.D_INNER // synth.HEADDIM
    rng = np.random.default_rng(5000)
    mix = [synth.mixer_params(rng, H) for _ in range(L)]
    dec = Mamba2Decoder(
        lambda k, l: torch.from_numpy(synth.layer_weight(cfg[k], synth.decode_seed(f"{k}_w", l))
                                      ).to(dev),
        lambda l: mix[l], lambda l: torch.ones(synth.D_MODEL), L, synth.D_MODEL, H,
        keep=keep, g=128, batch=batch, device=dev, fused=fused, stack=stack)
    for l in range(L):
        conv, ssm = synth.mixer_states(rng, batch, H)
        dec.set_states(l, torch.from_numpy(conv).to(dev), torch.from_numpy(ssm).to(dev))
    dec.emb.copy_(torch.from_numpy(rng.standard_normal((batch, synth.D_MODEL))
                                   .astype(np.float32)).to(dev))

    def timed(fn, n):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(2_000_000)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    n = max(tokens, 10)
    us_eager = timed(dec.token, n)
    us_graph = None
    try:
        dec.capture()
        us_graph = timed(dec.replay, n)
    except RuntimeError as e:  # a launch that cannot be captured
        log(f"decode blocks (stack={dec.stack}): no graph capture ({str(e)[:120]})")
    nb = dec.bytes_per_token()
    best = us_graph if us_graph is not None else us_eager
    res = {"layers": L, "kept_fp16_layers": sorted(dec.keep), "batch": batch,
           "fused": dec.fused, "one_launch": dec.stack,
           "launches_per_token": dec.launches_per_token(), "bytes_per_token": nb,
           "us_per_token_eager": round(us_eager, 2),
           "us_per_token_graph": None if us_graph is None else round(us_graph, 2),
           "GBps_best": round(nb / (best * 1e-6) / 1e9, 1),
           "frac_hbm_best": round(nb / (best * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
           "tokens_per_s_best": round(batch / (best * 1e-6), 1),
           "what": "48 Mamba-2 1.3B blocks in layer order (pre-norm, in_proj 8512x2048, "
                   "conv + FP16 SSM state + gated RMSNorm, out_proj 2048x4096) + final norm, "
                   "one token per batch row, states carried over"}
    del dec
    torch.cuda.empty_cache()
    return res


def decode_mixed_stack(dev, tokens, batch=1):
    """Layer-selective quantization (Sec. 7, Table 10): the 48-layer decode
    token with the first two and last two blocks kept in FP16 (2 bytes per
    weight, tm_dgemv) and the other 44 ternary: three launches per token (the
    ternary arenas of both projection kinds in one, tm_tgemv_pair, then each
    kind's FP16 arena).  Warm (one set of arenas) and cold (tokens cycling
    over copies, >= 1.1 GiB)."""
    import torch
    from paper_2606_18114_amd import synth
    from paper_2606_18114_amd.stack import DecodeStack, keep_first_last

    cfg = {"in": synth.DECODE_IN, "out": synth.DECODE_OUT}
    L = synth.N_LAYERS
    keep = keep_first_last(L, 2)
    st = DecodeStack(
        lambda k, l: torch.from_numpy(synth.layer_weight(cfg[k], synth.decode_seed(f"{k}_w", l))
                                      ).to(dev),
        L, {k: (c.N, c.K) for k, c in cfg.items()}, keep=keep, g=128, eps=1e-5, batch=batch,
        device=dev)
    for k, c in cfg.items():
        xs = np.stack([synth.layer_acts(batch, c.K, synth.decode_seed(f"{k}_x", l))
                       for l in range(L)])
        st.set_inputs(k, torch.from_numpy(xs.view(np.int16)).to(dev).view(torch.bfloat16))
    nb = st.bytes_per_token()
    copies = [None] + [st.arena_copy() for _ in range(int(np.ceil(ROTATE_BYTES / nb)) - 1)]
    res = {"kept_layers": keep, "bytes_per_token": nb, "batch": batch,
           "launches_per_token": 3}
    for mode in ("warm", "cold"):
        pick = (lambda t: None) if mode == "warm" else (lambda t: copies[t % len(copies)])
        for t in range(2 * len(copies)):
            st.token(arenas=pick(t))
        torch.cuda.synchronize()
        n = max(tokens, 5) * len(copies)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(2_000_000)
        e0.record()
        for t in range(n):
            st.token(arenas=pick(t))
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / n
        res[mode] = {"us_per_token": round(us, 2), "GBps": round(nb / (us * 1e-6) / 1e9, 1),
                     "frac_hbm": round(nb / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)}
    res["copies_cold"] = len(copies)
    res["what"] = ("48 layers (in_proj 8512x2048 + out_proj 2048x4096), layers 0, 1, 46, 47 "
                   "in float16, the rest 2-bit codes + fp16 scales, batch 1, all layers of a "
                   "kind per launch")
    del copies, st
    return res


def decode_per_layer(ops, dec, L, tokens):
    """Decode as a model runs it, layer by layer: in_proj of layer l, then its
    out_proj, each launch carrying one matrix (4.4 MB or 2.1 MB of codes).
    The SSM between the two projections is outside this library, so each GEMV
    reads its input from the arena.  Timed with Python launches and as one
    captured HIP graph of the 96 launches per token; the graph's outputs are
    checked bit for bit against the eager ones."""
    import torch

    def token():
        for layer in range(L):
            for kind in ("in", "out"):
                d = dec[kind]
                sl = slice(layer, layer + 1)
                ops.tgemv(d["x"][sl], d["codes"][sl], d["s16"][sl], d["cfg"].g, y=d["y"][sl])

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        torch.cuda._sleep(2_000_000)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(tokens):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / tokens

    eager_us = timed(token)
    ref = {k: dec[k]["y"].clone() for k in ("in", "out")}
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        token()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        token()
    for k in ("in", "out"):
        dec[k]["y"].fill_(float("nan"))
    graph_us = timed(graph.replay)
    same = all(torch.equal(dec[k]["y"], ref[k]) for k in ("in", "out"))
    nbytes = 0
    for k in ("in", "out"):
        c = dec[k]["cfg"]
        B = dec[k]["x"].shape[1]
        nbytes += L * (c.N * c.K / 4 + 2 * c.N * c.K / c.g + 2 * B * c.K + 4 * B * c.N)
    del graph
    return {"launches_per_token": 2 * L,
            "us_per_token_eager": round(eager_us, 2),
            "us_per_token_graph": round(graph_us, 2),
            "GBps_graph": round(nbytes / (graph_us * 1e-6) / 1e9, 1),
            "graph_outputs_equal_eager": bool(same),
            "what": "48 x (in_proj 8512x2048, then out_proj 2048x4096), one tgemv launch per "
                    "matrix in layer order, batch " + str(dec["in"]["x"].shape[1]) +
                    "; the SSM between the projections is not part of this library"}


def micro(args):
    """`--micro`: the measured ceilings alone, as one JSON line."""
    print(json.dumps({"micro": measure_ceilings(), "peaks": {"bf16_TFLOPs": PEAK_BF16_TFLOPS,
                                                             "hbm_GBps": PEAK_HBM_GBPS},
                      "what": MICRO_WHAT}), flush=True)


MICRO_WHAT = ("MFMA loop: 4 waves per SIMD, independent bf16 MFMA chains per wave (4 of "
              "32x32x16 or 8 of 16x16x32) on operands loaded once; the ceiling is the faster "
              "shape; read stream: 1 GiB in contiguous 16 KiB chunks per wave, "
              "16 waves per CU; medians of 5 runs; decode pattern: the same read stream "
              "over the decode step's codes and scales (48 in_proj, then 48 out_proj "
              "matrices, two launches per token), 20 tokens back to back")


def measure_ceilings():
    """Measured denominators: what this GPU sustains on a plain MFMA loop and a
    plain read stream (libtm_micro.so), and, for context, a device copy and
    hipBLASLt (torch.mm) on the in_proj forward shape."""
    import ctypes
    import torch
    from paper_2606_18114_amd import build as B

    if not os.path.exists(B.MICRO_OUT):
        B.build()
    lib = ctypes.CDLL(B.MICRO_OUT)
    lib.tmm_grid_threads.restype = ctypes.c_int
    lib.tmm_mfma_loop.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                  ctypes.c_void_p]
    lib.tmm_read_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p]
    lib.tmm_decode_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                      ctypes.c_void_p, ctypes.c_void_p]
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    st = torch.cuda.current_stream().cuda_stream
    threads = lib.tmm_grid_threads()

    def timed(fn, reps=5, warm=2):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return float(np.median(ts))

    def check(rc):
        if rc != 0:
            raise RuntimeError(f"micro kernel launch failed: {rc}")

    out = torch.empty(threads, dtype=torch.float32, device=dev)
    iters = 20000
    fl = 2.0 * 32 * 32 * 16 * 4 * iters * (threads // 64)
    res = {}
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    for label, opnd in (("random", torch.randn(1024, generator=gen, device=dev)),
                        ("zero", torch.zeros(1024, device=dev))):
        o16 = opnd.to(torch.bfloat16)
        for shape in (32, 16):
            sec = timed(lambda: check(lib.tmm_mfma_loop(o16.data_ptr(), iters, shape,
                                                        out.data_ptr(), st)))
            res[f"mfma_bf16_{shape}x{shape}_loop_{label}_TFLOPs"] = round(fl / sec / 1e12, 1)
    res["mfma_bf16_loop_random_TFLOPs"] = max(res["mfma_bf16_32x32_loop_random_TFLOPs"],
                                              res["mfma_bf16_16x16_loop_random_TFLOPs"])
    buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    buf.random_(0, 256, generator=gen)
    words = torch.empty(threads, dtype=torch.int32, device=dev)
    sec = timed(lambda: check(lib.tmm_read_stream(buf.data_ptr(), buf.numel(), words.data_ptr(), st)))
    res["hbm_read_stream_1GiB_GBps"] = round(buf.numel() / sec / 1e9, 1)
    dst = torch.empty_like(buf)
    sec = timed(lambda: dst.copy_(buf))
    res["device_copy_1GiB_GBps"] = round(2 * buf.numel() / sec / 1e9, 1)
    del buf, dst
    # the same read stream in the decode step's launch pattern: the packed
    # codes and half-precision scales of the 48 in_proj and of the 48
    # out_proj matrices in two buffers, read one after the other as tokens
    # back to back, one event pair around the run (as the serving timing)
    from paper_2606_18114_amd import synth
    sizes = []
    for c in (synth.DECODE_IN, synth.DECODE_OUT):
        nb = synth.N_LAYERS * (c.N * c.K // 4 + 2 * c.N * c.K // c.g)
        sizes.append(nb - nb % 16384)
    pat = [torch.randint(0, 256, (nb,), dtype=torch.uint8, device=dev, generator=gen)
           for nb in sizes]

    def token():
        for b in pat:
            check(lib.tmm_read_stream(b.data_ptr(), b.numel(), words.data_ptr(), st))
    tokens = 20
    sec = timed(lambda: [token() for _ in range(tokens)], reps=3, warm=1)
    res["hbm_read_stream_decode_pattern_GBps"] = round(sum(sizes) * tokens / sec / 1e9, 1)
    del pat
    # base-3 packing against the 2-bit format: the 48 in_proj matrices' codes
    # streamed and decoded into the matrix-core operand nibbles (five codes
    # per byte from a table, or the 2-bit shift-and-mask), in copies rotated
    # over > 1 GiB so that both stream from HBM
    c = synth.DECODE_IN
    codes = synth.N_LAYERS * c.N * c.K
    b3 = {}
    for fmt, per_byte in ((2, 4), (3, 5)):
        nb = -(-codes // per_byte)
        nb += (-nb) % 16384
        copies = [torch.randint(0, 243 if fmt == 3 else 256, (nb,), dtype=torch.uint8,
                                device=dev, generator=gen) for _ in range(-(-(1 << 30) // nb) + 1)]

        def run(f):
            for b in copies:
                check(lib.tmm_decode_stream(b.data_ptr(), b.numel(), f, words.data_ptr(), st))

        def plain():
            for b in copies:
                check(lib.tmm_read_stream(b.data_ptr(), b.numel(), words.data_ptr(), st))
        sec = timed(lambda: run(fmt), reps=3, warm=1) / len(copies)
        sec_read = timed(plain, reps=3, warm=1) / len(copies)
        b3[f"format{fmt}"] = {"bytes": nb, "bits_per_code": round(8.0 * nb / codes, 3),
                              "decode_us": round(sec * 1e6, 2), "read_only_us": round(sec_read * 1e6, 2),
                              "Gcodes_per_s": round(codes / sec / 1e9, 1)}
        del copies
    b3["base3_vs_2bit_time"] = round(b3["format3"]["decode_us"] / b3["format2"]["decode_us"], 3)
    b3["what"] = ("codes of the 48 in_proj layers (8512 x 2048 each) streamed from HBM and "
                  "decoded to the FP4 operand nibbles: format 2 = the 2-bit codes, format 3 = "
                  "base-3 packing (5 codes per byte, 1.6 bits); decode_us per pass, read_only_us "
                  "the same bytes without the decode")
    res["base3_packing_probe"] = b3
    M, N, K = 16384, 8512, 2048
    X = torch.randn((M, K), generator=gen, device=dev).to(torch.bfloat16)
    Wt = (torch.randn((N, K), generator=gen, device=dev) * 0.02).to(torch.bfloat16).t().contiguous()
    sec = timed(lambda: torch.mm(X, Wt))
    res["torch_mm_bf16_in_proj_TFLOPs"] = round(2.0 * M * N * K / sec / 1e12, 1)
    del X, Wt
    torch.cuda.empty_cache()
    return res


def group_sweep(ops, dev, reps):
    """Group-size workload: the in_proj weights (8512 x 2048, with outliers)
    ternarized and applied to 2048 x 2048 bf16 activations for g = 32 .. 512.
    Per g: zero ratio (the kernel's count) and NRMSE of the quantizer,
    ternarize GB/s and forward TFLOP/s.  (Parity at every g is the tests'
    job, at this full shape included.)"""
    import torch
    from paper_2606_18114_amd import synth

    N, K, M = synth.IN_PROJ_N, synth.D_MODEL, 2048
    W_h = synth.layer_weight(synth.C3, synth.SEED_W)
    X_h = synth.layer_acts(M, K, synth.SEED_X)
    W = torch.from_numpy(W_h).to(dev)
    X = torch.from_numpy(X_h.view(np.int16)).to(dev).view(torch.bfloat16)
    Y = torch.empty((M, N), dtype=torch.float32, device=dev)
    eye = torch.eye(K, dtype=torch.bfloat16, device=dev)
    w_norm = float(torch.linalg.vector_norm(W.double()))
    rows = []
    for g in synth.C5_GROUPS:
        codes = torch.empty((N, K // 4), dtype=torch.uint8, device=dev)
        scales = torch.empty((N, K // g), dtype=torch.float32, device=dev)
        zc = torch.empty((1,), dtype=torch.int64, device=dev)
        for _ in range(3):
            ops.ternarize_pack(W, g, 1e-5, codes=codes, scales=scales, zero_count=zc)
            ops.tgemm_fwd(X, codes, scales, g, Y=Y)
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
        torch.cuda._sleep(2_000_000)
        for e in ev:
            e[0].record()
            ops.ternarize_pack(W, g, 1e-5, codes=codes, scales=scales, zero_count=zc)
            e[1].record()
            ops.tgemm_fwd(X, codes, scales, g, Y=Y)
            e[2].record()
        torch.cuda.synchronize()
        t_tern = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        t_fwd = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
        # the dequantized weights q * s through the forward kernel itself: with
        # X = I every output is a single exact product
        What_t = ops.tgemm_fwd(eye, codes, scales, g)
        nrmse = float(torch.linalg.vector_norm((W - What_t.t()).double()) / w_norm)
        z = int(zc.item())
        tern_bytes = N * K * (4 + 0.25 + 4 / g)
        fl = 2.0 * M * N * K
        rows.append({
            "g": g, "zero_ratio": round(z / (N * K), 5), "nrmse": round(nrmse, 5),
            "ternarize_ms": round(t_tern, 4),
            "ternarize_GBps": round(tern_bytes / t_tern / 1e6, 1),
            "fwd_ms": round(t_fwd, 4), "fwd_TFLOPs": round(fl / t_fwd / 1e9, 1),
            "fwd_frac_mfma": round(fl / t_fwd / 1e9 / PEAK_BF16_TFLOPS, 4)})
    return {"workload": f"group sweep: in_proj W {N}x{K} (1% Laplace outliers), "
                        f"X bf16 {M}x{K}, warm", "rows": rows}


def small_configs(ops, dev, reps):
    """The single linear layer (W 256 x 512, X 16 x 512, g = 128) as a latency:
    ternarize + forward per call, both launched back to back and timed with
    one event pair around many calls; and the out_proj forward (W 2048 x 4096,
    X 4096 x 4096) as a throughput."""
    import torch
    from paper_2606_18114_amd import synth

    def bf16(bits):
        return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)

    res = {}
    # single linear: latency of one ternarize + forward
    c1 = synth.C1
    W_h, X_h = synth.single_linear_inputs(c1)
    W, X = torch.from_numpy(W_h).to(dev), bf16(X_h)
    codes = torch.empty((c1.N, c1.K // 4), dtype=torch.uint8, device=dev)
    scales = torch.empty((c1.N, c1.K // c1.g), dtype=torch.float32, device=dev)
    zc = torch.empty((1,), dtype=torch.int64, device=dev)
    Y = torch.empty((c1.M, c1.N), dtype=torch.float32, device=dev)

    def c1_call():
        ops.ternarize_pack(W, c1.g, c1.eps, codes=codes, scales=scales, zero_count=zc,
                           want_f16=False)
        ops.tgemm_fwd(X, codes, scales, c1.g, Y=Y)

    def per_call_us(fn, n):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(2_000_000)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / n

    n = max(reps, 50) * 4
    t_c1 = per_call_us(c1_call, n)
    t_fwd = per_call_us(lambda: ops.tgemm_fwd(X, codes, scales, c1.g, Y=Y), n)
    t_tern = per_call_us(lambda: ops.ternarize_pack(W, c1.g, c1.eps, codes=codes, scales=scales,
                                                    zero_count=zc, want_f16=False), n)
    # a captured graph of the two calls: the launch cost a serving loop pays
    gr = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        c1_call()
        with torch.cuda.graph(gr, stream=side):
            c1_call()
    torch.cuda.current_stream().wait_stream(side)
    t_graph = per_call_us(gr.replay, n)
    fl1 = 2.0 * c1.M * c1.N * c1.K
    res["single_linear"] = {
        "workload": "single ternary linear: W fp32 256x512, X bf16 16x512, g=128",
        "us_ternarize_plus_fwd": round(t_c1, 2), "us_fwd": round(t_fwd, 2),
        "us_ternarize": round(t_tern, 2), "us_graph_replay": round(t_graph, 2),
        "fwd_GFLOPs": round(fl1 / (t_fwd * 1e-6) / 1e9, 2)}
    # out_proj: forward throughput
    c2 = synth.C2
    W2 = torch.from_numpy(synth.layer_weight(c2, synth.SEED_W)).to(dev)
    X2 = bf16(synth.layer_acts(c2.M, c2.K, synth.SEED_X))
    codes2 = torch.empty((c2.N, c2.K // 4), dtype=torch.uint8, device=dev)
    scales2 = torch.empty((c2.N, c2.K // c2.g), dtype=torch.float32, device=dev)
    Y2 = torch.empty((c2.M, c2.N), dtype=torch.float32, device=dev)
    tern2 = lambda: ops.ternarize_pack(W2, c2.g, c2.eps, codes=codes2, scales=scales2,
                                       zero_count=zc, want_f16=False)
    tern2()
    t_fwd2 = per_call_us(lambda: ops.tgemm_fwd(X2, codes2, scales2, c2.g, Y=Y2), max(reps, 20))
    t_tern2 = per_call_us(tern2, max(reps, 20))
    fl2 = 2.0 * c2.M * c2.N * c2.K
    tb2 = c2.N * c2.K * (4 + 0.25 + 4 / c2.g)
    res["out_proj"] = {
        "workload": "out_proj: W fp32 2048x4096, X bf16 4096x4096, g=128, fp32 out",
        "fwd_us": round(t_fwd2, 2), "fwd_TFLOPs": round(fl2 / (t_fwd2 * 1e-6) / 1e12, 1),
        "fwd_frac_mfma": round(fl2 / (t_fwd2 * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "ternarize_us": round(t_tern2, 2),
        "ternarize_GBps_warm": round(tb2 / (t_tern2 * 1e-6) / 1e9, 1)}
    return res


def sweep_g(args):
    """--sweep-g: the group-size workload alone, one JSON line per g."""
    import torch
    from paper_2606_18114_amd import ops

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sw = group_sweep(ops, dev, max(args.steps, 5))
    for row in sw["rows"]:
        print(json.dumps(dict(workload=sw["workload"], **row)), flush=True)


if __name__ == "__main__":
    main()
