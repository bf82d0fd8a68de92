"""Zero-ratio probe of the scale parameterizations on a synthetic objective.

Sec. 4 of the paper reports that a learnable per-group scale drives the zero
ratio of a QAT-from-pretrained Mamba-2 towards 90% (zero-ratio collapse),
while the recomputed absmean settles near 26%, and the appendix reports that
a decoupled learned magnitude barely moves.  The trained model and its data
are not available here, so this probe runs the same three layers on a
synthetic stand-in: a student TernaryLinear initialised from a "pretrained"
float teacher W_t (N(0, 0.02), 1% Laplace outliers) is trained by AdamW to
match the teacher's outputs on N(0, 1) bfloat16 inputs (distillation with a
mean-squared loss), and the zero ratio, the relative output error and the
mean scale are logged along the way.  It shows how each parameterization
responds to the same gradient signal; it is not a reproduction of the
paper's numbers.

    python -m paper_2606_18114_amd.collapse_probe [--steps 300] [--lr 1e-3]

Prints one JSON line per mode with the trajectory.  Needs a GPU.
"""

from __future__ import annotations

import argparse
import json

import numpy as np
import torch

from . import synth
from .qat import TernaryLinear


def run(mode: str, steps: int, lr: float, wd: float, N: int, K: int, tokens: int,
        seed: int, log_every: int):
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(seed)
    Wt = torch.from_numpy(synth.weights(rng, N, K, outliers=True)).to(dev)
    layer = TernaryLinear.from_weight(Wt.clone(), g=128, scale_mode=mode)
    opt = torch.optim.AdamW(layer.parameters(), lr=lr, weight_decay=wd)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    traj = []
    for step in range(steps + 1):
        x = torch.randn((tokens, K), generator=gen, device=dev).to(torch.bfloat16)
        with torch.no_grad():
            target = x.float() @ Wt.t()
        y = layer(x)
        loss = ((y - target) ** 2).mean()
        if step % log_every == 0 or step == steps:
            rel = float((loss.detach() / (target ** 2).mean()).sqrt())
            entry = {"step": step, "zero_ratio": round(layer.zero_ratio(), 5),
                     "rel_output_error": round(rel, 5)}
            if layer.scale is not None:
                entry["mean_scale"] = float(layer.scale.detach().mean())
            traj.append(entry)
        if step == steps:
            break
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
    return traj


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--lr", type=float, default=1e-3)
    ap.add_argument("--wd", type=float, default=0.0)
    ap.add_argument("--n", type=int, default=2048)
    ap.add_argument("--k", type=int, default=2048)
    ap.add_argument("--tokens", type=int, default=4096)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--log-every", type=int, default=25)
    ap.add_argument("--modes", default="absmean,decoupled,learnable")
    a = ap.parse_args()
    assert torch.cuda.is_available(), "the probe runs the library's kernels: it needs a GPU"
    for mode in a.modes.split(","):
        traj = run(mode, a.steps, a.lr, a.wd, a.n, a.k, a.tokens, a.seed, a.log_every)
        print(json.dumps({"mode": mode, "steps": a.steps, "lr": a.lr, "weight_decay": a.wd,
                          "shape": [a.n, a.k], "tokens_per_step": a.tokens,
                          "trajectory": traj}), flush=True)


if __name__ == "__main__":
    main()
