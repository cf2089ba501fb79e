"""Offline profile of f_comp (Sec. VI-A): the time this GPU needs to run the
expert FFNs of the tokens it hosts, as a function of that token count lambda.

The profiled step is one ``moe_grouped_ffn`` call (the routed experts' grouped
SwiGLU FFN, the step whose time the paper's Eq. 2 models) with lambda rows
spread evenly over the experts a GPU hosts, for one model's expert shape.  The
points are fitted by a convex piecewise-linear model (``fit_convex_pwl``), the
form the placement LP takes.  Rows and weights are synthetic (seeded); the
weights of every hosted expert are distinct tensors, rotated over enough
copies to exceed the last-level cache, so small-lambda calls stream them from
HBM as a decode step does.

    python -m paper_2607_08782_amd.fcomp --config mixtral_8x7b --experts 2 \\
        --out profiles/fcomp_mixtral_8x7b.json
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys

import numpy as np
import torch

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    __package__ = "paper_2607_08782_amd"

from . import moe, synth  # noqa: E402
from .placement import fit_convex_pwl  # noqa: E402

DEFAULT_LAMBDAS = (0, 8, 16, 32, 64, 96, 128, 192, 256, 384, 512, 768, 1024, 1536, 2048,
                   3072, 4096, 6144, 8192)


def even_offsets(lam: int, n: int):
    base, rem = divmod(lam, n)
    sizes = [base + (1 if s < rem else 0) for s in range(n)]
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)


def profile(cfg_name: str, n_experts: int, lambdas=DEFAULT_LAMBDAS, reps: int = 10,
            warmup: int = 2, seed: int = 0, device: str = "cuda"):
    """Median microseconds of one moe_grouped_ffn call for each lambda."""
    cfg = synth.CONFIGS[cfg_name]
    d, f = cfg.d, cfg.f
    gen = torch.Generator(device="cpu").manual_seed(seed)
    std = 0.02

    def w(*shape):
        return (torch.randn(*shape, generator=gen) * std).to(torch.bfloat16).to(device)

    # enough distinct weight sets that consecutive calls cannot find the previous
    # call's weights in the 256 MB last-level cache
    set_bytes = n_experts * 3 * d * f * 2
    n_sets = max(1, -(-(512 << 20) // set_bytes))
    tables = []
    for _ in range(n_sets):
        w13 = [w(2 * f, d) for _ in range(n_experts)]
        w2 = [w(d, f) for _ in range(n_experts)]
        tables.append(moe.WeightTable(w13, w2))
    cap = max(max(lambdas), 1)
    x = torch.randn(cap, d, generator=gen).to(torch.bfloat16).to(device)
    y = torch.empty(cap, d, dtype=torch.bfloat16, device=device)
    ws = moe.workspace(moe.moe_grouped_ffn_ws_bytes(moe.MOE_BF16, cap, d, f, n_experts), device)
    points = []
    for lam in lambdas:
        off = torch.from_numpy(even_offsets(int(lam), n_experts)).to(device)
        for r in range(warmup):
            moe.moe_grouped_ffn(x, off, tables[r % n_sets], cap_rows=cap, y_perm=y, ws=ws)
        times = []
        for r in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            moe.moe_grouped_ffn(x, off, tables[r % n_sets], cap_rows=cap, y_perm=y, ws=ws)
            b.record()
            b.synchronize()
            times.append(a.elapsed_time(b) * 1e3)
        points.append((int(lam), float(statistics.median(times))))
        print("lambda %6d: %9.1f us" % points[-1], flush=True)
    return points


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--config", default="mixtral_8x7b", choices=sorted(synth.CONFIGS))
    ap.add_argument("--experts", type=int, default=2, help="experts hosted by the GPU")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--out", default=None)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("f_comp is profiled on the GPU; no GPU is visible")
    pts = profile(args.config, args.experts, reps=args.reps)
    # lambda = 0 (a GPU that receives no token) costs only the empty launches; a
    # convex model through it would undercut the weight-streaming floor of every
    # small lambda, so the fit uses lambda > 0 and the record keeps the point
    fit = [p for p in pts if p[0] > 0]
    pieces = fit_convex_pwl([p[0] for p in fit], [p[1] for p in fit])
    rec = {"config": args.config, "hosted_experts": args.experts, "unit": "microseconds",
           "step": "one moe_grouped_ffn call, lambda rows split evenly over the hosted experts",
           "points": pts, "pieces": pieces,
           "command": "python -m paper_2607_08782_amd.fcomp --config %s --experts %d --reps %d --out %s"
                      % (args.config, args.experts, args.reps, args.out)}
    text = json.dumps(rec, indent=1)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text + "\n")
    print(text)


if __name__ == "__main__":
    main()
