"""Offline profile of f_comp (Sec. VI-A): the time this GPU needs to run the
expert FFNs of the tokens it hosts, as a function of that token count lambda
and of how many of its experts those tokens reach.

The profiled step is one ``moe_grouped_ffn`` call (the routed experts' grouped
SwiGLU FFN, the step whose time the paper's Eq. 2 models) with lambda rows
spread evenly over `a` of the experts a GPU hosts (the others get none), for
one model's expert shape.  Eq. 2 prices the step by lambda alone; a
decode-sized step is instead set by the weights it streams, a x 3 d f x 2
bytes, so the profile covers a grid of (lambda, a).  The points with every
hosted expert active are fitted by a convex piecewise-linear model of lambda
(``fit_convex_pwl``), the whole grid by a convex piecewise-linear model of
(lambda, a) (``fit_convex_pwl2``, planes of the lower convex hull); both are
forms the placement LP takes.  Rows and weights are synthetic (seeded); the
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
from .placement import comp_eval, fit_convex_pwl, pwl_eval  # noqa: E402

DEFAULT_LAMBDAS = (0, 8, 16, 32, 64, 96, 128, 192, 256, 384, 512, 768, 1024, 1536, 2048,
                   3072, 4096, 6144, 8192)


def even_offsets(lam: int, n: int, active: int = None):
    """Group offsets of lam rows spread evenly over the first `active` of n groups."""
    active = n if active is None else active
    base, rem = divmod(lam, active) if active else (0, 0)
    sizes = [base + (1 if s < rem else 0) if s < active else 0 for s in range(n)]
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)


def fit_convex_pwl2(points):
    """Convex piecewise-linear t(lambda, a) = max over planes (slope, slope_a,
    intercept): the planes of the lower convex hull of the (lambda, a, t) points,
    so the model passes through or under every point.  Planes that fall with
    lambda or a (measurement noise at small loads) are dropped and replaced by a
    flat plane at the smallest time, as the one-variable fit does."""
    from scipy.spatial import ConvexHull

    P = np.asarray(points, dtype=np.float64)
    scale = np.maximum(np.abs(P).max(axis=0), 1.0)
    hull = ConvexHull(P / scale, qhull_options="Qt")
    planes = []
    for eq in hull.equations:
        nl, na, nt, off = eq[0] / scale[0], eq[1] / scale[1], eq[2] / scale[2], eq[3]
        if nt >= -1e-9:                                   # upper or vertical facet
            continue
        a, c, b = -nl / nt, -na / nt, -off / nt
        if a < -1e-9 or c < -1e-9:
            continue
        if not any(abs(a - p[0]) <= 1e-9 * (1 + abs(a)) and abs(c - p[1]) <= 1e-6 * (1 + abs(c))
                   and abs(b - p[2]) <= 1e-6 * (1 + abs(b)) for p in planes):
            planes.append((float(max(a, 0.0)), float(max(c, 0.0)), float(b)))
    planes.append((0.0, 0.0, float(P[:, 2].min())))
    return planes


def profile(cfg_name: str, n_experts: int, lambdas=DEFAULT_LAMBDAS, reps: int = 10,
            warmup: int = 2, seed: int = 0, device: str = "cuda", active=None):
    """Median microseconds of one moe_grouped_ffn call for each lambda (rows over
    `active` of the hosted experts, all of them by default)."""
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
        off = torch.from_numpy(even_offsets(int(lam), n_experts, active)).to(device)
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
        print("lambda %6d over %s experts: %9.1f us" % (points[-1][0], active or n_experts,
                                                        points[-1][1]), flush=True)
    return points


def grid_lambdas(a: int, lambdas=DEFAULT_LAMBDAS):
    """The lambdas of the grid row with `a` active experts: at least one row each."""
    return [lam for lam in lambdas if lam >= a]


def summary(paths):
    """Markdown summary of profile records (the lambda curve, the (lambda, a) grid,
    both fits and their worst relative error on the grid)."""
    lines = ["# f_comp profiles: time of one `moe_grouped_ffn` call vs. the tokens a GPU "
             "processes and the experts they reach", "",
             "The placement optimizer (Sec. VI-A) prices computation with f_comp, profiled "
             "offline.  Each point is the median of the timed calls (HIP events on the launch "
             "stream) of the routed-expert grouped FFN with lambda rows split evenly over a of "
             "the GPU's hosted experts (the others get no rows); weights are seeded synthetic "
             "bf16 tensors rotated over enough copies (at least 512 MB) that no call finds the "
             "previous call's weights in the 256 MB last-level cache.  Fits: convex "
             "piecewise-linear in lambda through the lower convex hull of the lambda > 0 points "
             "with every hosted expert active (Eq. 2's form), and convex piecewise-linear in "
             "(lambda, a) through the lower convex hull of the whole grid.  MI355X, ROCm 7.2.",
             "",
             "Summary command: `python -m paper_2607_08782_amd.fcomp --summary %s`"
             % " ".join(paths), ""]
    for path in paths:
        with open(path) as fh:
            rec = json.load(fh)
        cfg = synth.CONFIGS[rec["config"]]
        lines += ["## %s experts (d=%d, f=%d), %d hosted experts" % (
            rec["config"], cfg.d, cfg.f, rec["hosted_experts"]), "",
            "Command: `%s`" % rec["command"], "",
            "Pieces of lambda (slope us/token, intercept us): " +
            ", ".join("(%.4f, %.1f)" % tuple(p) for p in rec["pieces"]), ""]
        if "pieces_2d" in rec:
            err = rec["fit_error_2d"]
            lines += ["Planes of (lambda, a) (us/token, us/active expert, us): " +
                      ", ".join("(%.4f, %.2f, %.1f)" % tuple(p) for p in rec["pieces_2d"]), "",
                      "Worst relative error on the grid: %.0f %% for the lambda-only model, "
                      "%.0f %% for the (lambda, a) model." % (
                          100 * err["lambda_only_max_rel"], 100 * err["lambda_and_active_max_rel"]),
                      ""]
            acts = sorted({int(p[1]) for p in rec["points_2d"]})
            lams = sorted({int(p[0]) for p in rec["points_2d"]})
            t = {(int(p[0]), int(p[1])): p[2] for p in rec["points_2d"]}
            lines += ["| lambda | " + " | ".join("a = %d" % a for a in acts) + " |",
                      "|---|" + "---|" * len(acts)]
            for lam in lams:
                lines.append("| %d | " % lam + " | ".join(
                    "%.1f" % t[(lam, a)] if (lam, a) in t else "" for a in acts) + " |")
        else:
            lines += ["| lambda | us |", "|---|---|"]
            lines += ["| %d | %.1f |" % (lam, us) for lam, us in rec["points"]]
        lines.append("")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--summary", nargs="+", metavar="RECORD",
                    help="print the markdown summary of these profile records and exit")
    ap.add_argument("--config", default="mixtral_8x7b", choices=sorted(synth.CONFIGS))
    ap.add_argument("--experts", type=int, default=2, help="experts hosted by the GPU")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--grid", action="store_true",
                    help="also profile fewer active experts and fit f_comp(lambda, a)")
    ap.add_argument("--out", default=None)
    args = ap.parse_args(argv)
    if args.summary:
        print(summary(args.summary))
        return
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
           "command": "python -m paper_2607_08782_amd.fcomp --config %s --experts %d --reps %d%s --out %s"
                      % (args.config, args.experts, args.reps, " --grid" if args.grid else "",
                         args.out)}
    if args.grid:
        # (lambda, a, t): the rows of every a < all from their own runs, a = all from above
        grid = [(lam, args.experts, t) for lam, t in fit]
        for a in sorted({max(1, args.experts * q // 4) for q in (1, 2, 3)} - {args.experts}):
            grid += [(lam, a, t) for lam, t in profile(args.config, args.experts,
                                                         grid_lambdas(a), reps=args.reps,
                                                         active=a)]
        pieces2 = fit_convex_pwl2(grid)
        model1 = pwl_eval(pieces, [g[0] for g in grid])
        model2 = comp_eval(pieces2, [g[0] for g in grid], [g[1] for g in grid])
        meas = np.array([g[2] for g in grid])
        rec.update({
            "step_2d": "one moe_grouped_ffn call, lambda rows split evenly over a of the "
                       "hosted experts (the others get none)",
            "points_2d": grid, "pieces_2d": pieces2,
            "fit_error_2d": {
                "lambda_only_max_rel": float(np.max(np.abs(model1 - meas) / meas)),
                "lambda_and_active_max_rel": float(np.max(np.abs(model2 - meas) / meas))}})
    text = json.dumps(rec, indent=1)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text + "\n")
    print(text)


if __name__ == "__main__":
    main()
