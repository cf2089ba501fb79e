"""Proactive vs. reactive vs. static placement on a drifting workload (Sec. III,
Finding 3; Sec. VI), measured on this GPU.

For each batch of a drifting sequence (Qwen1.5-MoE-shaped layer: 60 experts, 8
GPUs, top-4; the expert popularity is re-drawn every 4 batches) the GPU routes
every GPU's slice of the batch and counts tokens per expert
(``moe_route_topk`` + ``moe_expert_histogram``), giving the workload matrix W_b
(Sec. VI-A).  Three placements are compared on each batch:

* static: the placement computed once from the first batch, kept;
* reactive: the optimizer's placement for the previous batch (the best a
  system that reacts to observed load can do);
* proactive: the optimizer's placement for the batch itself (Director with a
  perfect predictor).

Each is priced with the model of Eq. 1-4, using f_comp profiled on this GPU
(``profiles/fcomp_qwen15_moe_a27b.json``) and f_comm = 5 us + bytes / 153 GB/s
per peer (one xGMI link; a model, not a measurement), and its computation side
is also measured: the straggler GPU's expert step is run for real (its share of
the batch packaged by ``moe_permute`` and pushed through ``moe_grouped_ffn``) and
timed.

    python -m paper_2607_08782_amd.placement_study --out profiles/placement_qwen15_drift.md
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np
import torch

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    __package__ = "paper_2607_08782_amd"

from . import moe, placement as pl, synth  # noqa: E402
from .migration import WINDOW_MARGIN  # noqa: E402
from .layer import LayerShare  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LINK_BYTES_PER_US = 153e9 / 1e6
LINK_LATENCY_US = 5.0


def workload(inp, cfg, G):
    T = inp.X.shape[0]
    W = np.zeros((G, cfg.E), np.int64)
    for j in range(G):
        Xj = inp.X[j * T // G:(j + 1) * T // G].contiguous()
        _, idx, _ = moe.moe_route_topk(Xj, inp.Wr, inp.bias, cfg.k, renorm=True, want_logits=False)
        counts, _ = moe.moe_expert_histogram(idx, cfg.E)
        W[j] = counts.cpu().numpy()
    return W


def straggler_ffn_us(inp, cfg, x_map, weights, reps=5):
    """Measured time of the routed-expert FFN step of the busiest GPU."""
    G = x_map.shape[1]
    worst = 0.0
    for dev in range(G):
        local = [int(e) for e in np.nonzero(x_map[:, dev])[0]]
        if not local:
            continue
        share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, x_map, dev,
                           [weights[e][0] for e in local], [weights[e][1] for e in local])
        share.run()
        times = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            share.routed_ffn(fused=False)
            b.record()
            b.synchronize()
            times.append(a.elapsed_time(b) * 1e3)
        worst = max(worst, statistics.median(times))
    return worst


def migration_rows(cfg, G, T, weights, plans, f_comp, dev=0, reps=3):
    """For each change of the proactive placement on `dev`: bytes brought in, the
    copies scheduled into the FFN windows of the following steps, the steps needed,
    the FFN time with and without copies in flight, and the wait at window close."""
    from .migration import ExpertStore, Migrator, measure_h2d_rate, run_step

    store = ExpertStore([w[0] for w in weights], [w[1] for w in weights])
    rate = measure_h2d_rate()                                   # bytes per us
    out = []
    for b in range(1, len(plans)):
        P_old, P_new = plans[b - 1], plans[b]
        x_old = np.zeros((cfg.E, G), np.uint8); x_old[np.arange(cfg.E), P_old[0]] = 1
        x_new = np.zeros((cfg.E, G), np.uint8); x_new[np.arange(cfg.E), P_new[0]] = 1
        inc = set(np.nonzero(x_new[:, dev])[0]) - set(np.nonzero(x_old[:, dev])[0])
        if not inc or x_new[:, dev].sum() != x_old[:, dev].sum():
            continue
        inp = synth.make_layer(cfg, T, seed=0, device="cuda", batch=b, experts="none")
        mig = Migrator(store, x_old, dev, spare=len(inc), chunk_bytes=1 << 20)
        w13, w2 = mig.weights()
        share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, x_old, dev, w13, w2)
        base = {}
        for _ in range(reps):
            run_step(share, None, 0, base)
        # what closing a window costs with nothing copied in it (the stream join)
        join = [run_step(share, mig, 0, None, empty=True) * 1e3 for _ in range(2 * reps + 1)]
        lam = int(share.perm["group_offsets"][-1])
        act = int((torch.diff(share.perm["group_offsets"]) > 0).sum())
        window_us = float(pl.comp_eval(f_comp, lam, act))
        moved = mig.plan(x_new)
        # the first window from f_comp at half the uncontended copy rate (copies run
        # slower beside the computation), the next ones from the last window's rate
        mig.budget_bytes = int(WINDOW_MARGIN * window_us * rate / 2)
        mig.window_ms = statistics.median(base["ffn"])      # the FFN without copies
        during, stalls, steps = {}, [], 0
        while not mig.finished:
            st = run_step(share, mig, None, during)
            stalls.append(0.0 if st is None else st * 1e3)
            steps += 1
        torch.cuda.synchronize()
        ffn_alone = statistics.median(base["ffn"]) * 1e3
        ffn_copy = statistics.median(during["ffn"]) * 1e3
        out.append({"batch": b, "experts_in": len(inc), "mbytes": moved / 1e6, "rate_gbs": rate / 1e3,
                    "window_us": window_us, "steps": steps, "ffn_us": ffn_alone,
                    "ffn_copy_us": ffn_copy, "slowdown": ffn_copy / ffn_alone - 1.0,
                    "copy_rate_gbs": moved / (sum(during["copy"]) * 1e-3) / 1e9,
                    "max_stall_us": max(stalls), "median_stall_us": statistics.median(stalls),
                    "join_us": statistics.median(join)})
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--batches", type=int, default=16)
    ap.add_argument("--cmax", type=int, default=8)
    ap.add_argument("--out", default=None)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the study routes and times on the GPU; no GPU is visible")
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    G, T = cfg.G, cfg.T("batch")
    prof = json.load(open(os.path.join(ROOT, "profiles", "fcomp_qwen15_moe_a27b.json")))
    # f_comp of the load and the active-expert count when the profile has its grid
    f_comp = [tuple(p) for p in prof.get("pieces_2d", prof["pieces"])]
    f_comm = [(1.0 / LINK_BYTES_PER_US, LINK_LATENCY_US)]
    d_bytes = cfg.d * 2.0
    weights = [synth.expert_weights(cfg, e, 0, "cuda") for e in range(cfg.E)]
    rows, P_prev, P_static = [], None, None
    opt_s, proactive = [], []
    for b in range(args.batches):
        inp = synth.make_layer(cfg, T, seed=0, device="cuda", batch=b, experts="none")
        W = workload(inp, cfg, G)
        t0 = time.perf_counter()
        res = pl.place(W[None], G, args.cmax, d_bytes, f_comp, f_comm, seed=b)
        opt_s.append(time.perf_counter() - t0)
        # the paper's procedure alone: binary search, iterative rounding, completion
        alg1 = pl.place(W[None], G, args.cmax, d_bytes, f_comp, f_comm, seed=b, polish=False)
        if P_static is None:
            P_static = res.P
        plans = {"static": P_static, "reactive": P_prev if P_prev is not None else P_static,
                 "proactive": res.P, "alg1": alg1.P}
        row = {"batch": b, "beta_star": res.beta_star, "alg1_beta_star": alg1.beta_star}
        for name, P in plans.items():
            comp, comm = pl.layer_latencies(W[None].astype(np.float64), P, d_bytes, f_comp, f_comm)
            x_map = np.zeros((cfg.E, G), np.uint8)
            x_map[np.arange(cfg.E), P[0]] = 1
            row[name] = {"model_us": float(comp[0] + comm[0]), "comp_us": float(comp[0]),
                         "comm_us": float(comm[0]),
                         "measured_ffn_us": straggler_ffn_us(inp, cfg, x_map, weights)}
        rows.append(row)
        P_prev = res.P
        proactive.append(res.P)
        print("batch %2d: beta* %.1f | static %.1f | reactive %.1f | proactive %.1f | Alg. 1 alone "
              "%.1f (model us)" % (b, res.beta_star, row["static"]["model_us"],
                                   row["reactive"]["model_us"], row["proactive"]["model_us"],
                                   row["alg1"]["model_us"]), flush=True)
    mean = lambda k, f: statistics.mean(r[k][f] for r in rows)
    lines = ["# Proactive vs. reactive vs. static placement on a drifting workload", "",
             "Qwen1.5-MoE-A2.7B-shaped layer (d=2048, 60 experts, top-4, f=1408), 8 GPUs, C_max = %d,"
             % args.cmax,
             "%d batches of %d tokens (a GPU slice each of %d), popularity re-drawn every %d batches;"
             % (args.batches, T, T // G, cfg.drift_every),
             "synthetic seeded inputs.  Model: Eq. 1-4 with f_comp profiled on this GPU (%s) and"
             % ("a convex piecewise-linear function of the GPU's load and of its active experts"
                if "pieces_2d" in prof else "a convex piecewise-linear function of the load"),
             "f_comm = %.0f us + bytes / 153 GB/s per peer (modelled link).  Measured: the busiest"
             % LINK_LATENCY_US,
             "GPU's `moe_grouped_ffn` step under each placement, median of 5 timed calls.",
             "Proactive = the optimizer as the library runs it (Alg. 1, then a move/swap polish that",
             "is not the paper's, keeping the polished greedy placement when it is better); Alg. 1",
             "alone = binary search, iterative rounding and completion only.", "",
             "Command: `python -m paper_2607_08782_amd.placement_study --batches %d --cmax %d --out %s`"
             % (args.batches, args.cmax, args.out), "",
             "| batch | beta* (LP) | static model | reactive model | proactive model | Alg. 1 alone model | proactive T/beta* | Alg. 1 alone T/beta* | static FFN | reactive FFN | proactive FFN | Alg. 1 alone FFN |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %d | %.1f | %.1f | %.1f | %.1f | %.1f | %.3f | %.3f | %.1f | %.1f | %.1f | %.1f |" % (
            r["batch"], r["beta_star"], r["static"]["model_us"], r["reactive"]["model_us"],
            r["proactive"]["model_us"], r["alg1"]["model_us"],
            r["proactive"]["model_us"] / r["beta_star"], r["alg1"]["model_us"] / r["beta_star"],
            r["static"]["measured_ffn_us"], r["reactive"]["measured_ffn_us"],
            r["proactive"]["measured_ffn_us"], r["alg1"]["measured_ffn_us"]))
    lines.append("| mean | %.1f | %.1f | %.1f | %.1f | %.1f | %.3f | %.3f | %.1f | %.1f | %.1f | %.1f |" % (
        statistics.mean(r["beta_star"] for r in rows), mean("static", "model_us"),
        mean("reactive", "model_us"), mean("proactive", "model_us"), mean("alg1", "model_us"),
        statistics.mean(r["proactive"]["model_us"] / r["beta_star"] for r in rows),
        statistics.mean(r["alg1"]["model_us"] / r["beta_star"] for r in rows),
        mean("static", "measured_ffn_us"), mean("reactive", "measured_ffn_us"),
        mean("proactive", "measured_ffn_us"), mean("alg1", "measured_ffn_us")))
    lines += ["", "All times in microseconds.  Optimizer wall time per batch (host CPU): "
              "median %.2f s, max %.2f s." % (statistics.median(opt_s), max(opt_s)), ""]
    mrows = migration_rows(cfg, G, T, weights, proactive, f_comp)
    lines += ["## Migrating to each new proactive placement (GPU 0, Sec. V-B)", "",
              "Incoming experts are copied from pinned host memory (standing in for the peer",
              "GPUs; a host-to-device copy on the DMA engines) into spare buffers, chunk by chunk,",
              "inside the FFN window of the following steps, and the step waits for them where",
              "the window closes (where the combine's all-to-all would start); the computation is",
              "enqueued before the copies, which wait for the window's opening on the device.",
              "Chunks of 1 MB.  The first window gets %.2f x f_comp(lambda, a of GPU 0) x half the"
              % WINDOW_MARGIN,
              "uncontended copy rate; every later window the bytes the last window's copies moved per ms",
              "(with the FFN running), times the FFN's time without copies, times %.2f.  The batch"
              % WINDOW_MARGIN,
              "keeps being served on the old placement meanwhile.  The wait at the window's",
              "close includes the stream join itself, measured with windows that copy nothing",
              "(join); late = wait - join.  Copy GB/s in windows = bytes over the windows' open-to-",
              "last-copy times (joins included).", "",
              "| batch | experts in | MB | copy GB/s alone | copy GB/s in windows | first window us | steps | FFN us alone | FFN us with copies | FFN slowdown | join us | median / max late us |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for m in mrows:
        lines.append("| %d | %d | %.1f | %.1f | %.1f | %.1f | %d | %.1f | %.1f | %.0f %% | %.1f | %.1f / %.1f |" % (
            m["batch"], m["experts_in"], m["mbytes"], m["rate_gbs"], m["copy_rate_gbs"],
            m["window_us"], m["steps"], m["ffn_us"], m["ffn_copy_us"], 100 * m["slowdown"],
            m["join_us"], m["median_stall_us"] - m["join_us"], m["max_stall_us"] - m["join_us"]))
    lines.append("")
    text = "\n".join(lines)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    print(text)


if __name__ == "__main__":
    main()
