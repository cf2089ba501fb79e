"""The layer share at every model shape and regime, measured on this GPU.

For each shape (Mixtral-8x7B, DeepSeek-V2-Lite, Qwen1.5-MoE-A2.7B and
Qwen3-30B-A3B-shaped shares; prefill and decode batches) and each seed 0-4:
synthetic inputs of that shape (seeded normal hidden states and weights, Zipf
popularity bias, the benchmark placement), the five calls captured in one HIP
graph, and the step timed over graph replays, for the share as LayerShare sets
itself up (the row copy x_perm elided for bf16 batches of at least 16384
token-expert assignments; shared experts inside the routed call up to 4096
tokens) and for the share on its first-built path (packaged row copy, shared
experts as a call of their own on a second stream); the FFN call of the default
share is timed the same way on its own (for batches of at most 64 tokens with k
<= 2 that call also writes the combine; with the shared experts inside, it runs
them too).  Reported: tokens/s, the FFN's rate against the bf16 MFMA peak (6 d f
per row) and against HBM (weights of the active experts read once plus the rows
in and out), mean and spread over the seeds.

Cache hygiene: when the local expert weights total less than 1 GB (they would
otherwise stay in the 256 MB last-level cache between replays), the replays
cycle through enough copies of them to touch at least 1 GB.

    python -m paper_2607_08782_amd.layer_study --out profiles/layer_by_shape.md
"""
from __future__ import annotations

import argparse
import math
import os
import statistics
import sys

import numpy as np
import torch

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    __package__ = "paper_2607_08782_amd"

from . import moe, synth  # noqa: E402
from .layer import LayerShare  # noqa: E402

PEAK_BF16_FLOPS = 2.5e15
PEAK_HBM_BYTES = 8.0e12
REGIMES = [("mixtral_8x7b", "prefill"), ("mixtral_8x7b", "decode"),
           ("deepseek_v2_lite", "prefill"), ("deepseek_v2_lite", "decode"),
           ("qwen15_moe_a27b", "batch"),
           ("qwen3_30b_a3b", "prefill"), ("qwen3_30b_a3b", "decode")]


def _graph(fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _time(graphs, steps, warmup=3):
    for i in range(warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(steps):
        graphs[i % len(graphs)].replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) * 1e3 / steps          # us per step


def measure(name, regime, seed, steps):
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    inp = synth.make_layer(cfg, T, seed=seed, device="cuda")
    wbytes = sum(w.numel() * 2 for w in inp.w13) + sum(w.numel() * 2 for w in inp.w2)
    copies = 1 if wbytes >= 1e9 else int(math.ceil(1e9 / max(wbytes, 1)))
    shares, fshares = [], []
    for c in range(copies):
        w13 = inp.w13 if c == 0 else [w.clone() for w in inp.w13]
        w2 = inp.w2 if c == 0 else [w.clone() for w in inp.w2]
        shares.append(LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2,
                                 shared=inp.shared, coact=cfg.coact))
        fshares.append(LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2,
                                  shared=inp.shared, coact=cfg.coact, gather_in_ffn=False,
                                  shared_in_ffn=False))
    for s in shares + fshares:
        s.run()
    torch.cuda.synchronize()
    s0 = shares[0]
    go = s0.perm["group_offsets"].cpu().numpy()
    sizes = np.diff(go)
    N, active = int(go[-1]), int((sizes > 0).sum())
    step_graphs = [_graph(s.run) for s in shares]
    first_graphs = [_graph(s.run) for s in fshares]

    ffn_graphs = [_graph(s.routed_ffn) for s in shares]
    # the two step variants interleaved (default, first-built, first-built, default),
    # each the mean of its two runs: the first timed run of a shape runs a few %
    # slower than later ones (clocks, first touches), which would favour whichever
    # variant came second
    _time(step_graphs, steps)
    step_us = _time(step_graphs, steps)
    first_us = _time(first_graphs, steps)
    first_us = (first_us + _time(first_graphs, steps)) / 2
    step_us = (step_us + _time(step_graphs, steps)) / 2
    ffn_us = _time(ffn_graphs, steps)
    flops = 6.0 * cfg.d * cfg.f * N
    # out: y_perm, or, when the call combines, y with the row maps and gates it reads
    out_bytes = (T * cfg.d * 2 + T * cfg.k * 8.0) if s0.fused_combine else N * cfg.d * 2
    fbytes = active * 3.0 * cfg.d * cfg.f * 2 + N * cfg.d * 2 + out_bytes
    nb = s0.n_shared_blocks
    if nb:
        # the call also runs the shared experts' blocks over every token
        flops += 6.0 * cfg.d * cfg.f * nb * T
        fbytes += nb * 3.0 * cfg.d * cfg.f * 2 + T * cfg.d * 2 + nb * T * cfg.d * 2
    out = {"T": T, "N": N, "active": active, "slots": len(sizes), "copies": copies, "blocks": nb,
           "step_us": step_us, "tok_s": T / (step_us * 1e-6), "ffn_us": ffn_us,
           "first_us": first_us,
           "ffn_tflops": flops / (ffn_us * 1e-6) / 1e12, "ffn_gbs": fbytes / (ffn_us * 1e-6) / 1e9}
    del step_graphs, first_graphs, ffn_graphs, shares, fshares
    torch.cuda.synchronize()
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--seeds", type=int, default=5)
    ap.add_argument("--steps", type=int, default=20, help="timed replays (decode: 10x)")
    ap.add_argument("--cases", default=None, help="comma-separated name/regime pairs")
    ap.add_argument("--out", default=None)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the study runs on the GPU; no GPU is visible")
    cases = REGIMES if not args.cases else [tuple(c.split("/")) for c in args.cases.split(",")]
    rows = []
    for name, regime in cases:
        steps = args.steps * (10 if regime == "decode" else 1)
        res = []
        for seed in range(args.seeds):
            res.append(measure(name, regime, seed, steps))
            print("  %s/%s seed %d: step %.1f us, FFN %.1f us" % (name, regime, seed,
                                                               res[-1]["step_us"], res[-1]["ffn_us"]),
                  flush=True)
        m = lambda k: statistics.mean(r[k] for r in res)
        sd = lambda k: statistics.pstdev(r[k] for r in res)
        row = {"name": name, "regime": regime, "res": res, "m": m, "sd": sd}
        rows.append(row)
        print("%s/%s: step %.1f us (%.3g tok/s), first-built path step %.1f us, FFN %.1f us = %.0f TFLOP/s, "
              "%.0f GB/s; N %.0f, active %.1f, copies %d" % (name, regime, m("step_us"), m("tok_s"),
                                                            m("first_us"), m("ffn_us"),
                                          m("ffn_tflops"), m("ffn_gbs"), m("N"), m("active"),
                                          res[0]["copies"]), flush=True)
    lines = ["# The layer share at every model shape and regime", "",
             "Synthetic seeded inputs of each shape (normal hidden states, N(0, 0.02) weights, Zipf",
             "popularity bias, the benchmark placement with this GPU = device 0).  Step = the five",
             "calls as one HIP graph replay; FFN = the routed experts' FFN call as the step makes it",
             "(`moe_grouped_ffn`; `moe_grouped_ffn_combine` for batches of at most 64 tokens with",
             "k <= 2, which also writes the combined output; `moe_grouped_ffn_rows_shared` with the",
             "shared experts' blocks of width f as leading groups where the share runs them inside",
             "the routed call, their work then counted too) replayed on its own.  Mean (± population std) over seeds 0-%d; %d timed replays per"
             % (args.seeds - 1, args.steps),
             "seed for prefill-sized batches, %d for decode.  FFN rate against the bf16 MFMA peak"
             % (args.steps * 10),
             "(2.5 PFLOP/s, algorithmic 6·d·f·N flop) and against HBM (8 TB/s, algorithmic bytes: the",
             "active local experts' weights once, x_perm in, y_perm or the combined y out).  Weight",
             "copies: replays cycle through this many copies of the local expert weights (≥ 1 GB",
             "touched).",
             "Step: the share as LayerShare sets itself up (the row copy x_perm elided -- moe_permute",
             "writes the row maps only and the FFN reads the token rows through row_token -- for bf16",
             "batches of at least 16384 token-expert assignments; shared experts as leading groups of",
             "the routed call up to 4096 tokens).  First-built path: the same share with the packaged",
             "row copy and the shared experts as a call of their own on a second stream.", "",
             "Command: `python -m paper_2607_08782_amd.layer_study --seeds %d --steps %d --out %s`"
             % (args.seeds, args.steps, args.out), "",
             "| shape / regime | T | rows here N | active / local experts | shared blocks in the call | weight copies | step us | tokens/s | first-built path step us | FFN us | FFN TFLOP/s (% bf16 peak) | FFN GB/s (% HBM peak) |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        m, sd, res = r["m"], r["sd"], r["res"]
        lines.append("| %s/%s | %d | %.0f | %.1f / %d | %d | %d | %.1f ± %.1f | %.3g | %.1f | %.1f ± %.1f | %.0f (%.1f %%) | %.0f (%.1f %%) |" % (
            r["name"], r["regime"], res[0]["T"], m("N"), m("active"), res[0]["slots"],
            res[0]["blocks"], res[0]["copies"], m("step_us"), sd("step_us"), m("tok_s"), m("first_us"), m("ffn_us"),
            sd("ffn_us"),
            m("ffn_tflops"), 100 * m("ffn_tflops") * 1e12 / PEAK_BF16_FLOPS, m("ffn_gbs"),
            100 * m("ffn_gbs") * 1e9 / PEAK_HBM_BYTES))
    lines.append("")
    text = "\n".join(lines)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(text)
    print(text)


if __name__ == "__main__":
    main()
