"""Benchmark: one GPU's share of a Mixtral-8x7B-shaped MoE layer on MI355X.

A step is one pass of the whole share (gate scores + top-k, histograms,
packaging, grouped SwiGLU FFN, weighted combine) over one batch of synthetic
tokens already resident in HBM.  The headline is the prefill batch (T=4096);
the decode batch (T=64) is reported beside it.  `gather_in_ffn` reports the
same step with the row copy x_perm elided (the expert FFN reads the token rows
through the row map), and whether its output matches bit for bit; the
headline keeps the packaged copy.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME:REGIME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2607_08782_amd import moe, synth  # noqa: E402
from paper_2607_08782_amd.layer import LayerShare  # noqa: E402

METRIC = "MoE-layer tokens/s on 1 GPU; grouped-GEMM % bf16 MFMA peak; decode HBM GB/s"
PEAK_BF16_FLOPS = 2.5e15        # MI355X dense bf16 MFMA
PEAK_HBM_BYTES = 8.0e12         # MI355X HBM3E
PHASES = ("route_topk", "histogram", "permute", "grouped_ffn", "shared_ffn", "combine")


def make_share(cfg, T, seed=0, weights=None):
    inp = synth.make_layer(cfg, T, seed=seed, device="cuda", experts="none" if weights else "local")
    w13, w2, shared = weights if weights else (inp.w13, inp.w2, inp.shared)
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2, shared=shared,
                       coact=cfg.coact)
    return inp, share, (w13, w2, shared)


def gathered_variant(inp, share, weights, cfg, steps, warmup):
    """The same share with the row copy x_perm elided (moe_permute writes the row maps
    only, moe_grouped_ffn_rows reads the token rows through row_token): step time from
    graph replays, and whether its output equals the packaged path's bit for bit."""
    w13, w2, shared = weights
    g = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2, shared=shared,
                   coact=cfg.coact, gather_in_ffn=True)
    share.run()
    g.run()
    torch.cuda.synchronize()
    equal = bool(torch.equal(share.y, g.y))
    ms = time_replays(capture(g.run), steps, warmup)
    return {"ms_per_step": ms, "tokens_per_s": share.T / (ms * 1e-3),
            "bitwise_equal_output": equal,
            "what": "row copy x_perm elided: moe_permute writes the row maps only and "
                    "moe_grouped_ffn_rows reads the token rows through row_token"}


def phase_calls(share):
    """The calls of LayerShare.run, one callable per phase."""
    def route():
        share.route()

    def histogram():
        moe.moe_expert_histogram(share.topk_idx, share.E, counts=share.counts, coact=share.coact)

    def permute():
        moe.moe_permute(share.X, share.topk_idx, share.topk_gate, share.counts, share.placement,
                        share.dev, E=share.E, cap_rows=share.cap_rows, out=share.perm,
                        ws=share.ws_perm)

    def grouped_ffn():
        if share.weights is not None:
            moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"], share.weights,
                                cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn)

    def shared_ffn():
        if share.shared_weights is not None:
            moe.moe_grouped_ffn(share.X, share.shared_offsets, share.shared_weights,
                                cap_rows=share.T, y_perm=share.y_shared, ws=share.ws_shared)

    def combine():
        moe.moe_combine(share.y_perm, share.perm["token_row"], share.topk_gate, share.y_shared,
                        T=share.T, d=share.d, y=share.y)

    return dict(route_topk=route, histogram=histogram, permute=permute, grouped_ffn=grouped_ffn,
                shared_ffn=shared_ffn, combine=combine)


def capture(fn):
    """One HIP graph of `fn`'s launches (captured on torch's capture stream)."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def time_replays(g, steps, warmup):
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def time_share(share, steps, warmup):
    """Step time from HIP-graph replays of the whole share.  Per-phase GPU time
    from an eager timed loop with an event after every call on the stream the
    calls are enqueued on (torch's current stream); the eager step time is
    reported beside the graph one."""
    calls = phase_calls(share)
    for _ in range(warmup):
        share.run()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(PHASES) + 1)]
           for _ in range(steps)]
    for i in range(steps):
        evs[i][0].record()
        for j, name in enumerate(PHASES):
            calls[name]()
            evs[i][j + 1].record()
    torch.cuda.synchronize()
    phases = {name: sum(ev[j].elapsed_time(ev[j + 1]) for ev in evs) / steps
              for j, name in enumerate(PHASES)}
    eager_ms = evs[0][0].elapsed_time(evs[-1][-1]) / steps
    ms = time_replays(capture(share.run), steps, warmup)
    share.run()
    torch.cuda.synchronize()
    return ms, phases, eager_ms


def measured_traffic(workload):
    """HBM bytes per moe_grouped_ffn call from the committed PMC record, or None
    when the record is missing or the FFN kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "ffn_traffic.json")
    try:
        rec = json.load(open(path))
        src = open(os.path.join(ROOT, rec["kernel_source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec.get("source_sha256") or workload not in rec:
        return None
    return rec[workload]["read"] + rec[workload]["write"]


def ffn_work(share, cfg):
    go = share.perm["group_offsets"].cpu().numpy()
    sizes = np.diff(go)
    N = int(go[-1])
    active = int((sizes > 0).sum())
    flops = 6.0 * cfg.d * cfg.f * N
    bytes_ = active * 3.0 * cfg.d * cfg.f * 2 + 2.0 * N * cfg.d * 2
    return N, active, flops, bytes_, sizes.tolist()


def cpu_baseline(cfg, inp_gpu, w13, w2, shared, T_full):
    """The oracle, as it stands, on a bounded sample of the same batch."""
    import oracle

    f32 = lambda t: t.detach().float().cpu().numpy()
    X = f32(inp_gpu.X)
    Wr, b = f32(inp_gpu.Wr), f32(inp_gpu.bias)
    W13 = [f32(w) for w in w13]
    W2 = [f32(w) for w in w2]
    SH = [(f32(a), f32(c)) for a, c in shared]

    def run(S):
        t0 = time.perf_counter()
        oracle.layer_share(X[:S], Wr, b, cfg.k, inp_gpu.placement, 0, W13, W2, shared=SH,
                           with_coact=cfg.coact)
        return time.perf_counter() - t0

    S0 = 16
    t0 = run(S0)
    S = int(min(T_full, max(S0, S0 * 20.0 / max(t0, 1e-6))))
    t = run(S)
    return {"value": S / t, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": "first %d of the %d tokens of the same batch through the whole share "
                      "(fp64 C loops), %.1f s" % (S, T_full, t)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral_8x7b:prefill")
    ap.add_argument("--decode", default="decode", help="regime reported beside the headline ('' = none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather-variant", action="store_true",
                    help="skip the gather_in_ffn timing (a profiled run then dispatches only the "
                         "packaged path, in the order profsum expects)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run a plain elementwise copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU's share of the layer; --gpus %d is not supported "
              "(multi-GPU expert parallelism is design-only in this build)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    moe.load_library()
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)                 # reads and writes n*4 bytes each
        torch.cuda.synchronize()
        del src, dst
    name, regime = args.workload.split(":")
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)

    inp, share, weights = make_share(cfg, T)
    ms, phases, eager_ms = time_share(share, args.steps, args.warmup)
    N, active, flops, fbytes, sizes = ffn_work(share, cfg)
    t_ffn = phases["grouped_ffn"] * 1e-3
    achieved = flops / t_ffn
    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "eager_ms_per_step": eager_ms,
        "launch": "each step is one HIP graph replay of the five C-ABI calls",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": "%s-shaped MoE layer share, %s batch T=%d: d=%d, E=%d routed experts, "
                        "top-%d, SwiGLU f=%d, %d of %d experts on this GPU (G=%d), Zipf s=%s"
                        % (name, regime, T, cfg.d, cfg.E, cfg.k, cfg.f, share.n_local, cfg.E,
                           cfg.G, cfg.zipf),
            "T": T, "d": cfg.d, "E": cfg.E, "k": cfg.k, "f": cfg.f, "G": cfg.G,
            "local_experts": share.n_local, "rows_here": N, "group_rows": sizes, "seed": 0,
        },
        "roofline": {
            "kernel": "moe_grouped_ffn (grouped_gemm_kernel<swiglu> + grouped_gemm_kernel<plain>)",
            "bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK_BF16_FLOPS / 1e12,
            "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_FLOPS,
            "traffic": measured_traffic("%s:%s" % (name, regime)), "traffic_unit": "bytes per launch",
            "algorithmic_flops_per_launch": flops, "avg_launch_us": t_ffn * 1e6,
        },
        "phases_us": {k: v * 1e3 for k, v in phases.items()},
    }
    if not args.no_gather_variant:
        out["gather_in_ffn"] = gathered_variant(inp, share, weights, cfg, args.steps, args.warmup)
    if args.decode and args.decode in dict(cfg.regimes) and args.decode != regime:
        Td = cfg.T(args.decode)
        dinp, dshare, _ = make_share(cfg, Td, weights=weights)
        dms, dph, deager = time_share(dshare, max(args.steps * 5, 50), args.warmup * 2)
        dN, dact, dfl, dby, dsizes = ffn_work(dshare, cfg)
        dt = dph["grouped_ffn"] * 1e-3
        out["decode"] = {
            "T": Td, "tokens_per_s": Td / (dms * 1e-3), "ms_per_step": dms,
            "eager_ms_per_step": deager, "rows_here": dN,
            "active_experts": dact,
            "roofline": {"kernel": "moe_grouped_ffn", "bound": "hbm",
                         "achieved": dby / dt / 1e9, "peak": PEAK_HBM_BYTES / 1e9, "unit": "GB/s",
                         "frac": dby / dt / PEAK_HBM_BYTES,
                         "traffic": measured_traffic("%s:%s" % (name, args.decode)),
                         "traffic_unit": "bytes per launch",
                         "algorithmic_bytes_per_launch": dby, "avg_launch_us": dt * 1e6},
            "phases_us": {k: v * 1e3 for k, v in dph.items()},
        }
        if not args.no_gather_variant:
            out["decode"]["gather_in_ffn"] = gathered_variant(
                dinp, dshare, weights, cfg, max(args.steps * 5, 50), args.warmup * 2)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, inp, *weights, T)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
