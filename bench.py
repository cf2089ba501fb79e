"""Benchmark: one GPU's share of an MoE layer on MI355X, at every model shape.

A step is one pass of the whole share (gate scores + top-k, histograms,
packaging, grouped SwiGLU FFN, weighted combine) over one batch of synthetic
tokens already resident in HBM, timed as replays of one HIP graph holding the
five C-ABI calls.  Replays cycle through copies of the local expert weights
until at least 1 GB of weights is touched, so no shape runs out of the 256 MB
last-level cache.

The headline is the Mixtral-8x7B-shaped prefill batch (T = 4096); its roofline
entry is the dominant kernel, the gate/up GEMM of the grouped FFN, timed live as
graph replays of the gate/up product alone (moe_grouped_ffn_products), beside the
whole FFN call.  The decode batch (T = 64) is reported beside it, and `shapes`
holds every other configured layer (the tiny fp32 layer, DeepSeek-V2-Lite and
Qwen3-30B-A3B prefill and decode, the 16-batch Qwen1.5-MoE drift sequence with
its placement swaps), each as LayerShare sets itself up (at the Qwen1.5-MoE and
DeepSeek-V2-Lite decode shapes the shared experts run inside the routed FFN
call, whose rate then counts their work too; `ffn_call` names what each call
launches).  `gather_in_ffn` reports the headline step with the row copy x_perm
elided.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME:REGIME]
                    [--shapes all|none] [--no-cpu-baseline] [--no-gather-variant]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import platform
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
PEAK_FP32_FLOPS = 157.3e12      # MI355X fp32 vector
PEAK_HBM_BYTES = 8.0e12         # MI355X HBM3E
PHASES = ("route_topk", "histogram", "permute", "grouped_ffn", "shared_ffn", "combine")
ROTATE_BYTES = 1e9              # weight bytes touched per cycle of replays
MAX_COPIES = 16
SHAPES = [("tiny_fp32", "batch"), ("deepseek_v2_lite", "prefill"), ("deepseek_v2_lite", "decode"),
          ("qwen15_moe_a27b", "drift"), ("qwen3_30b_a3b", "prefill"), ("qwen3_30b_a3b", "decode")]
DOMINANT = "grouped_gemm_kernel<true, false>"


# ---------------------------------------------------------------------------
# graphs and timing
# ---------------------------------------------------------------------------
def capture(fn):
    """One HIP graph of `fn`'s launches (captured on torch's capture stream)."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def time_replays(graphs, steps, warmup):
    """Average ms per replay, cycling through `graphs` (HIP events on the current
    stream, which each replay joins before and after)."""
    for i in range(warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        graphs[i % len(graphs)].replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def weight_bytes(inp):
    return sum(w.numel() * w.element_size() for w in inp.w13 + inp.w2)


def rotated_shares(cfg, inp, **kw):
    """LayerShares over copies of the local expert weights, enough copies to touch
    ROTATE_BYTES per cycle (the first share uses the generated weights)."""
    wb = weight_bytes(inp)
    copies = 1 if wb >= ROTATE_BYTES else int(math.ceil(ROTATE_BYTES / max(wb, 1)))
    if cfg.dtype == "f32":
        copies = 1                   # the tiny fp32 layer is a parity case, not a bandwidth one
    copies = min(copies, MAX_COPIES)
    shares = []
    for c in range(copies):
        w13 = inp.w13 if c == 0 else [w.clone() for w in inp.w13]
        w2 = inp.w2 if c == 0 else [w.clone() for w in inp.w2]
        shares.append(LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2,
                                 shared=inp.shared, coact=cfg.coact, **kw))
    return shares


def ffn_call(share, products=None):
    """The routed experts' FFN call as LayerShare.run makes it (LayerShare.routed_ffn:
    moe_grouped_ffn, or moe_grouped_ffn_combine when the share fuses the combine), or
    the given products of moe_grouped_ffn alone."""
    if products is None:
        return share.routed_ffn
    if share.gather_in_ffn:
        raise ValueError("a share that gathers its rows in the FFN has no x_perm to run "
                         "single products on")
    # with the share's own hints, as its step passes them to the whole call
    products |= share.ffn_products & (moe.MOE_FFN_SMALL_GROUPS | moe.MOE_FFN_LARGE_GROUPS)
    return lambda: moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"],
                                       share.weights, cap_rows=share.cap_rows, y_perm=share.y_perm,
                                       ws=share.ws_ffn, products=products)


def ffn_label(share):
    """What the routed experts' FFN call of `share` launches."""
    if share.shared_in_ffn:
        what = ("weight-streaming launches" if share.ffn_products & moe.MOE_FFN_SMALL_GROUPS
                else "gate/up and down tiled GEMMs")
        return ("moe_grouped_ffn_rows_shared call: the routed experts and the shared experts' "
                "%d blocks of width f in one call (%s, chunk sums)" % (share.n_shared_blocks, what))
    if share.fused_combine:
        return ("moe_grouped_ffn_combine call (weight-streaming launches, the combine in the "
                "down product's chunk sum)")
    if share.gather_in_ffn:
        what = ("weight-streaming launches" if share.ffn_products & moe.MOE_FFN_SMALL_GROUPS
                else "gate/up and down tiled GEMMs")
        return ("moe_grouped_ffn_rows call: rows read through the row map (%s, chunk sums)" % what)
    if share.ffn_products & moe.MOE_FFN_SMALL_GROUPS:
        return "moe_grouped_ffn call (weight-streaming launches, chunk sums)"
    if share.ffn_products & moe.MOE_FFN_LARGE_GROUPS:
        return "moe_grouped_ffn call (gate/up and down tiled GEMMs, chunk sums; every group tiled)"
    return "moe_grouped_ffn call (gate/up and down tiled GEMMs, streaming launches, chunk sums)"


def ffn_work(share, cfg):
    go = share.perm["group_offsets"].cpu().numpy()
    sizes = np.diff(go)
    N = int(go[-1])
    active = int((sizes > 0).sum())
    esz = 4 if cfg.dtype == "f32" else 2
    # weights of the active experts once, the rows in, and the rows out (y_perm), or,
    # when the call combines, the tokens' outputs y with their row maps and gates
    out = (share.T * cfg.d * esz + share.T * cfg.k * 8.0) if share.fused_combine else N * cfg.d * esz
    w = {"N": N, "active": active, "sizes": sizes.tolist(),
         "flops": 6.0 * cfg.d * cfg.f * N, "gate_up_flops": 4.0 * cfg.d * cfg.f * N,
         "bytes": active * 3.0 * cfg.d * cfg.f * esz + N * cfg.d * esz + out}
    if share.shared_in_ffn:
        # the call also runs the shared experts' blocks over every token: their
        # weights once, the token rows in, one output slice per block
        nb, T = share.n_shared_blocks, share.T
        w["shared_blocks"] = nb
        w["flops"] += 6.0 * cfg.d * cfg.f * nb * T
        w["gate_up_flops"] += 4.0 * cfg.d * cfg.f * nb * T
        w["bytes"] += nb * 3.0 * cfg.d * cfg.f * esz + T * cfg.d * esz + nb * T * cfg.d * esz
    return w


def phase_calls(share):
    """The calls of LayerShare.run, one callable per phase (for the eager breakdown)."""
    def route():
        share.route()

    def histogram():
        moe.moe_expert_histogram(share.topk_idx, share.E, counts=share.counts, coact=share.coact)

    def permute():
        share.package()

    def grouped_ffn():
        share.routed_ffn()

    def shared_ffn():
        share._shared_ffn()                # nothing when the shared experts share the call

    def combine():
        if not share.fused_combine:        # else part of grouped_ffn
            share.combine()

    return dict(route_topk=route, histogram=histogram, permute=permute, grouped_ffn=grouped_ffn,
                shared_ffn=shared_ffn, combine=combine)


def eager_phases(share, steps, warmup):
    """Per-phase GPU time of the calls launched one after another from Python, with
    an event after every call on torch's current stream (every call's stream)."""
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
    phases = {name: 1e3 * sum(ev[j].elapsed_time(ev[j + 1]) for ev in evs) / steps
              for j, name in enumerate(PHASES)}
    eager_ms = evs[0][0].elapsed_time(evs[-1][-1]) / steps
    return phases, eager_ms


def measured_traffic(workload, kernel=None):
    """HBM bytes per launch of `kernel` (or per moe_grouped_ffn call) from the
    committed PMC record, or None when the record is missing or the FFN source
    changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "ffn_traffic.json")
    try:
        rec = json.load(open(path))
        src = open(os.path.join(ROOT, rec["kernel_source"]), "rb").read()
        if hashlib.sha256(src).hexdigest() != rec.get("source_sha256"):
            return None
        w = rec["workloads"][workload]
        r = w["kernels"][kernel] if kernel else w["call"]
        return r["read"] + r["write"]
    except (OSError, ValueError, KeyError, TypeError):
        return None


# ---------------------------------------------------------------------------
# one workload
# ---------------------------------------------------------------------------
def measure(name, regime, steps, warmup, seed=0, dominant=False, eager=False):
    """Step and FFN times of one layer shape and regime (graph replays, rotated weights)."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    inp = synth.make_layer(cfg, T, seed=seed, device="cuda")
    shares = rotated_shares(cfg, inp)
    for s in shares:
        s.run()
    torch.cuda.synchronize()
    s0 = shares[0]
    out = {"T": T, "weight_copies": len(shares), "local_experts": s0.n_local}
    out["step_ms"] = time_replays([capture(s.run) for s in shares], steps, warmup)
    work = ffn_work(s0, cfg) if s0.weights is not None else None
    if work is not None:
        out.update(rows_here=work["N"], active_experts=work["active"], group_rows=work["sizes"])
        out["ffn_ms"] = time_replays([capture(ffn_call(s)) for s in shares], steps, warmup)
        if dominant:
            # the gate/up product alone: the tiled GEMM and its chunk sum (the share's
            # hint leaves out the streaming launch when every group is tiled), on the
            # packaged rows
            pshares = shares
            if s0.gather_in_ffn:
                # the same weight copies, packaged
                pshares = [LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0,
                                      s.weights.w13, s.weights.w2, shared=inp.shared,
                                      coact=cfg.coact, gather_in_ffn=False) for s in shares]
                for s in pshares:
                    s.run()
            gu = [capture(ffn_call(s, moe.MOE_FFN_GATE_UP)) for s in pshares]
            out["gate_up_ms"] = time_replays(gu, steps, warmup)
            del pshares
    if eager:
        out["phases_us"], out["eager_ms"] = eager_phases(s0, max(steps // 2, 3), warmup)
    return cfg, inp, shares, work, out


def drift_sequence(steps, seed=0):
    """Qwen1.5-MoE-shaped share over its 16-batch drift sequence: popularity re-ranked
    every 4 batches, the placement (and with it the local expert weights) swapped
    between batches.  One graph per batch; replays run the batches in order."""
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    T = cfg.T("batch")
    shares, works = [], []
    for b in range(cfg.batches):
        inp = synth.make_layer(cfg, T, seed=seed, device="cuda", batch=b)
        s = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared)
        s.run()
        shares.append(s)
    torch.cuda.synchronize()
    for s in shares:
        works.append(ffn_work(s, cfg))
    reps = max(2, steps // 8)
    step_ms = time_replays([capture(s.run) for s in shares], reps * cfg.batches, cfg.batches)
    ffn_ms = time_replays([capture(ffn_call(s)) for s in shares], reps * cfg.batches, cfg.batches)
    flops = sum(w["flops"] for w in works) / len(works)
    moved = sum(1 for a, b in zip(shares, shares[1:])
                if not np.array_equal(a.placement, b.placement))
    return {"T": T, "batches": cfg.batches, "placement_swaps": moved, "ffn_call": ffn_label(shares[0]),
            "weight_bytes_per_batch": sum(weight_bytes_of(s) for s in shares) / len(shares),
            "rows_here_mean": sum(w["N"] for w in works) / len(works),
            "step_ms": step_ms, "ffn_ms": ffn_ms,
            "tokens_per_s": T / (step_ms * 1e-3),
            "ffn": {"bound": "mfma", "achieved_TFLOPs": flops / (ffn_ms * 1e-3) / 1e12,
                    "frac": flops / (ffn_ms * 1e-3) / PEAK_BF16_FLOPS}}


def weight_bytes_of(share):
    return sum(w.numel() * w.element_size() for w in share.weights.w13 + share.weights.w2)


def shape_entry(name, regime, steps, warmup):
    if regime == "drift":
        return drift_sequence(steps)
    cfg, _, shares, work, m = measure(name, regime, steps, warmup)
    e = {"T": m["T"], "rows_here": m.get("rows_here"), "active_experts": m.get("active_experts"),
         "local_experts": m["local_experts"], "weight_copies": m["weight_copies"],
         "step_ms": m["step_ms"], "tokens_per_s": m["T"] / (m["step_ms"] * 1e-3),
         "ffn_ms": m.get("ffn_ms"), "ffn_call": ffn_label(shares[0])}
    if work is not None:
        t = m["ffn_ms"] * 1e-3
        if cfg.dtype == "f32":
            e["ffn"] = {"bound": "alu", "achieved_TFLOPs": work["flops"] / t / 1e12,
                        "frac": work["flops"] / t / PEAK_FP32_FLOPS}
        elif regime == "decode":
            e["ffn"] = {"bound": "hbm", "achieved_GBs": work["bytes"] / t / 1e9,
                        "frac": work["bytes"] / t / PEAK_HBM_BYTES}
        else:
            e["ffn"] = {"bound": "mfma", "achieved_TFLOPs": work["flops"] / t / 1e12,
                        "frac": work["flops"] / t / PEAK_BF16_FLOPS}
    del shares
    torch.cuda.synchronize()
    return e


def gathered_variant(cfg, inp, shares, steps, warmup):
    """The headline share on its other packaging path (with the row copy x_perm
    elided -- moe_permute writes the row maps only and moe_grouped_ffn_rows reads the
    token rows through row_token -- or with it, whichever the share does not use):
    step time from graph replays over the same weight copies, and whether its output
    equals the share's bit for bit."""
    gather = not shares[0].gather_in_ffn
    gs = [LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, s.weights.w13,
                     s.weights.w2, shared=inp.shared, coact=cfg.coact, gather_in_ffn=gather)
          for s in shares]
    shares[0].run()
    gs[0].run()
    torch.cuda.synchronize()
    equal = bool(torch.equal(shares[0].y, gs[0].y))
    ms = time_replays([capture(g.run) for g in gs], steps, warmup)
    what = ("row copy x_perm elided: moe_permute writes the row maps only and "
            "moe_grouped_ffn_rows reads the token rows through row_token") if gather else \
           "rows copied to x_perm by moe_permute and read from there by moe_grouped_ffn"
    return {"gather_in_ffn": gather, "ms_per_step": ms, "tokens_per_s": inp.T / (ms * 1e-3),
            "bitwise_equal_output": equal, "what": what}


# ---------------------------------------------------------------------------
# the oracle on the host
# ---------------------------------------------------------------------------
def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def _oracle_tokens_per_s(oracle, cfg, inp, S, threads=None):
    f32 = lambda t: t.detach().float().cpu().numpy()
    X = f32(inp.X)[:S]
    args = (f32(inp.Wr), f32(inp.bias), cfg.k, inp.placement, 0, [f32(w) for w in inp.w13],
            [f32(w) for w in inp.w2])
    sh = [(f32(a), f32(c)) for a, c in inp.shared]
    prev = oracle.num_threads()
    if threads:
        oracle.set_num_threads(threads)
    try:
        t0 = time.perf_counter()
        oracle.layer_share(X, *args, shared=sh, with_coact=cfg.coact)
        dt = time.perf_counter() - t0
    finally:
        if threads:
            oracle.set_num_threads(prev)
    return S / dt, dt


def cpu_baseline(cfg, inp, T_full, tiny_inp, dec_inp):
    """The oracle, as it stands, on bounded samples: the first S tokens of the headline
    batch at all host threads (S sized for about 15 s), and at one thread the whole
    tiny fp32 layer and the first tokens of the decode batch."""
    import oracle

    cores = oracle.num_threads()
    _oracle_tokens_per_s(oracle, cfg, inp, 16)              # thread pool and page-in
    rate0, t0 = _oracle_tokens_per_s(oracle, cfg, inp, 64)
    S = int(min(T_full, max(64, 64 * 15.0 / max(t0, 1e-6))))
    rate, t = _oracle_tokens_per_s(oracle, cfg, inp, S)
    out = {"value": rate, "unit": "tokens/s", "cores": cores, "kind": "oracle",
           "cpu_model": cpu_model(),
           "sample": "first %d of the %d tokens of the headline batch through the whole share "
                     "(fp64 C loops, OpenMP over %d host threads), %.1f s" % (S, T_full, cores, t)}
    single = {}
    tcfg = synth.CONFIGS["tiny_fp32"]
    reps, t1 = 0, 0.0
    while t1 < 1.0 and reps < 10000:                 # the whole layer, repeated for ~1 s
        t1 += _oracle_tokens_per_s(oracle, tcfg, tiny_inp, tiny_inp.T, threads=1)[1]
        reps += 1
    single["tiny_fp32"] = {"value": reps * tiny_inp.T / t1, "unit": "tokens/s",
                           "sample": "all %d tokens, %d times, %.2f s" % (tiny_inp.T, reps, t1)}
    S1 = min(dec_inp.T, 16)
    r, t2 = _oracle_tokens_per_s(oracle, cfg, dec_inp, S1, threads=1)
    single[cfg.name + ":decode"] = {"value": r, "unit": "tokens/s",
                                    "sample": "first %d of the %d decode tokens, %.1f s"
                                    % (S1, dec_inp.T, t2)}
    out["one_thread"] = single
    return out


# ---------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral_8x7b:prefill")
    ap.add_argument("--decode", default="decode", help="regime reported beside the headline ('' = none)")
    ap.add_argument("--shapes", default="all", choices=("all", "none"),
                    help="also measure every other configured layer shape")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gather-variant", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="first run a plain elementwise copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU's share of the layer; --gpus %d is not supported: this "
              "build runs on one GPU (how the layer would shard over GPUs is described, not built)"
              % args.gpus, file=sys.stderr)
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
    prefill = regime != "decode"

    cfg, inp, shares, work, m = measure(name, regime, args.steps, args.warmup, dominant=prefill,
                                        eager=True)
    ms = m["step_ms"]
    t_call = m["ffn_ms"] * 1e-3
    workload = "%s:%s" % (name, regime)
    call = {"kernel": ffn_label(shares[0]), "avg_launch_us": t_call * 1e6}
    if prefill:
        t_gu = m["gate_up_ms"] * 1e-3
        achieved = work["gate_up_flops"] / t_gu
        roofline = {"kernel": DOMINANT + ": the gate/up GEMM of the grouped FFN, timed as graph "
                              "replays of the gate/up product (moe_grouped_ffn_products)",
                    "bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK_BF16_FLOPS / 1e12,
                    "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_FLOPS,
                    "traffic": measured_traffic(workload, DOMINANT),
                    "traffic_unit": "bytes per launch",
                    "algorithmic_flops_per_launch": work["gate_up_flops"],
                    "avg_launch_us": t_gu * 1e6}
        call.update(bound="mfma", achieved=work["flops"] / t_call / 1e12, unit="TFLOP/s",
                    frac=work["flops"] / t_call / PEAK_BF16_FLOPS,
                    algorithmic_flops_per_call=work["flops"])
    else:
        achieved = work["bytes"] / t_call
        roofline = {"kernel": ffn_label(shares[0]), "bound": "hbm",
                    "achieved": achieved / 1e9, "peak": PEAK_HBM_BYTES / 1e9, "unit": "GB/s",
                    "frac": achieved / PEAK_HBM_BYTES, "traffic": measured_traffic(workload),
                    "traffic_unit": "bytes per launch", "algorithmic_bytes_per_launch": work["bytes"],
                    "avg_launch_us": t_call * 1e6}
    call["traffic"] = measured_traffic(workload)
    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "eager_ms_per_step": m["eager_ms"],
        "launch": "each step is one HIP graph replay of the five C-ABI calls; replays cycle "
                  "through %d copies of the local expert weights" % m["weight_copies"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": "%s-shaped MoE layer share, %s batch T=%d: d=%d, E=%d routed experts, "
                        "top-%d, SwiGLU f=%d, %d of %d experts on this GPU (G=%d), Zipf s=%s"
                        % (name, regime, T, cfg.d, cfg.E, cfg.k, cfg.f, m["local_experts"], cfg.E,
                           cfg.G, cfg.zipf),
            "T": T, "d": cfg.d, "E": cfg.E, "k": cfg.k, "f": cfg.f, "G": cfg.G,
            "local_experts": m["local_experts"], "rows_here": work["N"],
            "group_rows": work["sizes"], "seed": 0,
        },
        "roofline": roofline,
        "ffn_call": call,
        "phases_us": m["phases_us"],
    }
    if not args.no_gather_variant:
        out["gather_in_ffn"] = gathered_variant(cfg, inp, shares, args.steps, args.warmup)
    del shares
    torch.cuda.synchronize()
    dec_inp = None
    if args.decode and args.decode in dict(cfg.regimes) and args.decode != regime:
        dsteps = max(args.steps * 5, 50)
        _, dec_inp, dshares, dwork, dm = measure(name, args.decode, dsteps, args.warmup * 2,
                                                 eager=True)
        dt = dm["ffn_ms"] * 1e-3
        out["decode"] = {
            "T": dm["T"], "tokens_per_s": dm["T"] / (dm["step_ms"] * 1e-3),
            "ms_per_step": dm["step_ms"], "eager_ms_per_step": dm["eager_ms"],
            "rows_here": dwork["N"], "active_experts": dwork["active"],
            "weight_copies": dm["weight_copies"],
            "roofline": {"kernel": ffn_label(dshares[0]),
                         "bound": "hbm", "achieved": dwork["bytes"] / dt / 1e9,
                         "peak": PEAK_HBM_BYTES / 1e9, "unit": "GB/s",
                         "frac": dwork["bytes"] / dt / PEAK_HBM_BYTES,
                         "traffic": measured_traffic("%s:%s" % (name, args.decode)),
                         "traffic_unit": "bytes per launch",
                         "algorithmic_bytes_per_launch": dwork["bytes"], "avg_launch_us": dt * 1e6},
            "phases_us": dm["phases_us"],
        }
        del dshares
        torch.cuda.synchronize()
    if args.shapes == "all":
        out["shapes"] = {}
        for sname, sregime in SHAPES:
            key = "%s:%s" % (sname, sregime)
            out["shapes"][key] = shape_entry(sname, sregime, args.steps, args.warmup)
            print("[bench] %s done" % key, file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        tiny = synth.make_layer(synth.CONFIGS["tiny_fp32"], 64, seed=0, device="cuda")
        if dec_inp is None:
            dec_inp = synth.make_layer(cfg, cfg.T("decode") if "decode" in dict(cfg.regimes)
                                       else 8, seed=0, device="cuda")
        out["cpu_baseline"] = cpu_baseline(cfg, inp, T, tiny, dec_inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
