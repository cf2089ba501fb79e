"""Summaries of rocprofv3 runs of the default benchmark (`bench.py`).

The benchmark (run with --no-gather-variant) runs the prefill batch first (27
dispatches of every kernel: 3 warm-up + 10 eager timed + 3 + 10 graph replays
+ 1 final run), then the decode batch; the 28th gate-score dispatch marks the
boundary.

    # per-call HBM traffic of moe_grouped_ffn, read by bench.py for `roofline.traffic`
    python -m paper_2607_08782_amd.profsum traffic <FETCH_SIZE csv> <WRITE_SIZE csv> \
        --fetch-factor 2 --write-factor 1 --out profiles/ffn_traffic.json
    # per-kernel table: durations (kernel trace) and calibrated read / write MiB
    python -m paper_2607_08782_amd.profsum table <kernel-trace csv> <FETCH_SIZE csv> \
        <WRITE_SIZE csv> --fetch-factor 2 --write-factor 1
    # tiled-GEMM utilisation from a GRBM_GUI_ACTIVE / SQ_* counter run
    python -m paper_2607_08782_amd.profsum mfma <counter csv>
    # where one step's time goes, per kernel, for kernel traces of
    # `bench.py --workload NAME:REGIME --decode '' --no-gather-variant` runs
    python -m paper_2607_08782_amd.profsum breakdown LABEL=<kernel-trace csv> ...

The factors scale the counters to bytes: a plain copy kernel of known size
(`bench.py --calibrate-copy`) reads back FETCH_SIZE x factor = its bytes.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os

PREFILL_DISPATCHES = 27
FFN_KERNELS = ("grouped_gemm_kernel", "stream_gemm_kernel", "split_reduce_kernel")   # prefixes
FFN_SOURCE = "paper_2607_08782_amd/csrc/ffn.hip"


def short(name: str) -> str:
    return name.replace("void ", "").replace("moe::(anonymous namespace)::", "").split("(")[0]


def _mean(v):
    return sum(v) / len(v) if v else 0.0


def counter_by_regime(path: str, counter: str, factor: float):
    """Per kernel: lists of counter x factor (KiB -> bytes) for prefill and decode dispatches."""
    per, names = collections.defaultdict(float), {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            per[d] += float(r["Counter_Value"])
            names[d] = short(r["Kernel_Name"])
    gate = sorted(d for d in per if names[d].startswith("route_bf16_kernel"))
    boundary = gate[PREFILL_DISPATCHES] if len(gate) > PREFILL_DISPATCHES else max(per) + 1
    pre, dec = collections.defaultdict(list), collections.defaultdict(list)
    for d in sorted(per):
        if names[d].startswith("at::") or "rocclr" in names[d]:
            continue
        (pre if d < boundary else dec)[names[d]].append(per[d] * factor * 1024.0)
    return pre, dec


def traffic(fetch_csv, write_csv, ff, wf, out, repo="."):
    """Bytes per moe_grouped_ffn call: the streaming kernel runs twice per call."""
    with open(os.path.join(repo, FFN_SOURCE), "rb") as fh:
        sha = hashlib.sha256(fh.read()).hexdigest()
    res = {"kernel_source": FFN_SOURCE, "source_sha256": sha,
           "unit": "bytes per moe_grouped_ffn call (calibrated FETCH_SIZE + WRITE_SIZE)",
           "fetch_factor": ff, "write_factor": wf}
    for key, path, counter, fac in (("read", fetch_csv, "FETCH_SIZE", ff),
                                    ("write", write_csv, "WRITE_SIZE", wf)):
        pre, dec = counter_by_regime(path, counter, fac)
        for regime, per in (("prefill", pre), ("decode", dec)):
            tot = sum(_mean(v) * (2 if k.startswith("stream") else 1)
                      for k, v in per.items() if k.startswith(FFN_KERNELS))
            res.setdefault("mixtral_8x7b:" + regime, {})[key] = tot
    res["commands"] = [
        "rocprofv3 --pmc FETCH_SIZE --output-format csv -d gpurun_out/pf -o pf -- python -u "
        "bench.py --steps 10 --warmup 3 --no-cpu-baseline --no-gather-variant --calibrate-copy 1024",
        "rocprofv3 --pmc WRITE_SIZE --output-format csv -d gpurun_out/pw -o pw -- python -u "
        "bench.py --steps 10 --warmup 3 --no-cpu-baseline --no-gather-variant --calibrate-copy 1024"]
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    return res


def table(trace_csv, fetch_csv, write_csv, ff, wf):
    """Markdown table: per kernel, calls and mean duration per regime, mean MiB per dispatch."""
    with open(trace_csv) as fh:
        rows = sorted(csv.DictReader(fh), key=lambda r: int(r["Start_Timestamp"]))
    gate = [int(r["Start_Timestamp"]) for r in rows
            if short(r["Kernel_Name"]).startswith("route_bf16_kernel")]
    boundary = gate[PREFILL_DISPATCHES] if len(gate) > PREFILL_DISPATCHES else float("inf")
    pre_t, dec_t, order = collections.defaultdict(list), collections.defaultdict(list), []
    for r in rows:
        k = short(r["Kernel_Name"])
        if k.startswith("at::") or "rocclr" in k:
            continue
        if k not in order:
            order.append(k)
        dt = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0
        (pre_t if int(r["Start_Timestamp"]) < boundary else dec_t)[k].append(dt)
    frp, frd = counter_by_regime(fetch_csv, "FETCH_SIZE", ff)
    wrp, wrd = counter_by_regime(write_csv, "WRITE_SIZE", wf)
    mib = lambda v: _mean(v) / 2 ** 20
    lines = ["| kernel | prefill calls | prefill avg us | decode calls | decode avg us | "
             "prefill read MiB | prefill write MiB | decode read MiB | decode write MiB |",
             "|---|---|---|---|---|---|---|---|---|"]
    for k in order:
        pre, dec = pre_t.get(k, []), dec_t.get(k, [])
        lines.append("| `%s` | %d | %.1f | %d | %.1f | %.1f | %.1f | %.2f | %.2f |" % (
            k, len(pre), _mean(pre), len(dec), _mean(dec), mib(frp.get(k, [])),
            mib(wrp.get(k, [])), mib(frd.get(k, [])), mib(wrd.get(k, []))))
    return "\n".join(lines) + "\n"


def mfma(counter_csv, cus=256, simds=1024, xcds=8):
    """Median over the prefill dispatches of each tiled GEMM: duration, clock, MFMA-busy share
    of SIMD cycles, CU-busy share, MFMA flop per launch (512 flop per bf16 MOP)."""
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    meta = {}
    with open(counter_csv) as fh:
        for r in csv.DictReader(fh):
            d = int(r["Dispatch_Id"])
            per[d][r["Counter_Name"]] += float(r["Counter_Value"])
            meta[d] = (short(r["Kernel_Name"]),
                       (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    by_kernel = collections.defaultdict(list)
    for d in sorted(per):
        by_kernel[meta[d][0]].append(d)
    lines = ["| kernel | duration us | GPU clock | MFMA busy (of SIMD cycles) | CU busy | "
             "MFMA flop per launch | LDS bank conflicts |", "|---|---|---|---|---|---|---|"]
    med = lambda v: sorted(v)[len(v) // 2]
    for k, ds in by_kernel.items():
        ds = ds[:PREFILL_DISPATCHES]
        dur = [meta[d][1] for d in ds]
        clk = [per[d]["GRBM_GUI_ACTIVE"] / xcds / meta[d][1] for d in ds]
        cyc = [per[d]["GRBM_GUI_ACTIVE"] / xcds for d in ds]
        busy = [per[d]["SQ_VALU_MFMA_BUSY_CYCLES"] / (c * simds) for d, c in zip(ds, cyc)]
        cub = [per[d]["SQ_BUSY_CU_CYCLES"] / (c * cus) for d, c in zip(ds, cyc)]
        fl = [per[d]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 for d in ds]
        bc = [per[d]["SQ_LDS_BANK_CONFLICT"] for d in ds]
        lines.append("| `%s` | %.1f | %.2f GHz | %.1f %% | %.1f %% | %.4g | %.0f |" % (
            k, med(dur) * 1e6, med(clk) / 1e9, 100 * med(busy), 100 * med(cub), med(fl), med(bc)))
    return "\n".join(lines) + "\n"


def breakdown(runs, steps=PREFILL_DISPATCHES):
    """Markdown table per run: each kernel's launches per step, mean duration and
    time per step (every dispatch of a run belongs to one of its `steps` steps)."""
    lines = []
    for label, path in runs:
        with open(path) as fh:
            rows = sorted(csv.DictReader(fh), key=lambda r: int(r["Start_Timestamp"]))
        per, order = collections.defaultdict(list), []
        for r in rows:
            k = short(r["Kernel_Name"])
            if k.startswith("at::") or "rocclr" in k:
                continue
            if k not in order:
                order.append(k)
            per[k].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)
        total = sum(sum(v) for v in per.values()) / steps
        lines += ["#### %s" % label, "",
                  "| kernel | launches per step | mean us | us per step | share |",
                  "|---|---|---|---|---|"]
        for k in order:
            v = per[k]
            lines.append("| `%s` | %.2f | %.1f | %.1f | %.1f %% |" % (
                k, len(v) / steps, _mean(v), sum(v) / steps, 100 * sum(v) / steps / total))
        lines += ["| all kernels | | | %.1f | |" % total, ""]
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_csv")
    t.add_argument("write_csv")
    t.add_argument("--out", default="profiles/ffn_traffic.json")
    k = sub.add_parser("table")
    k.add_argument("trace_csv")
    k.add_argument("fetch_csv")
    k.add_argument("write_csv")
    for p in (t, k):
        p.add_argument("--fetch-factor", type=float, required=True)
        p.add_argument("--write-factor", type=float, required=True)
    u = sub.add_parser("mfma")
    u.add_argument("counter_csv")
    b = sub.add_parser("breakdown")
    b.add_argument("runs", nargs="+", help="LABEL=kernel-trace csv")
    args = ap.parse_args(argv)
    if args.cmd == "breakdown":
        print(breakdown([r.split("=", 1) for r in args.runs]), end="")
    elif args.cmd == "mfma":
        print(mfma(args.counter_csv), end="")
    elif args.cmd == "traffic":
        print(json.dumps(traffic(args.fetch_csv, args.write_csv, args.fetch_factor,
                                 args.write_factor, args.out), indent=1))
    else:
        print(table(args.trace_csv, args.fetch_csv, args.write_csv, args.fetch_factor,
                    args.write_factor), end="")


if __name__ == "__main__":
    main()
