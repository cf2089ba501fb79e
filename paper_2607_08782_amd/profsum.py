"""Summaries of rocprofv3 runs of `bench.py`, one workload per run.

Each profiled run measures one layer shape and regime alone
(`bench.py --workload NAME:REGIME --decode '' --shapes none --no-cpu-baseline
--no-gather-variant`), so every dispatch in its trace belongs to that workload.

    # per-kernel launch counts and mean durations (kernel trace)
    python -m paper_2607_08782_amd.profsum kernels <kernel_trace.csv>
    # HBM traffic per launch of each FFN kernel and per moe_grouped_ffn call, from a
    # FETCH_SIZE run and a WRITE_SIZE run of the same command with --calibrate-copy;
    # merged into profiles/ffn_traffic.json under the workload's name
    python -m paper_2607_08782_amd.profsum traffic NAME:REGIME <FETCH csv> <WRITE csv>
    # tiled-GEMM utilisation from a GRBM_GUI_ACTIVE / SQ_* counter run
    python -m paper_2607_08782_amd.profsum mfma <counter csv>
    # where one step's time goes, per kernel (kernel traces of layer_trace runs)
    python -m paper_2607_08782_amd.profsum breakdown --steps N LABEL=<kernel_trace.csv> ...

Counter calibration: the run's first kernel is a plain elementwise copy of
--calibrate-copy MiB (torch.neg: reads and writes that many bytes); the factors
that turn its FETCH_SIZE and WRITE_SIZE (KiB) into those bytes scale every other
dispatch's counters.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os

FFN_SOURCE = "paper_2607_08782_amd/csrc/ffn.hip"
# kernels of one routed-expert FFN call and their launches per call (the streaming
# kernel runs once per product; moe_grouped_ffn_combine ends with the combining
# chunk sum in place of split_reduce_kernel<false>)
FFN_CALL = {"grouped_gemm_kernel<true, false>": 1, "grouped_gemm_kernel<false, false>": 1,
            "stream_gemm_kernel<false>": 2, "split_reduce_kernel<true>": 1,
            "split_reduce_kernel<false>": 1}
FFN_CALL_PREFIX = {"stream_reduce_combine_kernel<": 1}


def per_call(kernel):
    """Launches of `kernel` in one routed-expert FFN call (0: not one of its kernels)."""
    if kernel in FFN_CALL:
        return FFN_CALL[kernel]
    return next((n for p, n in FFN_CALL_PREFIX.items() if kernel.startswith(p)), 0)
COPY_KERNEL = "neg_kernel"     # torch.neg's elementwise kernel carries this in its name


def short(name: str) -> str:
    return name.replace("void ", "").replace("moe::(anonymous namespace)::", "").split("(")[0]


def _mean(v):
    return sum(v) / len(v) if v else 0.0


def _med(v):
    return sorted(v)[len(v) // 2] if v else 0.0


def kernels(trace_csv):
    """Markdown table: each library kernel's launches and mean / median duration."""
    with open(trace_csv) as fh:
        rows = sorted(csv.DictReader(fh), key=lambda r: int(r["Start_Timestamp"]))
    per, order = collections.defaultdict(list), []
    for r in rows:
        k = short(r["Kernel_Name"])
        if k.startswith("at::") or "rocclr" in k:
            continue
        if k not in order:
            order.append(k)
        per[k].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)
    lines = ["| kernel | launches | mean us | median us |", "|---|---|---|---|"]
    for k in order:
        lines.append("| `%s` | %d | %.1f | %.1f |" % (k, len(per[k]), _mean(per[k]), _med(per[k])))
    return "\n".join(lines) + "\n"


def _counter(path, counter):
    """Per dispatch: (kernel name, counter value in KiB summed over its instances)."""
    per, names = collections.defaultdict(float), {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            per[d] += float(r["Counter_Value"])
            names[d] = r["Kernel_Name"]
    return [(names[d], per[d]) for d in sorted(per)]


def traffic(workload, fetch_csv, write_csv, copy_mib, out, repo="."):
    """Bytes per launch of each FFN kernel and per call, scaled by the copy kernel."""
    res = {}
    if os.path.exists(out):
        with open(out) as fh:
            res = json.load(fh)
    with open(os.path.join(repo, FFN_SOURCE), "rb") as fh:
        sha = hashlib.sha256(fh.read()).hexdigest()
    if res.get("source_sha256") != sha:
        res = {"workloads": {}}
    res.update({"kernel_source": FFN_SOURCE, "source_sha256": sha,
                "unit": "bytes per launch (FETCH_SIZE and WRITE_SIZE, KiB, times the factor a "
                        "plain copy of known size gives)"})
    w = {"kernels": {}, "call": {"read": 0.0, "write": 0.0}}
    copy_bytes = copy_mib * float(1 << 20)
    for key, path, counter in (("read", fetch_csv, "FETCH_SIZE"), ("write", write_csv, "WRITE_SIZE")):
        disp = _counter(path, counter)
        copies = [v for n, v in disp if COPY_KERNEL in n]
        if not copies:
            raise SystemExit("no calibration copy kernel in %s (run with --calibrate-copy)" % path)
        factor = copy_bytes / (copies[-1] * 1024.0)
        w[key + "_factor"] = factor
        per = collections.defaultdict(list)
        for n, v in disp:
            per[short(n)].append(v * 1024.0 * factor)
        for k, v in per.items():
            if per_call(k):
                w["kernels"].setdefault(k, {})[key] = _mean(v)
                w["call"][key] += _mean(v) * per_call(k)
    res["workloads"][workload] = w
    res.setdefault("commands", {})[workload] = [
        "rocprofv3 --pmc %s --output-format csv -d gpurun_out/pmc -o %s -- python -u bench.py "
        "--workload %s --decode '' --shapes none --steps 10 --warmup 3 --no-cpu-baseline "
        "--no-gather-variant --calibrate-copy %d" % (c, c.lower(), workload, copy_mib)
        for c in ("FETCH_SIZE", "WRITE_SIZE")]
    with open(out, "w") as fh:
        json.dump(res, fh, indent=1)
    return res


def mfma(counter_csv, cus=256, simds=1024, xcds=8):
    """Median over the dispatches of each tiled GEMM: duration, clock, MFMA-busy share
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
        if meta[d][0].startswith("grouped_gemm_kernel"):
            by_kernel[meta[d][0]].append(d)
    lines = ["| kernel | duration us | GPU clock | MFMA busy (of SIMD cycles) | CU busy | "
             "MFMA flop per launch | LDS bank conflicts |", "|---|---|---|---|---|---|---|"]
    for k, ds in by_kernel.items():
        dur = [meta[d][1] for d in ds]
        cyc = [per[d]["GRBM_GUI_ACTIVE"] / xcds for d in ds]
        clk = [c / meta[d][1] for d, c in zip(ds, cyc)]
        busy = [per[d]["SQ_VALU_MFMA_BUSY_CYCLES"] / (c * simds) for d, c in zip(ds, cyc)]
        cub = [per[d]["SQ_BUSY_CU_CYCLES"] / (c * cus) for d, c in zip(ds, cyc)]
        fl = [per[d]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 for d in ds]
        bc = [per[d]["SQ_LDS_BANK_CONFLICT"] for d in ds]
        lines.append("| `%s` | %.1f | %.2f GHz | %.1f %% | %.1f %% | %.4g | %.0f |" % (
            k, _med(dur) * 1e6, _med(clk) / 1e9, 100 * _med(busy), 100 * _med(cub), _med(fl),
            _med(bc)))
    return "\n".join(lines) + "\n"


def breakdown(runs, steps):
    """Markdown table per run: each kernel's launches per step, mean duration and
    time per step.  The dispatches counted are those after the last marker kernel
    (layer_trace launches one right before its `steps` steps), else all of them."""
    lines = []
    for label, path in runs:
        with open(path) as fh:
            rows = sorted(csv.DictReader(fh), key=lambda r: int(r["Start_Timestamp"]))
        marks = [i for i, r in enumerate(rows) if COPY_KERNEL in r["Kernel_Name"]]
        if marks:
            rows = rows[marks[-1] + 1:]
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
    k = sub.add_parser("kernels")
    k.add_argument("trace_csv")
    t = sub.add_parser("traffic")
    t.add_argument("workload")
    t.add_argument("fetch_csv")
    t.add_argument("write_csv")
    t.add_argument("--copy-mib", type=int, default=1024)
    t.add_argument("--out", default="profiles/ffn_traffic.json")
    u = sub.add_parser("mfma")
    u.add_argument("counter_csv")
    b = sub.add_parser("breakdown")
    b.add_argument("--steps", type=int, required=True)
    b.add_argument("runs", nargs="+", help="LABEL=kernel-trace csv")
    args = ap.parse_args(argv)
    if args.cmd == "kernels":
        print(kernels(args.trace_csv), end="")
    elif args.cmd == "breakdown":
        print(breakdown([r.split("=", 1) for r in args.runs], args.steps), end="")
    elif args.cmd == "mfma":
        print(mfma(args.counter_csv), end="")
    else:
        print(json.dumps(traffic(args.workload, args.fetch_csv, args.write_csv, args.copy_mib,
                                 args.out), indent=1))


if __name__ == "__main__":
    main()
