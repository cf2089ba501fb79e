"""A fixed number of layer-share steps of one workload, for kernel traces.

Builds the share of NAME:REGIME as the benchmark does (synthetic seed 0, the
benchmark placement, replays cycling through enough copies of the local expert
weights to touch at least 1 GB), captures one step per copy as a HIP graph,
replays them --warmup times, then launches a marker kernel (torch.neg on a
one-element tensor) and replays exactly --steps steps.  Every dispatch after the
marker belongs to those steps, which `profsum breakdown` relies on:

    rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/bd_TAG -o kt -- \\
        python -u -m paper_2607_08782_amd.layer_trace --workload NAME:REGIME --steps 20
    python -m paper_2607_08782_amd.profsum breakdown --steps 20 TAG=gpurun_out/bd_TAG/kt_kernel_trace.csv
"""
from __future__ import annotations

import argparse
import math

import torch

from . import synth
from .layer import LayerShare


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", required=True, help="NAME:REGIME")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the trace runs on the GPU; no GPU is visible")
    name, regime = args.workload.split(":")
    cfg = synth.CONFIGS[name]
    inp = synth.make_layer(cfg, cfg.T(regime), seed=0, device="cuda")
    wbytes = sum(w.numel() * w.element_size() for w in inp.w13 + inp.w2)
    copies = 1 if wbytes >= 1e9 else int(math.ceil(1e9 / max(wbytes, 1)))
    shares = []
    for c in range(copies):
        w13 = inp.w13 if c == 0 else [w.clone() for w in inp.w13]
        w2 = inp.w2 if c == 0 else [w.clone() for w in inp.w2]
        shares.append(LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, w13, w2,
                                 shared=inp.shared, coact=cfg.coact))
    for s in shares:
        s.run()
    torch.cuda.synchronize()
    graphs = []
    for s in shares:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            s.run()
        graphs.append(g)
    for i in range(args.warmup):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    torch.neg(torch.ones(1, device="cuda"))          # marker: the steps start after it
    for i in range(args.steps):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    print("%s: %d steps traced (%d weight copies)" % (args.workload, args.steps, copies), flush=True)


if __name__ == "__main__":
    main()
