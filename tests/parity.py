"""Shared parity machinery: run the HIP path and the oracle on the same seeded
inputs and compare step by step.

Protocol (every oracle input comes from the generator or from the oracle):
  1. gate scores: HIP logits vs oracle logits (float64), max-abs error within
     LOGIT_TOL * max|ref|;
  2. routing: the oracle's logits, rounded to fp32, are handed to both sides
     (the HIP side through MOE_LOGITS_IN); top-k indices, counts,
     co-activation, group offsets, row maps and send counts must match bit for
     bit, gates within GATE_TOL;
  3. expert FFN and weighted sum on that routing: within OUT_TOL * max|ref|
     (all rows at small sizes; at full sizes every row of each group's first
     and last 256-row tile, and the tokens whose rows all lie there).
The path the benchmark times (gate scores and top-k computed by the library,
no logits handed in) is checked by `check_timed_path`: the HIP logits within
LOGIT_TOL of the oracle's, then the oracle's steps 2-8 run on the HIP logits
must give the HIP selection bit for bit, gates within GATE_TOL, and the
outputs within OUT_TOL.
"""
from __future__ import annotations

import sys
from typing import Optional

import numpy as np
import torch

import oracle
from paper_2607_08782_amd import synth
from paper_2607_08782_amd.layer import LayerShare

LOGIT_TOL = {"bf16": 1e-4, "f32": 1e-5}
OUT_TOL = {"bf16": 2e-2, "f32": 1e-5}
GATE_TOL = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def np32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def close(got, ref, rel: float, what: str):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = float(np.max(np.abs(ref)))
    err = float(np.max(np.abs(got - ref)))
    assert err <= rel * scale + 1e-30, "%s: max-abs err %.3e > %.1e * max|ref| %.3e" % (
        what, err, rel, scale)
    return err / max(scale, 1e-30)


class Case:
    """One layer share on the GPU plus its CPU copies for the oracle."""

    def __init__(self, cfg: synth.LayerConfig, T: int, seed: int = 0, batch: int = 0,
                 dev: int = 0, gather_in_ffn=None):
        self.cfg = cfg
        self.T = T
        self.inp = synth.make_layer(cfg, T, seed=seed, device="cuda", batch=batch, dev=dev)
        i = self.inp
        self.share = LayerShare(i.X, i.Wr, i.bias, cfg.k, i.placement, dev, i.w13, i.w2,
                                shared=i.shared, renorm=True, coact=cfg.coact,
                                gather_in_ffn=gather_in_ffn)
        self.X = np32(i.X)
        self.Wr = np32(i.Wr)
        self.b = np32(i.bias)
        self._w = {}

    def weights(self, s: int):
        if s not in self._w:
            self._w[s] = (np32(self.inp.w13[s]), np32(self.inp.w2[s]))
        return self._w[s]

    def shared_np(self):
        return [(np32(a), np32(c)) for a, c in self.inp.shared]


def check_logits(case: Case):
    """Step 1: HIP gate scores vs the oracle's."""
    case.share.route()
    torch.cuda.synchronize()
    ref = oracle.router_logits(case.X, case.Wr, case.b)
    rel = close(np32(case.share.logits), ref, LOGIT_TOL[case.cfg.dtype], "logits")
    return ref, rel


def check_routing(case: Case, ref_logits: np.ndarray):
    """Step 2: same fp32 logits on both sides; integer outputs bit-exact."""
    L32 = ref_logits.astype(np.float32)
    case.share.run(logits_in=torch.from_numpy(L32).cuda())
    torch.cuda.synchronize()
    return check_routing_outputs(case, L32)


def check_routing_outputs(case: Case, L32: np.ndarray):
    """The share has run on fp32 logits L32: top-k, counts, co-activation and the
    packaging must be the oracle's on L32 bit for bit, gates within GATE_TOL."""
    cfg, share = case.cfg, case.share
    idx, gate = oracle.topk(L32, cfg.k, renorm=True)
    np.testing.assert_array_equal(share.topk_idx.cpu().numpy(), idx)
    close(np32(share.topk_gate), gate, GATE_TOL, "gates")       # gates <= 1: absolute check
    counts, coact = oracle.histogram(idx, cfg.E, cfg.coact)
    np.testing.assert_array_equal(share.counts.cpu().numpy(), counts)
    if cfg.coact:
        np.testing.assert_array_equal(share.coact.cpu().numpy(), coact)
    pm = oracle.permute(case.X, idx, gate, cfg.E, case.inp.placement, share.dev)
    N = pm["rows"]
    got = {k: v.cpu().numpy() for k, v in share.perm.items()
           if v is not None and k != "x_perm"}
    np.testing.assert_array_equal(got["group_offsets"], pm["group_offsets"])
    np.testing.assert_array_equal(got["row_token"][:N], pm["row_token"])
    np.testing.assert_array_equal(got["token_row"], pm["token_row"])
    np.testing.assert_array_equal(got["send_counts"], pm["send_counts"])
    close(got["row_gate"][:N], pm["row_gate"], GATE_TOL, "row_gate")
    if share.perm["x_perm"] is not None:
        np.testing.assert_array_equal(np32(share.perm["x_perm"][:N]), pm["x_perm"])
    return idx, gate, pm


def check_timed_path(case: Case):
    """The share as the benchmark runs it: `share.run()` with the library's own
    gate scores and top-k (the fused score + top-k kernels, the fp32 path, the
    tiled or split-K score kernels, whichever the shape takes).  The logits must
    be within LOGIT_TOL of the oracle's; the oracle's routing and packaging of
    those fp32 logits must equal the HIP outputs bit for bit.  Returns the
    routing for `check_ffn_and_combine` (the share's y is that of this run)."""
    share = case.share
    share.run()
    torch.cuda.synchronize()
    ref = oracle.router_logits(case.X, case.Wr, case.b)
    gl = np32(share.logits)
    close(gl, ref, LOGIT_TOL[case.cfg.dtype], "logits")
    return check_routing_outputs(case, gl)


TILE_ROWS = 256       # rows of the grouped GEMM's macro tile


def _sample_rows(lo: int, hi: int, n, rng) -> np.ndarray:
    """Rows of one group to check: all (None), the first and last TILE_ROWS-row
    tile ("tiles"), or n sampled rows including both ends."""
    if hi <= lo:
        return np.zeros(0, np.int64)
    if n is None:
        return np.arange(lo, hi)
    if n == "tiles":
        last = lo + ((hi - lo - 1) // TILE_ROWS) * TILE_ROWS
        return np.unique(np.concatenate([np.arange(lo, min(lo + TILE_ROWS, hi)),
                                         np.arange(last, hi)]))
    if hi - lo <= n:
        return np.arange(lo, hi)
    mid = rng.choice(np.arange(lo + 1, hi - 1), size=max(n - 2, 0), replace=False)
    return np.unique(np.concatenate([[lo, hi - 1], mid]))


def check_ffn_and_combine(case: Case, idx, gate, pm, sample=None, seed: int = 0,
                          max_tokens: int = 512):
    """Step 3: expert FFN rows and combined outputs.  sample=None: every row and
    token; "tiles": every row of each group's first and last 256-row tile, and
    up to max_tokens of the tokens whose local rows all lie in those tiles (plus
    the first tokens that have no local row); an int: that many rows per group
    and tokens."""
    cfg, share = case.cfg, case.share
    tol = OUT_TOL[cfg.dtype]
    rng = np.random.default_rng(seed)
    go = pm["group_offsets"]
    worst = 0.0
    ref_rows = {}
    for s in range(len(go) - 1):
        rows = _sample_rows(int(go[s]), int(go[s + 1]), sample, rng)
        if not len(rows):
            continue
        w13, w2 = case.weights(s)
        ref = oracle.expert_ffn(pm["x_perm"][rows], w13, w2)
        if not share.fused_combine:          # a fused call combines without writing y_perm
            worst = max(worst, close(np32(share.y_perm[torch.from_numpy(rows).cuda()]), ref, tol,
                                     "y_perm group %d" % s))
        for p, v in zip(rows.tolist(), ref):
            ref_rows[p] = v
    tr = pm["token_row"]
    if sample == "tiles":
        have = np.zeros(max(pm["rows"], 1), bool)
        have[list(ref_rows)] = True
        ok = np.all((tr < 0) | have[np.maximum(tr, 0)], axis=1)
        with_rows = np.nonzero(ok & np.any(tr >= 0, axis=1))[0]
        without = np.nonzero(np.all(tr < 0, axis=1))[0][:16]
        if len(with_rows) > max_tokens:
            with_rows = np.sort(rng.choice(with_rows, size=max_tokens, replace=False))
        toks = np.unique(np.concatenate([with_rows, without])).astype(np.int64)
    else:
        toks = _sample_rows(0, case.T, sample, rng)
    if not len(toks):
        return worst
    xs = case.X[toks]
    ref_y = np.zeros((len(toks), cfg.d))
    shared = case.shared_np()
    for (a, c) in shared:
        ref_y += oracle.expert_ffn(xs, a, c)
    if shared:
        close(share.shared_output()[torch.from_numpy(toks).cuda()].cpu().numpy(), ref_y, tol,
              "shared experts' output")
    local = oracle.local_slots(case.inp.placement, share.dev)
    slot = {e: s for s, e in enumerate(local)}
    for n, t in enumerate(toks):
        for r in range(cfg.k):
            p = int(tr[t, r])
            if p < 0:
                continue
            if p not in ref_rows:
                w13, w2 = case.weights(slot[int(idx[t, r])])
                ref_rows[p] = oracle.expert_ffn(case.X[t:t + 1], w13, w2)[0]
            ref_y[n] += gate[t, r] * ref_rows[p]
    worst = max(worst, close(np32(share.y[torch.from_numpy(toks).cuda()]), ref_y, tol, "y"))
    return worst


def check_end_to_end_routing(case: Case, ref_logits: np.ndarray):
    """HIP logits -> HIP top-k.  Where the oracle's k-th/(k+1)-th margin is wider
    than the logit tolerance the selection is unique and must match; elsewhere
    the HIP selection must be a valid top-k of its own logits.  Returns the
    fraction of tokens whose selected set differs from the oracle's."""
    cfg, share = case.cfg, case.share
    share.route()
    torch.cuda.synchronize()
    gl = np32(share.logits)
    gidx = share.topk_idx.cpu().numpy()
    oidx, _ = oracle.topk(ref_logits.astype(np.float32), cfg.k)
    srt = np.sort(ref_logits, axis=1)[:, ::-1]
    tol = LOGIT_TOL[cfg.dtype] * float(np.max(np.abs(ref_logits)))
    if cfg.k < cfg.E:
        margin = srt[:, cfg.k - 1] - srt[:, cfg.k]
        safe = margin > 4 * tol
    else:
        safe = np.ones(case.T, bool)
    np.testing.assert_array_equal(np.sort(gidx[safe], 1), np.sort(oidx[safe], 1))
    # validity of every HIP selection against its own logits (descending, ties to lower index)
    sel = np.take_along_axis(gl, gidx.astype(np.int64), 1)
    assert np.all(np.diff(sel, axis=1) <= 0)
    if cfg.k < cfg.E:
        rest = gl.copy()
        np.put_along_axis(rest, gidx.astype(np.int64), -np.inf, 1)
        assert np.all(sel[:, -1] >= rest.max(1))
    differ = np.any(np.sort(gidx, 1) != np.sort(oidx, 1), axis=1)
    return float(differ.mean())
