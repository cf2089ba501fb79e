"""The placement optimizer wired to the GPU layer (Sec. VI-A, Eq. 1 and Eq. 3).

Each GPU's workload row W[j] is the expert histogram the library computes for
that GPU's slice of the batch; the optimizer turns W into a placement; the same
batch, packaged by ``moe_permute`` under that placement, must then send every
GPU exactly the load Eq. 1 predicts (lambda_j), and the oracle's Eq. 3 volumes
summed over senders must agree with it.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import placement as op
from paper_2607_08782_amd import moe, placement as pl, synth
from paper_2607_08782_amd.layer import LayerShare

from parity import OUT_TOL, close, np32

pytestmark = pytest.mark.gpu


def _histograms(inp, cfg, G):
    """W[j][i]: tokens of GPU j's slice routed to expert i (route + histogram on the GPU)."""
    T = inp.X.shape[0]
    rows = []
    for j in range(G):
        Xj = inp.X[j * T // G:(j + 1) * T // G].contiguous()
        idx = torch.empty((Xj.shape[0], cfg.k), dtype=torch.int32, device="cuda")
        gate = torch.empty((Xj.shape[0], cfg.k), dtype=torch.float32, device="cuda")
        moe.moe_route_topk(Xj, inp.Wr, inp.bias, cfg.k, renorm=True, topk_idx=idx, topk_gate=gate,
                           want_logits=False)
        counts, _ = moe.moe_expert_histogram(idx, cfg.E)
        rows.append(counts.cpu().numpy())
    return np.stack(rows).astype(np.int64)


def test_optimized_placement_sends_each_gpu_its_eq1_load():
    cfg = synth.custom_config(d=256, E=16, k=4, f=128, G=4, zipf=1.2)
    G, T, C_max = 4, 512, 5
    inp = synth.make_layer(cfg, T, seed=3, device="cuda", experts="all")
    W = _histograms(inp, cfg, G)
    assert W.sum() == T * cfg.k
    f_comp = [(0.0, 20.0), (0.05, 0.0)]
    f_comm = [(1e6 / 153e9, 2.0)]
    res = pl.place(W[None], G, C_max, cfg.d * 2.0, f_comp, f_comm, seed=0)
    P = res.P[0]
    x = res.x[0]
    assert np.bincount(P, minlength=G).max() <= C_max
    lam = op.loads(W.tolist(), P.tolist(), G)                     # Eq. 1
    D = op.volumes(W.tolist(), P.tolist(), G, 1.0)               # Eq. 3 in tokens (d = 1)
    for k in range(G):
        assert lam[k] == sum(D[j][k] for j in range(G))
    for dev in range(G):
        local = [int(e) for e in np.nonzero(x[:, dev])[0]]
        share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, x, dev,
                           [inp.w13[e] for e in local], [inp.w2[e] for e in local])
        share.run()
        torch.cuda.synchronize()
        send = share.perm["send_counts"].cpu().numpy().tolist()
        assert send == [int(v) for v in lam]
        assert int(share.perm["group_offsets"][-1]) == int(lam[dev])


def _against_oracle(share, inp, cfg, P, what):
    """The share's last run against the oracle's layer on placement P, routed on the
    share's own logits: routing and row map bit for bit, y within the bf16 tolerance."""
    local = [int(e) for e in np.nonzero(P[:, share.dev])[0]]
    ref = oracle.layer_share(np32(inp.X), np32(inp.Wr), np32(inp.bias), cfg.k, P, share.dev,
                             [np32(inp.w13[e]) for e in local], [np32(inp.w2[e]) for e in local],
                             shared=[(np32(a), np32(c)) for a, c in inp.shared],
                             logits_f32=np32(share.logits))
    np.testing.assert_array_equal(share.topk_idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(share.perm["token_row"].cpu().numpy(), ref["token_row"])
    np.testing.assert_array_equal(share.perm["send_counts"].cpu().numpy(), ref["send_counts"])
    close(np32(share.y), ref["y"], OUT_TOL["bf16"], what)


@pytest.mark.parametrize("shared_f", [(), (256,)])
def test_migration_in_ffn_windows_keeps_serving_then_switches_exactly(shared_f):
    """Experts moving in are copied, chunk by chunk, into spare buffers inside the FFN
    windows of successive steps (Sec. V-B); every step during the migration gives the
    old placement's output bit for bit, and after the switch the layer gives bit for bit
    what a share built directly on the new placement gives.  The output before the
    migration and after the switch matches the oracle's layer on the old and the new
    placement.  With a shared expert of the routed width, the share runs it inside the
    routed experts' call."""
    from paper_2607_08782_amd.migration import ExpertStore, Migrator, run_step

    cfg = synth.custom_config(d=256, E=16, k=4, f=256, G=4, zipf=1.2, shared_f=shared_f)
    T = 256
    inp = synth.make_layer(cfg, T, seed=2, device="cuda", experts="all")
    P0 = np.ascontiguousarray(inp.placement, dtype=np.uint8)
    only = lambda j: [e for e in range(cfg.E) if P0[e].sum() == 1 and P0[e, j]]
    P1 = P0.copy()
    for a, b in zip(only(0)[:2], only(1)[:2]):          # two experts trade places 0 <-> 1
        P1[a, 0], P1[a, 1], P1[b, 0], P1[b, 1] = 0, 1, 1, 0
    assert P1[:, 0].sum() == P0[:, 0].sum() and not np.array_equal(P0, P1)
    store = ExpertStore(inp.w13, inp.w2)
    mig = Migrator(store, P0, 0, spare=2, chunk_bytes=32 << 10)
    w13, w2 = mig.weights()
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, P0, 0, w13, w2, shared=inp.shared)
    assert share.shared_in_ffn == bool(shared_f)
    share.run()
    torch.cuda.synchronize()
    y0 = share.y.clone()
    _against_oracle(share, inp, cfg, P0, "y before the migration")
    moved = mig.plan(P1)
    assert moved == 2 * store.nbytes(only(1)[0])
    steps = 0
    while not mig.finished:
        run_step(share, mig, budget_bytes=64 << 10)
        torch.cuda.synchronize()
        assert torch.equal(share.y, y0)
        steps += 1
    assert steps > 1 and mig.stats.bytes == moved
    w13n, w2n = mig.switch()
    share.set_placement(P1, w13n, w2n)
    share.run()
    torch.cuda.synchronize()
    _against_oracle(share, inp, cfg, P1, "y after the switch")
    local1 = [int(e) for e in np.nonzero(P1[:, 0])[0]]
    fresh = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, P1, 0, [inp.w13[e] for e in local1],
                       [inp.w2[e] for e in local1], shared=inp.shared)
    fresh.run()
    torch.cuda.synchronize()
    assert torch.equal(share.y, fresh.y)
    for e, t13, t2 in zip(local1, w13n, w2n):
        assert torch.equal(t13, inp.w13[e]) and torch.equal(t2, inp.w2[e])
