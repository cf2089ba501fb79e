"""HIP path vs the CPU oracle, on the GPU (marked `gpu`).

Small shapes check every output element and span several tiles with ragged
tails; the model-shaped layer shares check routing bit for bit at full size
and the FFN / combined outputs on every row of each group's first and last
256-row tile (all rows at decode sizes) and the tokens those rows serve.
Every shape is checked twice: with the oracle's logits handed in, and on the
path the benchmark times (the library's own gate scores and top-k), where the
oracle's routing of the HIP logits must equal the HIP routing bit for bit.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2607_08782_amd import moe, synth
from paper_2607_08782_amd.layer import LayerShare

from parity import (Case, check_end_to_end_routing, check_ffn_and_combine, check_logits,
                    check_routing, check_timed_path, close, np32, say, GATE_TOL, OUT_TOL)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    moe.load_library()          # fails loudly if the HIP library is not built
    yield


SMALL = {
    "tiny_fp32": (synth.CONFIGS["tiny_fp32"], 64),
    "bf16_ragged_replicas": (synth.custom_config(d=256, E=16, k=4, f=384, G=3, replicas=2,
                                                 zipf=1.2), 300),
    "bf16_two_shared": (synth.custom_config(d=128, E=12, k=3, f=192, shared_f=(128, 64), G=2,
                                            replicas=1, zipf=1.0), 200),
    "bf16_k1": (synth.custom_config(d=64, E=8, k=1, f=64, G=1), 130),
    "bf16_k_eq_E": (synth.custom_config(d=64, E=8, k=8, f=128, G=2), 70),
    "bf16_E128_coact": (synth.custom_config(d=128, E=128, k=8, f=64, G=9, replicas=2, zipf=1.5,
                                            coact=True), 257),
    "bf16_T1": (synth.custom_config(d=128, E=8, k=2, f=128, G=2), 1),
    "fp32_ragged": (synth.custom_config(dtype="f32", d=72, E=6, k=2, f=40, shared_f=(24,), G=2,
                                        replicas=1, zipf=1.0), 77),
    "bf16_k16_max": (synth.custom_config(d=128, E=64, k=16, f=64, G=3, replicas=2, zipf=1.1,
                                         coact=True), 150),
    "bf16_k12": (synth.custom_config(d=64, E=40, k=12, f=64, shared_f=(64,), G=2, replicas=1,
                                     zipf=1.0), 300),
    # the largest expert count, k and local group count the boundary takes (MOE_MAX_E = 256,
    # MOE_MAX_K = 16, 128 local slots = MOE_MAX_GROUPS), co-activation past the LDS bins
    "bf16_E256_k16_128_groups": (synth.custom_config(d=128, E=256, k=16, f=64, G=2, zipf=1.1,
                                                     coact=True), 300),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_shapes_every_element(name):
    cfg, T = SMALL[name]
    say("[case]", name, cfg, "T=%d" % T)
    case = Case(cfg, T)
    ref_logits, _ = check_logits(case)
    idx, gate, pm = check_routing(case, ref_logits)
    check_ffn_and_combine(case, idx, gate, pm, sample=None)
    check_end_to_end_routing(case, ref_logits)
    idx, gate, pm = check_timed_path(case)
    check_ffn_and_combine(case, idx, gate, pm, sample=None)


FULL = [
    ("mixtral_8x7b", "prefill"), ("mixtral_8x7b", "decode"),
    ("deepseek_v2_lite", "prefill"), ("deepseek_v2_lite", "decode"),
    ("qwen15_moe_a27b", "batch"),
    ("qwen3_30b_a3b", "decode"), ("qwen3_30b_a3b", "prefill"),
]


@pytest.mark.parametrize("name,regime", FULL)
def test_model_shaped_layer_share(name, regime):
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[case]", name, regime, "T=%d" % T)
    case = Case(cfg, T)
    ref_logits, _ = check_logits(case)
    idx, gate, pm = check_routing(case, ref_logits)
    say("  rows here", pm["rows"], "send_counts", pm["send_counts"].tolist())
    worst = check_ffn_and_combine(case, idx, gate, pm, sample="tiles")
    differ = check_end_to_end_routing(case, ref_logits)
    say("  worst rel err %.2e, top-k sets differing from the oracle: %.4f" % (worst, differ))


TIMED = [("tiny_fp32", "batch")] + FULL


@pytest.mark.parametrize("name,regime", TIMED)
def test_timed_path_matches_the_oracle(name, regime):
    """The share exactly as the benchmark runs it (share.run(): the library's own
    gate scores and top-k, e.g. the fused score + top-k epilogue at the Mixtral and
    DeepSeek-V2-Lite prefill shapes, the fp32 path of the tiny layer, the tiled
    score kernel at Qwen3 prefill, split-K partials at decode sizes).  The oracle
    routes and packages the HIP logits: indices, counts, co-activation and every
    row map bit for bit, gates within 1e-5; then its expert FFN and combine on
    that routing give y_perm and y within the output tolerance (every row of each
    group's first and last 256-row tile, all rows at decode sizes)."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[timed]", name, regime, "T=%d" % T)
    case = Case(cfg, T)
    idx, gate, pm = check_timed_path(case)
    worst = check_ffn_and_combine(case, idx, gate, pm, sample=None if T <= 256 else "tiles")
    say("  rows here", pm["rows"], "worst rel err %.2e" % worst)


def test_replica_split_hand_example():
    """The hand-evaluated replica split (tests/golden): expert 0 on three GPUs takes
    blocks of 2, 2 and 3 of its 7 tokens, expert 2 on two GPUs 2 and 2; every GPU's
    group offsets, row maps and send counts as written out by hand."""
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "replica_split_hand_example.json")))
    E, G, k = fx["E"], fx["G"], fx["k"]
    idx = np.array(fx["idx"], np.int32)
    T = idx.shape[0]
    L = np.zeros((T, E), np.float32)
    for t in range(T):
        L[t, idx[t, 0]] = 2.0
        L[t, idx[t, 1]] = 1.0
    cfg = synth.custom_config(d=64, E=E, k=k, f=64, G=G)
    pl = np.array(fx["placement"], np.uint8)
    for g in fx["per_gpu"]:
        inp, share = _share(cfg, T, placement=pl, dev=g["dev"])
        share.run(logits_in=torch.from_numpy(L).cuda())
        torch.cuda.synchronize()
        np.testing.assert_array_equal(share.topk_idx.cpu().numpy(), idx)
        N = g["group_offsets"][-1]
        np.testing.assert_array_equal(share.perm["group_offsets"].cpu().numpy(), g["group_offsets"])
        np.testing.assert_array_equal(share.perm["row_token"][:N].cpu().numpy(), g["row_token"])
        np.testing.assert_array_equal(share.perm["token_row"].cpu().numpy(), g["token_row"])
        np.testing.assert_array_equal(share.perm["send_counts"].cpu().numpy(), fx["send_counts"])
        np.testing.assert_array_equal(np32(share.perm["x_perm"][:N]),
                                      np32(inp.X)[g["row_token"]])


TILED = [  # (T, d, E, k): batches of >= 192 64-token tiles over > 32 experts take the tiled kernel
    (12225, 128, 33, 2),      # the smallest batch and width that take it; one K stage
    (12290, 256, 96, 8),      # two 32-expert tiles per wave
    (12300, 256, 130, 5),     # four (E > 128)
]


@pytest.mark.parametrize("T,d,E,k", TILED)
def test_tiled_gate_scores_and_topk_every_element(T, d, E, k):
    cfg = synth.custom_config(d=d, E=E, k=k, f=64, G=1)
    say("[tiled]", T, d, E, k)
    case = Case(cfg, T)
    check_logits(case)
    gl = np32(case.share.logits)
    oidx, og = oracle.topk(gl, k)
    np.testing.assert_array_equal(case.share.topk_idx.cpu().numpy(), oidx)
    close(np32(case.share.topk_gate), og, GATE_TOL, "gates")


SHORT = [  # (T, d, E, k): short batches over > 16 experts take the per-wave split-K score tiles
    (1, 2048, 128, 8),        # one token: 8 expert tiles x 32 K chunks
    (17, 512, 20, 3),         # ragged token and expert tiles (2 x 2), 8 chunks of 2 steps
    (64, 2048, 128, 8),       # Qwen3-30B-A3B-shaped decode
    (256, 2048, 64, 6),       # DeepSeek-V2-Lite-shaped decode, 16 chunks
    (100, 1024, 160, 4),      # E > 128 (ten expert tiles)
    (33, 160, 48, 2),         # K of five 32-wide steps in two uneven chunks
]


@pytest.mark.parametrize("T,d,E,k", SHORT)
def test_short_batch_gate_scores_and_topk_every_element(T, d, E, k):
    """Scores of short batches as per-wave 16 x 16 partial tiles over K chunks, summed
    in chunk order by the top-k launch: every logit against the oracle's, and the
    selection and gates exact given those logits."""
    cfg = synth.custom_config(d=d, E=E, k=k, f=64, G=1)
    say("[short]", T, d, E, k)
    case = Case(cfg, T)
    check_logits(case)
    gl = np32(case.share.logits)
    oidx, og = oracle.topk(gl, k)
    np.testing.assert_array_equal(case.share.topk_idx.cpu().numpy(), oidx)
    close(np32(case.share.topk_gate), og, GATE_TOL, "gates")


def test_drift_sequence_swaps_placement_without_reallocating():
    """Qwen1.5-MoE-shaped share: popularity re-ranked every 4 batches, placement
    swapped between batches by re-pointing the weight table."""
    cfg = synth.CONFIGS["qwen15_moe_a27b"]
    T = cfg.T("batch")
    base = Case(cfg, T, batch=0)
    share = base.share
    bufs = lambda: [t.data_ptr() for t in (share.y_perm, share.perm["row_token"], share.ws_ffn,
                                           share.y)]
    ptr_before = bufs()
    for b in (0, 3, 4, 9, 15):
        say("[case] drift batch", b)
        inp = synth.make_layer(cfg, T, seed=0, device="cuda", batch=b)
        share.set_inputs(inp.X, inp.bias)
        share.set_placement(inp.placement, inp.w13, inp.w2)
        case = Case.__new__(Case)
        case.cfg, case.T, case.inp, case.share = cfg, T, inp, share
        case.X, case.Wr, case.b, case._w = np32(inp.X), np32(inp.Wr), np32(inp.bias), {}
        ref_logits, _ = check_logits(case)
        idx, gate, pm = check_routing(case, ref_logits)
        check_ffn_and_combine(case, idx, gate, pm, sample="tiles", seed=b, max_tokens=128)
        idx, gate, pm = check_timed_path(case)
        check_ffn_and_combine(case, idx, gate, pm, sample="tiles", seed=b, max_tokens=128)
    assert bufs() == ptr_before


def _share(cfg, T, logits=None, placement=None, dev=0):
    inp = synth.make_layer(cfg, T, seed=1, device="cuda")
    pl = inp.placement if placement is None else placement
    local = [int(e) for e in np.nonzero(pl[:, dev])[0]]
    ws = [synth.expert_weights(cfg, e, 1, "cuda") for e in local]
    # the packaging checks read the row copy x_perm, so the share keeps it
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, pl, dev, [a for a, _ in ws],
                       [b for _, b in ws], shared=inp.shared, fuse_combine=False,
                       gather_in_ffn=False)
    return inp, share


def test_empty_batch():
    cfg = synth.custom_config(d=64, E=8, k=2, f=64, G=2)
    inp, share = _share(cfg, 0)
    share.run()
    torch.cuda.synchronize()
    assert share.perm["group_offsets"].cpu().numpy().tolist() == [0] * (share.n_local + 1)
    assert share.perm["send_counts"].cpu().numpy().tolist() == [0, 0]
    assert share.counts.cpu().numpy().tolist() == [0] * 8


def test_ties_all_equal_and_signed_zero_logits():
    cfg = synth.custom_config(d=64, E=8, k=3, f=64, G=1)
    T = 70
    inp, share = _share(cfg, T)
    L = np.full((T, 8), 0.75, np.float32)
    L[1] = [0.0, -0.0, 0.0, -0.0, -1.0, 0.0, -0.0, -2.0]
    L[2] = [-0.0, 1.0, -0.0, 1.0, 0.0, 1.0, 0.0, 3.0]
    share.run(logits_in=torch.from_numpy(L).cuda())
    torch.cuda.synchronize()
    gidx = share.topk_idx.cpu().numpy()
    assert gidx[0].tolist() == [0, 1, 2] and gidx[5].tolist() == [0, 1, 2]
    assert gidx[1].tolist() == [0, 1, 2]
    assert gidx[2].tolist() == [7, 1, 3]
    oidx, og = oracle.topk(L, 3)
    np.testing.assert_array_equal(gidx, oidx)
    close(np32(share.topk_gate), og, 1e-5, "gates")


@pytest.mark.parametrize("E", [1, 3, 8, 16, 17, 60, 64, 65, 128, 129, 200, 256])
@pytest.mark.parametrize("renorm", [True, False])
def test_topk_of_given_scores_with_ties_every_width(E, renorm):
    """Top-k over handed-in scores: few distinct levels (many ties), signed zeros,
    a ragged token count; indices bit-exact, gates within 1e-5."""
    T = 100
    rng = np.random.default_rng(E * 2 + renorm)
    L = (rng.integers(-3, 4, size=(T, E)) * 0.5).astype(np.float32)
    z = L == 0
    L[z] = np.where(rng.random(int(z.sum())) < 0.5, np.float32(-0.0), np.float32(0.0))
    L[: T // 2] += rng.standard_normal((T // 2, E)).astype(np.float32)
    Lg = torch.from_numpy(L).cuda()
    for k in sorted({1, min(2, E), min(E, 6), min(E, 16)}):
        say("[topk]", E, k, renorm)
        _, idx, gate = moe.moe_route_topk(None, None, None, k, logits=Lg, logits_in=True,
                                          renorm=renorm)
        torch.cuda.synchronize()
        oidx, og = oracle.topk(L, k, renorm=renorm)
        np.testing.assert_array_equal(idx.cpu().numpy(), oidx)
        close(np32(gate), og, 1e-5, "gates")


def test_every_token_to_one_expert_and_a_gpu_with_no_rows():
    cfg = synth.custom_config(d=128, E=8, k=2, f=128, G=2)
    T = 150
    pl = np.zeros((8, 2), np.uint8)
    pl[:4, 0] = 1
    pl[4:, 1] = 1
    L = np.zeros((T, 8), np.float32)
    L[:, 1] = 5.0
    L[:, 2] = 4.0                                # every token: experts 1, 2 (both on GPU 0)
    for dev, expect_rows in ((0, 2 * T), (1, 0)):
        inp, share = _share(cfg, T, placement=pl, dev=dev)
        share.run(logits_in=torch.from_numpy(L).cuda())
        torch.cuda.synchronize()
        go = share.perm["group_offsets"].cpu().numpy()
        assert go[-1] == expect_rows
        assert share.perm["send_counts"].cpu().numpy().tolist() == [2 * T, 0]
        if dev == 1:
            np.testing.assert_array_equal(share.perm["token_row"].cpu().numpy(), -1)
            np.testing.assert_array_equal(np32(share.y), 0.0)
        else:
            idx, gate = oracle.topk(L, 2)
            pm = oracle.permute(np32(inp.X), idx, gate, 8, pl, 0)
            np.testing.assert_array_equal(go, pm["group_offsets"])


@pytest.mark.parametrize("dev", [0, 2])
@pytest.mark.parametrize("T", [9000, 700])
def test_128_local_experts_with_replicas_on_three_gpus(T, dev):
    """128 local slots on each of three GPUs, half of each GPU's experts replicated on
    another: at T = 9000 the per-slot block scan holds 141 x 128 counts (two LDS tiles),
    at T = 700 the one-workgroup path runs.  Routing outputs bit-exact vs the oracle."""
    E, G = 256, 3
    cfg = synth.custom_config(d=64, E=E, k=8, f=64, G=G)
    pl = np.zeros((E, G), np.uint8)
    pl[0:128, 0] = 1
    pl[64:192, 1] = 1
    pl[192:256, 2] = 1
    pl[0:64, 2] = 1
    inp, share = _share(cfg, T, placement=pl, dev=dev)
    assert share.n_local == 128
    rng = np.random.default_rng(T + dev)
    L = (rng.standard_normal((T, E)) + np.linspace(2.0, 0.0, E)[None, :]).astype(np.float32)
    share.run(logits_in=torch.from_numpy(L).cuda())
    torch.cuda.synchronize()
    idx, gate = oracle.topk(L, cfg.k, renorm=True)
    np.testing.assert_array_equal(share.topk_idx.cpu().numpy(), idx)
    pm = oracle.permute(np32(inp.X), idx, gate, E, pl, dev)
    N = pm["rows"]
    got = {k: v.cpu().numpy() for k, v in share.perm.items() if v is not None and k != "x_perm"}
    np.testing.assert_array_equal(got["group_offsets"], pm["group_offsets"])
    np.testing.assert_array_equal(got["row_token"][:N], pm["row_token"])
    np.testing.assert_array_equal(got["token_row"], pm["token_row"])
    np.testing.assert_array_equal(got["send_counts"], pm["send_counts"])
    close(got["row_gate"][:N], pm["row_gate"], GATE_TOL, "row_gate")
    np.testing.assert_array_equal(np32(share.perm["x_perm"][:N]), pm["x_perm"])


@pytest.mark.parametrize("T,k,E,offset", [(0, 4, 13, 0), (1, 3, 13, 1), (37, 5, 13, 0),
                                            (64, 8, 128, 0), (512, 16, 128, 1), (513, 2, 7, 1),
                                            (3000, 8, 128, 0)])
def test_histogram_with_coactivation_every_bin(T, k, E, offset):
    """Short batches take the one-workgroup co-activation kernel (odd E: E*E not a
    multiple of 4; offset 1: an output not 16-byte aligned), longer ones the
    multi-block path after one clearing launch.  Bit-exact vs the oracle."""
    rng = np.random.default_rng(T * 31 + k + E)
    idx = np.array([rng.permutation(E)[:k] for _ in range(T)], np.int32).reshape(T, k)
    dev_idx = torch.from_numpy(idx).cuda()
    coact = torch.full((E * E + offset,), -7, dtype=torch.int32, device="cuda")[offset:].view(E, E)
    counts = torch.full((E,), -7, dtype=torch.int32, device="cuda")
    moe.moe_expert_histogram(dev_idx, E, counts=counts, coact=coact)
    torch.cuda.synchronize()
    rc, rco = oracle.histogram(idx, E, True)
    np.testing.assert_array_equal(counts.cpu().numpy(), rc)
    np.testing.assert_array_equal(coact.cpu().numpy(), rco)


def _both_paths(cfg, T, logits=None, seed=1):
    """The same share run with x_perm materialised and with the gather in the FFN."""
    inp = synth.make_layer(cfg, T, seed=seed, device="cuda")
    outs = []
    for gather in (False, True):
        share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                           shared=inp.shared, coact=cfg.coact, gather_in_ffn=gather,
                           fuse_combine=False, shared_in_ffn=False)
        share.run(logits_in=logits)
        torch.cuda.synchronize()
        N = int(share.perm["group_offsets"][-1])
        outs.append((share.y.clone(), share.y_perm[:N].clone(), share.perm["row_token"][:N].clone()))
    return outs


@pytest.mark.parametrize("name", list(SMALL))
def test_gather_in_ffn_is_bitwise_equal_to_the_packaged_path(name):
    """moe_permute with row maps only + moe_grouped_ffn_rows gives the same bits as
    moe_permute + moe_grouped_ffn (which the oracle checks): the rows are read from X
    through row_token instead of from the packaged copy."""
    cfg, T = SMALL[name]
    say("[gather]", name, "T=%d" % T)
    (y0, yp0, rt0), (y1, yp1, rt1) = _both_paths(cfg, T)
    assert torch.equal(rt0, rt1)
    assert torch.equal(yp0, yp1)
    assert torch.equal(y0, y1)


@pytest.mark.parametrize("sizes,d,f", [([64, 65, 1, 0, 200, 33], 256, 192),
                                       ([300, 96, 0, 70], 1024, 2048),
                                       ([5, 17, 1300], 256, 128),
                                       ([257, 256, 129, 65, 64, 3], 256, 256),
                                       ([200, 200, 200, 200, 200, 65, 64], 256, 2048)])
def test_gather_in_ffn_across_the_streaming_and_split_paths(sizes, d, f):
    """Group sizes on both sides of the streaming limits and mid-sized groups whose
    tiles split K: in a short call (few tiles) groups of up to 256 rows stream and a
    257-row group is tiled; with 16 gate/up column tiles per group (f = 2048) the
    200-row and 65-row groups make enough tiles to stay on the tiled kernel for that
    product, while the down product (one column tile per group at d = 256) streams
    them, so the two products split the groups differently.  The gathered path
    matches the packaged one bit for bit and the oracle's FFN of the packaged rows
    within the bf16 tolerance."""
    E = len(sizes)
    cfg = synth.custom_config(d=d, E=E, k=1, f=f, G=1)
    T = sum(sizes)
    owner = np.repeat(np.arange(E), sizes)
    np.random.default_rng(11).shuffle(owner)
    L = np.zeros((T, E), np.float32)
    L[np.arange(T), owner] = 1.0
    Lg = torch.from_numpy(L).cuda()
    (y0, yp0, _), (y1, yp1, rt) = _both_paths(cfg, T, logits=Lg)
    assert torch.equal(yp0, yp1) and torch.equal(y0, y1)
    inp = synth.make_layer(cfg, T, seed=1, device="cuda")
    X = np32(inp.X)
    idx, gate = oracle.topk(L, 1)
    pm = oracle.permute(X, idx, gate, E, inp.placement, 0)
    go = pm["group_offsets"]
    for s_ in range(E):
        if sizes[s_]:
            ref = oracle.expert_ffn(pm["x_perm"][go[s_]:go[s_ + 1]], np32(inp.w13[s_]), np32(inp.w2[s_]))
            close(np32(yp1[go[s_]:go[s_ + 1]]), ref, OUT_TOL["bf16"], "group %d" % s_)


@pytest.mark.parametrize("name,regime", [("mixtral_8x7b", "prefill"), ("mixtral_8x7b", "decode"),
                                         ("qwen3_30b_a3b", "prefill")])
def test_gather_in_ffn_at_model_shapes(name, regime):
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[gather-full]", name, regime, "T=%d" % T)
    (y0, yp0, _), (y1, yp1, _) = _both_paths(cfg, T, seed=0)
    assert torch.equal(yp0, yp1) and torch.equal(y0, y1)


@pytest.mark.parametrize("name,regime", [("mixtral_8x7b", "prefill"), ("mixtral_8x7b", "decode"),
                                         ("deepseek_v2_lite", "decode"), ("tiny_fp32", "batch")])
def test_ffn_products_one_at_a_time_equal_the_whole_call(name, regime):
    """moe_grouped_ffn_products: the gate/up product, then the down product on the
    same workspace, gives the bits of moe_grouped_ffn (the Mixtral prefill shape
    splits K over its last tiles, the decode shapes stream every group)."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[products]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=2, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared, coact=cfg.coact, fuse_combine=False,
                       shared_in_ffn=False, gather_in_ffn=False)
    share.run()
    torch.cuda.synchronize()
    N = int(share.perm["group_offsets"][-1])
    whole = share.y_perm[:N].clone()
    share.y_perm.zero_()
    for products in (moe.MOE_FFN_GATE_UP, moe.MOE_FFN_DOWN):
        moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"], share.weights,
                            cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn,
                            products=products)
    torch.cuda.synchronize()
    assert torch.equal(share.y_perm[:N], whole)


@pytest.mark.parametrize("name,regime", [("deepseek_v2_lite", "prefill"), ("qwen3_30b_a3b", "decode")])
def test_rows_products_one_at_a_time_equal_the_whole_call(name, regime):
    """moe_grouped_ffn_rows_products: the gate/up product (rows through row_token),
    then the down product on the same workspace, with and without the share's hint,
    gives the bits of moe_grouped_ffn_rows."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[rows products]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=7, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared, coact=cfg.coact, gather_in_ffn=True,
                       shared_in_ffn=False)
    share.run()
    torch.cuda.synchronize()
    N = int(share.perm["group_offsets"][-1])
    args = (share.X, share.perm["row_token"], share.perm["group_offsets"], share.weights)
    moe.moe_grouped_ffn_rows(*args, cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn)
    torch.cuda.synchronize()
    whole = share.y_perm[:N].clone()
    hint = share.ffn_products & (moe.MOE_FFN_SMALL_GROUPS | moe.MOE_FFN_LARGE_GROUPS)
    for extra in sorted({0, hint}):
        share.y_perm.zero_()
        for products in (moe.MOE_FFN_GATE_UP, moe.MOE_FFN_DOWN):
            moe.moe_grouped_ffn_rows(*args, cap_rows=share.cap_rows, y_perm=share.y_perm,
                                     ws=share.ws_ffn, products=products | extra)
        torch.cuda.synchronize()
        assert torch.equal(share.y_perm[:N], whole), "hint %d" % extra


@pytest.mark.parametrize("name,regime", [("mixtral_8x7b", "decode"), ("qwen3_30b_a3b", "decode"),
                                         ("deepseek_v2_lite", "decode")])
def test_small_groups_hint_leaves_the_outputs_bitwise_unchanged(name, regime):
    """Decode batches (at most 256 tokens, groups of a few dozen rows): every group is
    streamed with or without MOE_FFN_SMALL_GROUPS -- groups of at most 64 rows always
    are, and a larger one (the 256-row shared-expert group of the DeepSeek-V2-Lite
    shape) makes too few tiles for the tiled kernel -- so the hinted calls (no tiled
    launches) give the bits of the calls without the hint, routed and shared."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    assert T <= 256
    say("[small groups]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=3, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared, coact=cfg.coact, fuse_combine=False,
                       shared_in_ffn=False, gather_in_ffn=False)
    assert share.ffn_products & moe.MOE_FFN_SMALL_GROUPS
    share.run()
    torch.cuda.synchronize()
    N = int(share.perm["group_offsets"][-1])
    hinted = share.y_perm[:N].clone()
    share.y_perm.zero_()
    moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"], share.weights,
                        cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn)
    torch.cuda.synchronize()
    assert torch.equal(share.y_perm[:N], hinted)
    if share.shared_weights is not None:
        plain = torch.empty_like(share.y_shared)
        moe.moe_grouped_ffn(share.X, share.shared_offsets, share.shared_weights, cap_rows=share.T,
                            y_perm=plain, ws=share.ws_shared)
        torch.cuda.synchronize()
        assert torch.equal(plain[:T], share.y_shared[:T])


@pytest.mark.parametrize("name,regime", [("deepseek_v2_lite", "prefill"), ("qwen15_moe_a27b", "batch")])
def test_large_groups_hint_leaves_the_shared_call_bitwise_unchanged(name, regime):
    """The shared experts' call over T > 256 tokens (one group of T rows) takes
    MOE_FFN_LARGE_GROUPS in LayerShare.run: no streaming launches, bitwise the call
    without the hint."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[large groups]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=4, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared, coact=cfg.coact, shared_in_ffn=False)
    assert share.shared_products & moe.MOE_FFN_LARGE_GROUPS
    share.run()
    torch.cuda.synchronize()
    plain = torch.empty_like(share.y_shared)
    moe.moe_grouped_ffn(share.X, share.shared_offsets, share.shared_weights, cap_rows=share.T,
                        y_perm=plain, ws=share.ws_shared)
    torch.cuda.synchronize()
    assert torch.equal(plain[:T], share.y_shared[:T])


@pytest.mark.parametrize("name,regime", [("mixtral_8x7b", "prefill"), ("deepseek_v2_lite", "prefill"),
                                         ("qwen3_30b_a3b", "prefill")])
def test_large_groups_hint_leaves_the_routed_call_bitwise_unchanged(name, regime):
    """Prefill batches whose mean group holds at least 512 rows: LayerShare passes
    MOE_FFN_LARGE_GROUPS to the routed call (packaged rows at the Mixtral shape,
    rows gathered through row_token at the others), which leaves out the streaming
    launches; such a call tiles every group either way, so its outputs are the bits
    of the call without the hint."""
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[large groups, routed]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=6, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared, coact=cfg.coact, shared_in_ffn=False)
    assert share.ffn_products & moe.MOE_FFN_LARGE_GROUPS
    share.run()
    torch.cuda.synchronize()
    N = int(share.perm["group_offsets"][-1])
    hinted = share.y_perm[:N].clone()
    share.y_perm.zero_()
    if share.gather_in_ffn:
        moe.moe_grouped_ffn_rows(share.X, share.perm["row_token"], share.perm["group_offsets"],
                                 share.weights, cap_rows=share.cap_rows, y_perm=share.y_perm,
                                 ws=share.ws_ffn)
    else:
        moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"], share.weights,
                            cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn)
    torch.cuda.synchronize()
    assert torch.equal(share.y_perm[:N], hinted)


def test_large_groups_hint_broken_still_computes_every_group():
    """MOE_FFN_LARGE_GROUPS on groups that break it (empty, 1, 40, 64, 65, 200 and
    700 rows): every group goes to the tiled kernel instead of streaming and must
    still match the oracle; two runs agree bit for bit."""
    sizes = [0, 1, 40, 64, 65, 200, 700]
    E = len(sizes)
    cfg = synth.custom_config(d=256, E=E, k=1, f=192, G=1)
    T = sum(sizes)
    owner = np.repeat(np.arange(E), sizes)
    np.random.default_rng(11).shuffle(owner)
    L = np.zeros((T, E), np.float32)
    L[np.arange(T), owner] = 1.0
    inp, share = _share(cfg, T)
    share.run(logits_in=torch.from_numpy(L).cuda())
    torch.cuda.synchronize()
    go = share.perm["group_offsets"].cpu().numpy()
    assert np.diff(go).tolist() == sizes
    hinted = moe.MOE_FFN_GATE_UP | moe.MOE_FFN_DOWN | moe.MOE_FFN_LARGE_GROUPS
    outs = []
    for _ in range(2):
        share.y_perm.fill_(7.0)
        moe.moe_grouped_ffn(share.perm["x_perm"], share.perm["group_offsets"], share.weights,
                            cap_rows=share.cap_rows, y_perm=share.y_perm, ws=share.ws_ffn,
                            products=hinted)
        torch.cuda.synchronize()
        outs.append(share.y_perm[:T].clone())
    assert torch.equal(outs[0], outs[1])
    X = np32(inp.X)
    idx, gate = oracle.topk(L, 1)
    pm = oracle.permute(X, idx, gate, E, inp.placement, 0)
    for s in range(E):
        if sizes[s]:
            ref = oracle.expert_ffn(pm["x_perm"][go[s]:go[s + 1]], np32(share.weights.w13[s]),
                                    np32(share.weights.w2[s]))
            close(np32(outs[0][go[s]:go[s + 1]]), ref, OUT_TOL["bf16"], "group %d" % s)


@pytest.mark.parametrize("d,f,group_rows", [(64, 64, 5000), (128, 64, 6000), (64, 128, 5000)])
def test_many_short_k_tiles_per_workgroup(d, f, group_rows):
    """One and two K stages per tile (K = 64 or 128) with more tiles than workgroups:
    each workgroup runs several tiles back to back, so the next tile's first stages
    are loaded during the last step of the one before (and with one stage per tile,
    in the peeled step).  Every group against the oracle, two runs bit for bit."""
    n = 16
    sizes = [group_rows + 37 * s for s in range(n)]          # ragged last m-tiles
    N = sum(sizes)
    say("[short-K tiles]", "d", d, "f", f, "rows", N)
    cfg = synth.custom_config(d=d, E=n, k=1, f=f, G=1)
    x = synth.normal((N, d), 21, "x", 0, 1.0, "cuda", torch.bfloat16)
    ws = [synth.expert_weights(cfg, s, 21, "cuda") for s in range(n)]
    table = moe.WeightTable([a for a, _ in ws], [b for _, b in ws])
    offs = torch.tensor(np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32), device="cuda")
    outs = []
    for _ in range(2):
        outs.append(moe.moe_grouped_ffn(x, offs, table, cap_rows=N).clone())
        torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    X = np32(x)
    go = offs.cpu().numpy()
    for s in range(n):
        ref = oracle.expert_ffn(X[go[s]:go[s + 1]], np32(ws[s][0]), np32(ws[s][1]))
        close(np32(outs[0][go[s]:go[s + 1]]), ref, OUT_TOL["bf16"], "group %d" % s)


FUSED = [("mixtral_8x7b", "decode", None), ("qwen3_30b_a3b", "decode", None),
         ("shared_T50", "batch", synth.custom_config(d=256, E=16, k=4, f=256, shared_f=(128, 64),
                                                     G=3, replicas=2, zipf=1.2, T=50)),
         ("T1", "batch", synth.custom_config(d=128, E=8, k=2, f=128, G=2, T=1)),
         ("k16", "batch", synth.custom_config(d=128, E=64, k=16, f=64, G=3, replicas=2, zipf=1.1,
                                              T=60))]


@pytest.mark.parametrize("name,regime,custom", FUSED)
def test_fused_ffn_combine_is_bitwise_the_ffn_then_the_combine(name, regime, custom):
    """moe_grouped_ffn_combine (the down product's chunk sum writing the gate-weighted
    combine, y_perm never written) gives the bits of moe_grouped_ffn + moe_combine,
    with shared experts (joined from their stream), one token, and k = 16."""
    cfg = custom if custom is not None else synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[fused]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=5, device="cuda")
    fused, plain = (LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                               shared=inp.shared, coact=cfg.coact, fuse_combine=fz,
                               shared_in_ffn=False)
                    for fz in (True, False))
    assert fused.fused_combine and not plain.fused_combine
    fused.y.fill_(7.0)
    fused.run()
    plain.run()
    torch.cuda.synchronize()
    assert torch.equal(fused.y[:T], plain.y[:T])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fused.run()
    for _ in range(3):
        fused.y.fill_(7.0)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(fused.y[:T], plain.y[:T])


def test_very_long_batch_routing_and_packaging_every_element():
    """T = 100000 tokens at a small width: the long-batch paths of the gate (tiled
    scores), histogram (several workgroups), permute (count / scan / scatter over
    1563 blocks) and combine, routing outputs bit-exact and the combined output on
    sampled tokens within the bf16 tolerance."""
    cfg = synth.custom_config(d=64, E=48, k=4, f=64, G=2, replicas=1, zipf=1.2, coact=True)
    say("[long]", "T=100000")
    case = Case(cfg, 100000, gather_in_ffn=False)       # the row copy is checked too
    ref_logits, _ = check_logits(case)
    idx, gate, pm = check_routing(case, ref_logits)
    check_ffn_and_combine(case, idx, gate, pm, sample=64)


def test_gpu_hosting_no_expert_returns_shared_output_only():
    cfg = synth.custom_config(d=128, E=4, k=2, f=64, shared_f=(128,), G=2)
    pl = np.zeros((4, 2), np.uint8)
    pl[:, 0] = 1
    inp, share = _share(cfg, 90, placement=pl, dev=1)
    assert share.n_local == 0
    share.run()
    torch.cuda.synchronize()
    ys = oracle.expert_ffn(np32(inp.X), np32(inp.shared[0][0]), np32(inp.shared[0][1]))
    close(np32(share.y), ys, OUT_TOL["bf16"], "shared-only y")


def test_repeated_runs_are_bitwise_identical():
    cfg = synth.custom_config(d=256, E=16, k=4, f=256, G=3, replicas=2, zipf=1.2, coact=True)
    inp, share = _share(cfg, 500)
    share.coact = torch.empty((16, 16), dtype=torch.int32, device="cuda")
    outs = []
    for _ in range(3):
        share.run()
        torch.cuda.synchronize()
        outs.append([share.y.clone(), share.coact.clone(), share.perm["row_token"].clone()])
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert torch.equal(a, b)


def test_doubling_w2_doubles_expert_outputs_exactly():
    cfg = synth.custom_config(d=128, E=8, k=2, f=192, G=2)
    inp, share = _share(cfg, 200)
    share.run()
    torch.cuda.synchronize()
    y1 = share.y_perm.clone()
    N = int(share.perm["group_offsets"][-1])
    share.set_placement(share.placement, share.weights.w13, [2 * w for w in share.weights.w2])
    share.run()
    torch.cuda.synchronize()
    assert torch.equal(share.y_perm[:N], 2 * y1[:N])


def test_group_sizes_around_the_streaming_threshold():
    """Sizes 64 / 65 / 1 / 0 / 200 / 33 at f = 192: the two groups above 64 rows make
    only 4 gate/up tiles, so this short call streams every group (the 65- and 200-row
    ones included); each group must match the oracle."""
    sizes = [64, 65, 1, 0, 200, 33]
    E = len(sizes)
    cfg = synth.custom_config(d=256, E=E, k=1, f=192, G=1)
    T = sum(sizes)
    owner = np.repeat(np.arange(E), sizes)
    np.random.default_rng(5).shuffle(owner)
    L = np.zeros((T, E), np.float32)
    L[np.arange(T), owner] = 1.0
    inp, share = _share(cfg, T)
    share.run(logits_in=torch.from_numpy(L).cuda())
    torch.cuda.synchronize()
    go = share.perm["group_offsets"].cpu().numpy()
    assert np.diff(go).tolist() == sizes
    X = np32(inp.X)
    idx, gate = oracle.topk(L, 1)
    pm = oracle.permute(X, idx, gate, E, inp.placement, 0)
    for s in range(E):
        if sizes[s]:
            w13 = np32(share.weights.w13[s])
            w2 = np32(share.weights.w2[s])
            ref = oracle.expert_ffn(pm["x_perm"][go[s]:go[s + 1]], w13, w2)
            close(np32(share.y_perm[go[s]:go[s + 1]]), ref, OUT_TOL["bf16"], "group %d" % s)


def _random_sizes(rng):
    """1-12 groups drawn from empty, <= 64, 65-256 and 257-600 rows."""
    n = int(rng.integers(1, 13))
    kinds = rng.choice(4, size=n, p=[0.15, 0.35, 0.35, 0.15])
    lo, hi = (0, 1, 65, 257), (0, 64, 256, 600)
    sizes = [int(rng.integers(lo[c], hi[c] + 1)) for c in kinds]
    if sum(sizes) == 0:
        sizes[0] = 1
    return sizes


@pytest.mark.parametrize("seed", range(8))
def test_random_group_sizes_across_the_streaming_limits(seed):
    """Random mixes of group sizes and shapes: which groups stream and which are tiled
    is decided on the device per product (64 or 256 rows, by the tile count), and every
    launch of the call must agree on it, or rows of H or y_perm would be left unwritten
    or written twice.  Every group must match the oracle, and two runs must agree bit
    for bit."""
    rng = np.random.default_rng(100 + seed)
    sizes = _random_sizes(rng)
    d = int(rng.choice([128, 256, 512]))
    f = int(rng.choice([128, 384, 1024, 2048]))
    say("[random groups]", "seed", seed, "d", d, "f", f, "sizes", sizes)
    E = len(sizes)
    cfg = synth.custom_config(d=d, E=E, k=1, f=f, G=1)
    T = sum(sizes)
    owner = np.repeat(np.arange(E), sizes)
    rng.shuffle(owner)
    L = np.zeros((T, E), np.float32)
    L[np.arange(T), owner] = 1.0
    inp, share = _share(cfg, T)
    Lg = torch.from_numpy(L).cuda()
    share.run(logits_in=Lg)
    torch.cuda.synchronize()
    first = share.y_perm[:T].clone()
    share.run(logits_in=Lg)
    torch.cuda.synchronize()
    assert torch.equal(first, share.y_perm[:T])
    go = share.perm["group_offsets"].cpu().numpy()
    assert np.diff(go).tolist() == sizes
    X = np32(inp.X)
    idx, gate = oracle.topk(L, 1)
    pm = oracle.permute(X, idx, gate, E, inp.placement, 0)
    for s in range(E):
        if sizes[s]:
            ref = oracle.expert_ffn(pm["x_perm"][go[s]:go[s + 1]], np32(share.weights.w13[s]),
                                    np32(share.weights.w2[s]))
            close(np32(share.y_perm[go[s]:go[s + 1]]), ref, OUT_TOL["bf16"], "group %d" % s)


def test_mid_sized_groups_split_k_in_the_tiled_kernel():
    """Groups of 300 / 96 / 0 / 70 rows at d=1024, f=2048: the 96- and 70-row groups
    stream (a short call), the 300-row group gives the tiled kernel 32 gate/up tiles
    (16 K stages) and 8 down tiles (32 K stages) for 256 CUs, so both products split K
    (2 and 4 chunks) and finish in the reduce kernel.  Each group must match the
    oracle, and two runs must agree bit for bit (chunks are summed in order)."""
    sizes = [300, 96, 0, 70]
    E = len(sizes)
    cfg = synth.custom_config(d=1024, E=E, k=1, f=2048, G=1)
    T = sum(sizes)
    owner = np.repeat(np.arange(E), sizes)
    np.random.default_rng(9).shuffle(owner)
    L = np.zeros((T, E), np.float32)
    L[np.arange(T), owner] = 1.0
    inp, share = _share(cfg, T)
    Lg = torch.from_numpy(L).cuda()
    share.run(logits_in=Lg)
    torch.cuda.synchronize()
    first = share.y_perm[:T].clone()
    share.run(logits_in=Lg)
    torch.cuda.synchronize()
    assert torch.equal(first, share.y_perm[:T])
    go = share.perm["group_offsets"].cpu().numpy()
    assert np.diff(go).tolist() == sizes
    X = np32(inp.X)
    idx, gate = oracle.topk(L, 1)
    pm = oracle.permute(X, idx, gate, E, inp.placement, 0)
    for s in range(E):
        if sizes[s]:
            w13 = np32(share.weights.w13[s])
            w2 = np32(share.weights.w2[s])
            ref = oracle.expert_ffn(pm["x_perm"][go[s]:go[s + 1]], w13, w2)
            close(np32(share.y_perm[go[s]:go[s + 1]]), ref, OUT_TOL["bf16"], "group %d" % s)


def test_shared_expert_branch_on_a_second_stream_is_bitwise_equal():
    """The shared experts' FFN forked onto a second stream (the default) gives the
    same bits as the whole share on one stream, eagerly and over graph replays with
    new hidden states copied in between."""
    cfg = synth.custom_config(d=256, E=16, k=4, f=256, shared_f=(128, 64), G=2, replicas=1,
                              zipf=1.1)
    T = 300
    inp = synth.make_layer(cfg, T, seed=4, device="cuda")
    one, two = (LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                           shared=inp.shared, overlap_shared=ov) for ov in (False, True))
    one.run()
    two.run()
    torch.cuda.synchronize()
    assert torch.equal(one.y[:T], two.y[:T])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        two.run()
    gen = torch.Generator(device="cuda").manual_seed(5)
    for _ in range(3):
        inp.X.copy_(torch.randn(inp.X.shape, device="cuda", generator=gen).to(inp.X.dtype))
        g.replay()
        one.run()
        torch.cuda.synchronize()
        assert torch.equal(one.y[:T], two.y[:T])


def test_graph_replays_match_eager_runs():
    """The whole share captured once in a HIP graph: every replay (with new hidden
    states copied in eagerly between replays) must equal an eager run bit for bit."""
    cfg = synth.custom_config(d=256, E=16, k=4, f=256, shared_f=(128,), G=3, replicas=2,
                              zipf=1.2)
    inp, share = _share(cfg, 300)
    share.coact = torch.empty((16, 16), dtype=torch.int32, device="cuda")
    assert share.ws_route is not None                   # the split-K gate path is exercised

    def snap():
        N = int(share.perm["group_offsets"][-1])
        return [share.y.clone(), share.topk_idx.clone(), share.counts.clone(), share.coact.clone(),
                share.perm["token_row"].clone(), share.y_perm[:N].clone(), share.logits.clone()]

    share.run()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        share.run()
    torch.cuda.synchronize()
    for i in range(4):
        share.X.copy_(synth.normal(tuple(share.X.shape), 100 + i, "X", 0, 1.0, "cuda", torch.bfloat16))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snap()
        share.run()
        torch.cuda.synchronize()
        ref = snap()
        for a, b in zip(got, ref):
            assert torch.equal(a, b), "replay %d differs from the eager run" % i


@pytest.mark.parametrize("k,d", [(3, 512), (8, 512), (16, 1024), (8, 2048)])
def test_combine_with_compacted_rows_is_exact_on_exact_values(k, d):
    """Rows of whole wave widths at k > 2 take the combine that compacts each token's
    local rows: tokens with none, some and all of their k rows here, in every order.
    Values are small integers and the gates powers of two, so every sum is exact in
    fp32 and bf16 and the output must equal the oracle's bit for bit."""
    say("[combine compact]", "k=%d d=%d" % (k, d))
    rng = np.random.default_rng(k * 1000 + d)
    T = 301
    local = rng.integers(0, k + 1, size=T)
    local[:3] = (0, k, 1)
    N = int(local.sum())
    rows = rng.permutation(N)
    token_row = np.full((T, k), -1, np.int32)
    p = 0
    for t in range(T):
        slots = rng.choice(k, size=int(local[t]), replace=False)
        for r in slots:
            token_row[t, r] = rows[p]
            p += 1
    gate = rng.choice(np.array([0.25, 0.5, 1.0], np.float32), size=(T, k)).astype(np.float32)
    y_perm = rng.integers(-2, 3, size=(max(N, 1), d)).astype(np.float32)
    y_shared = rng.integers(-2, 3, size=(T, d)).astype(np.float32)
    for ys in (None, y_shared):
        got = moe.moe_combine(torch.from_numpy(y_perm).bfloat16().cuda(),
                              torch.from_numpy(token_row).cuda(), torch.from_numpy(gate).cuda(),
                              None if ys is None else torch.from_numpy(ys).bfloat16().cuda(),
                              T=T, d=d)
        torch.cuda.synchronize()
        ref = oracle.combine(y_perm, token_row, gate, ys, T, d, k)
        np.testing.assert_array_equal(np32(got[:T]), ref.astype(np.float32))


# ---------------------------------------------------------------------------
# shared experts as leading groups of the routed experts' call
# ---------------------------------------------------------------------------
def _rand_bf16(shape, gen, scale):
    return (torch.randn(shape, generator=gen) * scale).to(torch.bfloat16)


@pytest.mark.parametrize("dtype,sizes,n_shared,T,d,f,hint", [
    ("bf16", [130, 0, 7, 300, 64, 65], 3, 200, 256, 128, 0),
    ("bf16", [40, 1, 0, 256, 17], 2, 256, 128, 192, moe.MOE_FFN_SMALL_GROUPS),
    ("bf16", [900, 5, 600], 1, 700, 128, 128, moe.MOE_FFN_LARGE_GROUPS),
    ("bf16", [], 4, 300, 128, 64, 0),                       # no routed group at all
    ("f32", [33, 0, 70], 2, 50, 72, 40, 0),
])
def test_rows_shared_call_every_row(dtype, sizes, n_shared, T, d, f, hint):
    """moe_grouped_ffn_rows_shared: n_shared leading groups of T rows (every token
    once, rows [s T, (s+1) T)), then the routed groups (rows counted from n_shared T,
    read through row_token), in one call; every output row against the oracle's
    expert FFN on the row's token and its group's weights (ragged and empty routed
    groups, streamed and tiled sizes, both hints, fp32)."""
    say("[rows shared]", dtype, sizes, "n_shared=%d T=%d d=%d f=%d hint=%d" % (n_shared, T, d, f, hint))
    gen = torch.Generator().manual_seed(sum(sizes) + 31 * n_shared + T)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    n_groups, N = len(sizes), sum(sizes)
    groups = n_shared + n_groups
    x = (torch.randn((T, d), generator=gen)).to(tdt)
    w13 = [(torch.randn((2 * f, d), generator=gen) * d ** -0.5).to(tdt) for _ in range(groups)]
    w2 = [(torch.randn((d, f), generator=gen) * f ** -0.5).to(tdt) for _ in range(groups)]
    cap = N + 3                                              # rows past the groups stay untouched
    routed_tok = torch.randint(0, T, (cap,), generator=gen, dtype=torch.int32)
    lead = n_shared * T
    row_token = torch.cat([torch.arange(T, dtype=torch.int32).repeat(n_shared), routed_tok])
    offsets = torch.tensor(np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32))
    y = torch.full((lead + cap, d), 5.0, dtype=tdt).cuda()
    wt = moe.WeightTable([w.cuda() for w in w13], [w.cuda() for w in w2])
    moe.moe_grouped_ffn_rows_shared(x.cuda(), row_token.cuda(), offsets.cuda(), wt, n_shared,
                                    cap_rows=cap, y_perm=y, products=3 | hint)
    torch.cuda.synchronize()
    got = np32(y)
    xs = np32(x)
    tol = OUT_TOL[dtype]
    starts = [s * T for s in range(n_shared)] + [lead + int(o) for o in offsets[:-1]]
    counts = [T] * n_shared + list(sizes)
    tok = np32(row_token).astype(np.int64)
    for g in range(groups):
        a, n = starts[g], counts[g]
        if n == 0:
            continue
        ref = oracle.expert_ffn(xs[tok[a:a + n]], np32(w13[g]), np32(w2[g]))
        close(got[a:a + n], ref, tol, "group %d" % g)
    assert np.all(got[lead + N:] == 5.0)


@pytest.mark.parametrize("n_shared", [0, 1, 2, 3, 5])
@pytest.mark.parametrize("k,d", [(2, 512), (8, 512), (6, 72)])
def test_combine_shared_slices_exact(n_shared, k, d):
    """moe_combine_shared: the routed sum, then n_shared slices in order; on values
    exact in bf16 and fp32 the output equals the oracle's combine of the slices'
    sum bit for bit, and n_shared = 1 is moe_combine bit for bit."""
    say("[combine shared]", "n_shared=%d k=%d d=%d" % (n_shared, k, d))
    rng = np.random.default_rng(n_shared * 100 + k * 10 + d)
    T = 190
    local = rng.integers(0, k + 1, size=T)
    N = int(local.sum())
    rows = rng.permutation(N)
    token_row = np.full((T, k), -1, np.int32)
    p = 0
    for t in range(T):
        for r in rng.choice(k, size=int(local[t]), replace=False):
            token_row[t, r] = rows[p]
            p += 1
    gate = rng.choice(np.array([0.25, 0.5, 1.0], np.float32), size=(T, k)).astype(np.float32)
    y_perm = rng.integers(-2, 3, size=(max(N, 1), d)).astype(np.float32)
    sl = rng.integers(-2, 3, size=(max(n_shared, 1), T, d)).astype(np.float32)
    dev = lambda a: torch.from_numpy(a).bfloat16().cuda()
    got = moe.moe_combine_shared(dev(y_perm), torch.from_numpy(token_row).cuda(),
                                 torch.from_numpy(gate).cuda(), dev(sl) if n_shared else None,
                                 n_shared, T=T, d=d)
    torch.cuda.synchronize()
    ref = oracle.combine(y_perm, token_row, gate, sl[:n_shared].sum(0) if n_shared else None,
                         T, d, k)
    np.testing.assert_array_equal(np32(got[:T]), ref.astype(np.float32))
    if n_shared == 1:
        one = moe.moe_combine(dev(y_perm), torch.from_numpy(token_row).cuda(),
                              torch.from_numpy(gate).cuda(), dev(sl[0]), T=T, d=d)
        torch.cuda.synchronize()
        assert torch.equal(one, got)


@pytest.mark.parametrize("T", [300, 64, 1])
def test_layer_share_with_shared_experts_in_the_routed_call(T):
    """LayerShare(shared_in_ffn=True): the shared experts (widths 2f and f, cut into
    three blocks of width f) run as leading groups of the routed call and the combine
    adds their slices.  y matches the oracle's layer share on the same routing and
    the two-stream share within the output tolerance, the blocks' summed output
    matches the oracle's shared experts, and graph replays with new hidden states
    give the eager run's bits."""
    cfg = synth.custom_config(d=256, E=16, k=4, f=128, shared_f=(256, 128), G=2, replicas=1,
                              zipf=1.1)
    say("[shared in ffn]", "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=9, device="cuda")
    merged = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                        shared=inp.shared)
    two = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                     shared=inp.shared, shared_in_ffn=False)
    assert merged.shared_in_ffn and merged.n_shared_blocks == 3 and not two.shared_in_ffn
    merged.run()
    two.run()
    torch.cuda.synchronize()
    assert torch.equal(merged.topk_idx, two.topk_idx)
    X, Wr, b = np32(inp.X), np32(inp.Wr), np32(inp.bias)
    ref = oracle.layer_share(X, Wr, b, cfg.k, inp.placement, 0, [np32(w) for w in inp.w13],
                             [np32(w) for w in inp.w2],
                             shared=[(np32(a), np32(c)) for a, c in inp.shared],
                             logits_f32=np32(merged.logits))
    tol = OUT_TOL["bf16"]
    np.testing.assert_array_equal(np32(merged.topk_idx), ref["idx"])
    close(np32(merged.y[:T]), ref["y"], tol, "y (shared in the routed call)")
    close(np32(merged.y[:T]), np32(two.y[:T]), tol, "y vs the two-stream share")
    close(merged.shared_output().cpu().numpy(), ref["y_shared"], tol, "shared experts' output")
    N = int(merged.perm["group_offsets"][-1])
    close(np32(merged.y_perm[:N]), ref["y_perm"], tol, "routed rows")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        merged.run()
    gen = torch.Generator(device="cuda").manual_seed(11)
    for _ in range(3):
        inp.X.copy_(torch.randn(inp.X.shape, device="cuda", generator=gen).to(inp.X.dtype))
        g.replay()
        torch.cuda.synchronize()
        replayed = merged.y[:T].clone()
        merged.run()
        torch.cuda.synchronize()
        assert torch.equal(replayed, merged.y[:T])


def test_empty_batch_with_shared_experts_takes_the_two_call_path():
    """A batch of no tokens with shared experts whose widths suit the routed call:
    the share keeps the shared experts' own call (their leading groups would hold
    no rows) and a step runs without error."""
    cfg = synth.custom_config(d=128, E=8, k=2, f=64, shared_f=(128,), G=2)
    inp = synth.make_layer(cfg, 0, seed=1, device="cuda")
    share = LayerShare(inp.X, inp.Wr, inp.bias, cfg.k, inp.placement, 0, inp.w13, inp.w2,
                       shared=inp.shared)
    assert not share.shared_in_ffn
    share.run()
    torch.cuda.synchronize()
