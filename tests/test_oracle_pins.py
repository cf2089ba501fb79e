"""Pins of the CPU oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: every expected value comes from
a different route (a library routine, a closed form, brute force on a tiny
input, or an invariant).  Each group names the step of the layer it pins:
gate scores, top-k and weighted sum (Sec. II-A), packaging for the hosting
GPUs (Sec. II-B), workload counts, Eq. (1) load and Eq. (3) volume (Sec. VI-A).
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from paper_2607_08782_amd import synth


def _rng(seed=0):
    return np.random.default_rng(seed)


def _bf16_exact(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).float().numpy()


# ----------------------------------------------------------------------------- gate scores
def test_logits_match_numpy_float64_matmul():
    r = _rng(1)
    T, d, E = 37, 96, 11
    X = _bf16_exact(r.standard_normal((T, d)))
    Wr = _bf16_exact(0.02 * r.standard_normal((E, d)))
    b = r.standard_normal(E).astype(np.float32)
    got = oracle.router_logits(X, Wr, b)
    ref = X.astype(np.float64) @ Wr.astype(np.float64).T + b.astype(np.float64)
    # standard dot-product bound in double: |err| <= gamma_d * sum |x_i w_i|
    bound = (d + 1) * 2.0 ** -52 * (np.abs(X).astype(np.float64) @ np.abs(Wr).astype(np.float64).T + np.abs(b))
    assert np.all(np.abs(got - ref) <= bound + 1e-300)


def test_logits_one_hot_rows_pick_router_columns():
    r = _rng(2)
    T, d, E = 5, 7, 3            # E != d catches a transposed router operand
    X = np.zeros((T, d), np.float32)
    cols = [0, 3, 6, 2, 5]
    for t, c in enumerate(cols):
        X[t, c] = 1.0
    Wr = r.standard_normal((E, d)).astype(np.float32)
    b = r.standard_normal(E).astype(np.float32)
    got = oracle.router_logits(X, Wr, b)
    for t, c in enumerate(cols):
        np.testing.assert_array_equal(got[t], Wr[:, c].astype(np.float64) + b.astype(np.float64))
    np.testing.assert_array_equal(oracle.router_logits(np.zeros((2, d), np.float32), Wr, b),
                                  np.tile(b.astype(np.float64), (2, 1)))


# ----------------------------------------------------------------------------- top-k
@pytest.mark.parametrize("E,k", [(8, 2), (64, 6), (60, 4), (128, 8), (5, 5), (9, 1)])
def test_topk_is_stable_descending_sort(E, k):
    r = _rng(E * 31 + k)
    T = 200
    # few distinct levels -> many exact ties; includes -0.0 and +0.0
    L = r.integers(-3, 4, size=(T, E)).astype(np.float32) * 0.5
    L[L == 0] = np.where(r.random((L == 0).sum()) < 0.5, -0.0, 0.0)
    idx, _ = oracle.topk(L, k)
    ref = np.argsort(-L, axis=1, kind="stable")[:, :k]
    np.testing.assert_array_equal(idx, ref)


def test_topk_all_equal_and_full_order():
    L = np.full((3, 7), 1.25, np.float32)
    idx, g = oracle.topk(L, 3)
    np.testing.assert_array_equal(idx, np.tile(np.arange(3), (3, 1)))
    np.testing.assert_allclose(g, 1.0 / 3.0, rtol=0, atol=1e-15)
    L2 = np.array([[3.0, -1.0, 3.0, 0.5, -0.0, 0.0]], np.float32)
    idx2, _ = oracle.topk(L2, 6)
    np.testing.assert_array_equal(idx2[0], [0, 2, 3, 4, 5, 1])


def test_gates_closed_forms_and_softmax():
    r = _rng(3)
    T, E, k = 50, 16, 4
    L = (2.0 * r.standard_normal((T, E))).astype(np.float32)
    idx1, g1 = oracle.topk(L, 1)
    assert np.all(g1 == 1.0)                     # exp(0)/exp(0)
    idx, g = oracle.topk(L, k, renorm=True)
    sel = np.take_along_axis(L.astype(np.float64), idx, 1)
    np.testing.assert_allclose(g, scipy.special.softmax(sel, axis=1), rtol=1e-13, atol=0)
    np.testing.assert_allclose(g.sum(1), 1.0, rtol=0, atol=1e-14)
    assert np.all(np.diff(g, axis=1) <= 0)       # descending logit -> descending gate
    idx_n, g_n = oracle.topk(L, k, renorm=False)
    full = scipy.special.softmax(L.astype(np.float64), axis=1)
    np.testing.assert_allclose(g_n, np.take_along_axis(full, idx_n, 1), rtol=1e-13, atol=0)
    # two selected experts: the gate is the logistic function of the logit gap
    L2 = np.array([[0.0, 1.0, 0.5, -4.0]], np.float32)
    idx2, g2 = oracle.topk(L2, 2)
    np.testing.assert_array_equal(idx2[0], [1, 2])
    assert abs(g2[0, 0] - 1.0 / (1.0 + math.exp(-0.5))) < 1e-15


# ----------------------------------------------------------------------------- workload counts
def test_histogram_bincount_and_coactivation_brute_force():
    r = _rng(4)
    T, E, k = 300, 12, 3
    idx = np.stack([r.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts, coact = oracle.histogram(idx, E, with_coact=True)
    np.testing.assert_array_equal(counts, np.bincount(idx.ravel(), minlength=E))
    brute = np.zeros((E, E), np.int64)
    for t in range(T):
        s = set(int(v) for v in idx[t])
        for a in range(E):
            for b in range(E):
                brute[a, b] += (a in s) and (b in s)
    np.testing.assert_array_equal(coact, brute)
    assert counts.sum() == T * k
    np.testing.assert_array_equal(coact, coact.T)
    np.testing.assert_array_equal(np.diag(coact), counts)
    np.testing.assert_array_equal(coact.sum(1), k * counts)
    assert coact.sum() == T * k * k


# ----------------------------------------------------------------------------- packaging
def _random_routing(r, T, E, k):
    return np.stack([r.permutation(E)[:k] for _ in range(T)]).astype(np.int32)


def test_permute_single_gpu_is_a_stable_sort():
    r = _rng(5)
    T, E, k, d = 150, 9, 3, 6
    idx = _random_routing(r, T, E, k)
    gate = r.random((T, k))
    X = r.standard_normal((T, d)).astype(np.float32)
    pm = oracle.permute(X, idx, gate, E, np.ones((E, 1), np.uint8), 0)
    order = np.argsort(idx.ravel(), kind="stable")
    assert pm["rows"] == T * k
    np.testing.assert_array_equal(pm["row_token"], order // k)
    np.testing.assert_array_equal(pm["row_gate"], gate.ravel()[order])
    tr = np.empty(T * k, np.int64)
    tr[order] = np.arange(T * k)
    np.testing.assert_array_equal(pm["token_row"].ravel(), tr)
    np.testing.assert_array_equal(pm["group_offsets"],
                                  np.concatenate([[0], np.cumsum(np.bincount(idx.ravel(), minlength=E))]))
    # permutation identity: every kept assignment carries its token's row, bit for bit
    for t in range(T):
        for q in range(k):
            np.testing.assert_array_equal(pm["x_perm"][pm["token_row"][t, q]], X[t])
    np.testing.assert_array_equal(pm["send_counts"], [T * k])


def _placement_with_replicas(r, E, G, extra):
    x = np.zeros((E, G), np.uint8)
    x[np.arange(E), r.integers(0, G, E)] = 1
    for e in r.choice(E, extra, replace=False):
        x[e, r.choice(G, r.integers(2, G + 1), replace=False)] = 1
    return x


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_permute_partition_over_gpus_with_replicas(seed):
    r = _rng(10 + seed)
    T, E, k, G = 211, 16, 4, 5
    idx = _random_routing(r, T, E, k)
    gate = r.random((T, k))
    X = r.standard_normal((T, 3)).astype(np.float32)
    pl = _placement_with_replicas(r, E, G, extra=5)
    kept = np.zeros((T, k), np.int64)
    sends = []
    host_tokens = {}
    for dev in range(G):
        pm = oracle.permute(X, idx, gate, E, pl, dev)
        sends.append(pm["send_counts"])
        assert pm["send_counts"][dev] == pm["rows"] == pm["group_offsets"][-1]
        kept += pm["token_row"] >= 0
        local = oracle.local_slots(pl, dev)
        go = pm["group_offsets"]
        for s, e in enumerate(local):
            toks = pm["row_token"][go[s]:go[s + 1]]
            assert np.all(np.diff(toks) > 0)                 # ascending token order
            assert np.all(np.any(idx[toks] == e, axis=1))    # rows really chose e
            host_tokens[(e, dev)] = toks
    np.testing.assert_array_equal(kept, np.ones((T, k)))       # each assignment exactly once
    for s in sends[1:]:
        np.testing.assert_array_equal(s, sends[0])
    assert sends[0].sum() == T * k
    counts = np.bincount(idx.ravel(), minlength=E)
    for e in range(E):
        hosts = list(np.nonzero(pl[e])[0])
        sizes = [len(host_tokens[(e, j)]) for j in hosts]
        assert sum(sizes) == counts[e] and max(sizes) - min(sizes) <= 1
        for a, b in zip(hosts, hosts[1:]):                   # contiguous blocks by GPU id
            if len(host_tokens[(e, a)]) and len(host_tokens[(e, b)]):
                assert host_tokens[(e, a)][-1] < host_tokens[(e, b)][0]


def test_replica_split_hand_example():
    """The replica load split, evaluated by hand (tests/golden): an expert with
    c_e tokens on n_e hosts gives its q-th host (ascending GPU id) the ranks
    [floor(q c_e / n_e), floor((q+1) c_e / n_e)).  At c_e = 7 over 3 hosts the
    blocks are 2, 2, 3 rows; a ceiling rule (3, 2, 2) fails here."""
    import json
    import os
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                     "replica_split_hand_example.json")))
    idx = np.array(fx["idx"], np.int32)
    pl = np.array(fx["placement"], np.uint8)
    gate = np.ones(idx.shape)
    X = np.arange(idx.shape[0] * 2, dtype=np.float32).reshape(-1, 2)
    for g in fx["per_gpu"]:
        pm = oracle.permute(X, idx, gate, fx["E"], pl, g["dev"])
        np.testing.assert_array_equal(pm["group_offsets"], g["group_offsets"])
        np.testing.assert_array_equal(pm["row_token"], g["row_token"])
        np.testing.assert_array_equal(pm["token_row"], g["token_row"])
        np.testing.assert_array_equal(pm["send_counts"], fx["send_counts"])
        np.testing.assert_array_equal(pm["x_perm"], X[g["row_token"]])


def test_send_counts_are_eq1_load_and_eq3_volume():
    r = _rng(6)
    T, E, k, G, d = 400, 20, 2, 4, 8
    idx = _random_routing(r, T, E, k)
    pl = np.zeros((E, G), np.uint8)
    host = r.integers(0, G, E)
    pl[np.arange(E), host] = 1
    pm = oracle.permute(None, idx, np.ones((T, k)), E, pl, 1)
    W = np.bincount(idx.ravel(), minlength=E)
    lam = [sum(W[i] for i in range(E) if host[i] == j) for j in range(G)]     # Eq. (1)
    np.testing.assert_array_equal(pm["send_counts"], lam)
    D = [d * sum(W[i] for i in range(E) if host[i] == j) for j in range(G)]   # Eq. (3)
    np.testing.assert_array_equal(d * pm["send_counts"], D)


def test_permute_rejects_bad_placement_and_capacity():
    idx = np.array([[0, 1], [1, 2]], np.int32)
    pl = np.array([[1, 0], [0, 1], [0, 0]], np.uint8)          # expert 2 has no host
    with pytest.raises(ValueError):
        oracle.permute(None, idx, np.ones((2, 2)), 3, pl, 0)
    pl[2, 0] = 1
    with pytest.raises(ValueError):
        oracle.permute(None, idx, np.ones((2, 2)), 3, pl, 0, cap_rows=1)


def test_permute_device_without_rows_and_empty_batch():
    idx = np.array([[0, 1], [1, 0]], np.int32)
    pl = np.array([[1, 0, 0], [1, 0, 0], [0, 1, 1]], np.uint8)
    pm = oracle.permute(None, idx, np.ones((2, 2)), 3, pl, 2)
    assert pm["rows"] == 0 and np.all(pm["token_row"] == -1)
    np.testing.assert_array_equal(pm["group_offsets"], [0, 0])
    pm0 = oracle.permute(None, np.zeros((0, 2), np.int32), np.zeros((0, 2)), 3, pl, 0)
    assert pm0["rows"] == 0 and np.all(pm0["send_counts"] == 0)


# ----------------------------------------------------------------------------- expert FFN
def _torch_swiglu(x, W13, W2):
    x = torch.from_numpy(np.asarray(x, np.float64))
    W13 = torch.from_numpy(np.asarray(W13, np.float64))
    W2 = torch.from_numpy(np.asarray(W2, np.float64))
    f = W13.shape[0] // 2
    h = torch.nn.functional.silu(x @ W13[:f].T) * (x @ W13[f:].T)
    return (h @ W2.T).numpy()


def test_ffn_matches_torch_float64_silu_and_matmul():
    r = _rng(7)
    n, d, f = 13, 24, 40                 # d != f catches a transposed W2
    x = _bf16_exact(r.standard_normal((n, d)))
    W13 = _bf16_exact(0.3 * r.standard_normal((2 * f, d)))
    W2 = _bf16_exact(0.3 * r.standard_normal((d, f)))
    got = oracle.expert_ffn(x, W13, W2)
    np.testing.assert_allclose(got, _torch_swiglu(x, W13, W2), rtol=1e-12, atol=1e-12)
    # gate and up halves are not interchangeable
    swapped = np.concatenate([W13[f:], W13[:f]])
    assert np.max(np.abs(got - _torch_swiglu(x, swapped, W2))) > 1e-3


def test_ffn_silu_closed_forms():
    r = _rng(8)
    n, d, f = 6, 10, 7
    x = r.standard_normal((n, d)).astype(np.float32)
    W1 = r.standard_normal((f, d)).astype(np.float32)
    W3 = r.standard_normal((f, d)).astype(np.float32)
    W2 = r.standard_normal((d, f)).astype(np.float32)
    x64, W1d, W3d, W2d = (a.astype(np.float64) for a in (x, W1, W3, W2))
    # SiLU(a) - SiLU(-a) = a  (since sigmoid(a) + sigmoid(-a) = 1): a bilinear closed form
    y_pos = oracle.expert_ffn(x, np.concatenate([W1, W3]), W2)
    y_neg = oracle.expert_ffn(x, np.concatenate([-W1, W3]), W2)
    bilinear = ((x64 @ W1d.T) * (x64 @ W3d.T)) @ W2d.T
    np.testing.assert_allclose(y_pos - y_neg, bilinear, rtol=1e-11, atol=1e-11)
    # large positive gate pre-activation: SiLU(a) = a in double; large negative: 0
    big = np.zeros((1, d), np.float32)
    big[0, 0] = 1.0
    W1b = np.zeros((f, d), np.float32)
    W1b[:, 0] = 64.0
    yb = oracle.expert_ffn(big, np.concatenate([W1b, W3]), W2)
    np.testing.assert_allclose(yb[0], W2d @ (64.0 * W3d[:, 0]), rtol=1e-14, atol=0)
    yn = oracle.expert_ffn(big, np.concatenate([-W1b, W3]), W2)
    assert np.max(np.abs(yn)) < 1e-20
    # scaling W2 by two doubles the output exactly
    np.testing.assert_array_equal(oracle.expert_ffn(x, np.concatenate([W1, W3]), 2 * W2), 2 * y_pos)


# ----------------------------------------------------------------------------- weighted sum
def test_combine_identity_experts_return_the_input():
    r = _rng(9)
    T, E, k, d = 40, 6, 3, 5
    X = r.standard_normal((T, d)).astype(np.float32)
    L = r.standard_normal((T, E)).astype(np.float32)
    idx, g = oracle.topk(L, k)
    pm = oracle.permute(X, idx, g, E, np.ones((E, 1), np.uint8), 0)
    y = oracle.combine(pm["x_perm"], pm["token_row"], g, None, T, d, k)
    np.testing.assert_allclose(y, X, rtol=0, atol=1e-14 * np.abs(X).max() * k)
    ys = r.standard_normal((T, d))
    y2 = oracle.combine(pm["x_perm"], pm["token_row"], g, ys, T, d, k)
    np.testing.assert_allclose(y2, X + ys, rtol=0, atol=1e-13)


def test_worked_three_expert_example():
    """Hand-derived: one-hot tokens make the logits equal router entries, so the
    gates are logistic functions of logit gaps and each expert (f = 1) reduces to
    v * SiLU(w1) * w3 with scalars read off the weights."""
    X = np.array([[1, 0], [0, 1]], np.float32)
    Wr = np.array([[0.0, 0.0], [1.0, 1.0], [0.5, -2.0]], np.float32)   # logits t0=[0,1,.5], t1=[0,1,-2]
    W13 = [np.array([[1.0, -1.0], [2.0, 0.5]], np.float32),            # rows: W1 (gate), W3 (up)
           np.array([[0.0, 3.0], [1.0, 1.0]], np.float32),
           np.array([[-2.0, 1.0], [0.25, 4.0]], np.float32)]
    W2 = [np.array([[1.0], [2.0]], np.float32),
          np.array([[-1.0], [0.5]], np.float32),
          np.array([[4.0], [1.0]], np.float32)]
    out = oracle.layer_share(X, Wr, None, 2, np.ones((3, 1), np.uint8), 0, W13, W2)
    sig = lambda z: 1.0 / (1.0 + math.exp(-z))
    silu = lambda z: z * sig(z)
    np.testing.assert_array_equal(out["idx"], [[1, 2], [1, 0]])
    g0 = sig(0.5)            # token 0: experts 1 (logit 1) and 2 (logit 0.5)
    g1 = sig(1.0)            # token 1: experts 1 (logit 1) and 0 (logit 0)
    np.testing.assert_allclose(out["gate"], [[g0, 1 - g0], [g1, 1 - g1]], rtol=1e-15)
    # token 0 reads column 0 of each expert's W13; token 1 reads column 1
    e1_t0 = silu(0.0) * 1.0 * np.array([-1.0, 0.5])
    e2_t0 = silu(-2.0) * 0.25 * np.array([4.0, 1.0])
    e1_t1 = silu(3.0) * 1.0 * np.array([-1.0, 0.5])
    e0_t1 = silu(-1.0) * 0.5 * np.array([1.0, 2.0])
    np.testing.assert_allclose(out["y"][0], g0 * e1_t0 + (1 - g0) * e2_t0, rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(out["y"][1], g1 * e1_t1 + (1 - g1) * e0_t1, rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(out["counts"], [1, 2, 1])


@pytest.mark.parametrize("cfg_name", ["tiny_fp32", "custom_shared"])
def test_whole_layer_is_the_textbook_per_token_sum(cfg_name):
    """Sec. II-A: y_t = sum over selected experts of gate * FFN_e(x_t) (+ shared experts),
    computed per token over ALL experts with a membership mask (no packaging)."""
    if cfg_name == "tiny_fp32":
        cfg = synth.CONFIGS["tiny_fp32"]
        T = 24
    else:
        cfg = synth.custom_config(d=32, E=6, k=3, f=16, shared_f=(24, 8), T=20, zipf=1.2)
        T = 20
    inp = synth.make_layer(cfg, T, seed=3, experts="all")
    X = inp.X.float().numpy()
    Wr = inp.Wr.float().numpy()
    b = inp.bias.numpy()
    W13 = [w.float().numpy() for w in inp.w13]
    W2 = [w.float().numpy() for w in inp.w2]
    sh = [(a.float().numpy(), c.float().numpy()) for a, c in inp.shared]
    out = oracle.layer_share(X, Wr, b, cfg.k, np.ones((cfg.E, 1), np.uint8), 0, W13, W2, shared=sh)
    ref = np.zeros((T, cfg.d))
    for t in range(T):
        for e in range(cfg.E):
            hit = np.nonzero(out["idx"][t] == e)[0]
            if len(hit):
                ref[t] += out["gate"][t, hit[0]] * _torch_swiglu(X[t:t + 1], W13[e], W2[e])[0]
        for (a, c) in sh:
            ref[t] += _torch_swiglu(X[t:t + 1], a, c)[0]
    np.testing.assert_allclose(out["y"], ref, rtol=1e-11, atol=1e-12)
