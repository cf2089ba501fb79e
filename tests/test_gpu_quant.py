"""Quantized routing predictor on the GPU vs the oracle (Sec. V-A; marked `gpu`).

* moe_quantize_e4m3: codes and scales bit-exact against oracle.quant on the
  same bf16 / fp32 values (zero rows, subnormal codes, ragged widths).
* moe_route_topk_e4m3: every gate score against the oracle's exact float64
  scores within the fp32 summation bound; top-k indices bit-exact and gates
  within 1e-5 against oracle.topk on the GPU's own scores (the decision is
  taken on the same fp32 values on both sides).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import quant as oq
from paper_2607_08782_amd import moe, synth

from parity import GATE_TOL, close, np32, say

pytestmark = pytest.mark.gpu

U = 2.0 ** -24          # fp32 unit roundoff


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    moe.load_library()
    yield


def _check_quant(x: torch.Tensor):
    q, s = moe.moe_quantize_e4m3(x)
    torch.cuda.synchronize()
    rq, rs = oq.quantize_rows(np32(x))
    np.testing.assert_array_equal(s.cpu().numpy(), rs)
    np.testing.assert_array_equal(q.cpu().numpy(), rq)
    return q, s


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("rows,cols", [(1, 1), (7, 72), (5, 100), (300, 256), (33, 4096),
                                       (3, 12296), (0, 64)])
def test_quantize_is_bit_exact(dtype, rows, cols):
    say("[quant]", dtype, rows, cols)
    g = torch.Generator().manual_seed(rows * 131 + cols)
    x = torch.randn(rows, cols, generator=g).to(dtype)
    if rows > 2:
        x[1] = 0.0                                   # zero row: scale 1, all codes 0
        x[2] *= 1e-3
        x[2, 0] = 50.0                               # one large value: the rest lands on subnormals
    _check_quant(x.cuda())


def test_quantize_unaligned_rows_take_the_element_path():
    g = torch.Generator().manual_seed(5)
    flat = torch.randn(9 * 256 + 1, generator=g).to(torch.bfloat16).cuda()
    x = flat[1:].view(9, 256)                        # 2-byte offset: no 16-byte loads
    assert x.is_contiguous() and x.data_ptr() % 16 != 0
    _check_quant(x)


def _scores_bound(xq, sx, wq, sw, bias, d):
    """Per-element bound of an fp32 sum of d exact products in any order
    (2u per addition, to allow truncating adders), plus the two scale products
    and the bias addition."""
    A = np.abs(oq.e4m3_decode(xq)) @ np.abs(oq.e4m3_decode(wq)).T
    A = A * np.asarray(sx, np.float64)[:, None] * np.asarray(sw, np.float64)[None, :]
    b = 0.0 if bias is None else np.abs(np.asarray(bias, np.float64))[None, :]
    return (2 * d + 8) * U * A + 4 * U * (A + b) + 1e-30


def _check_route(X: torch.Tensor, Wr: torch.Tensor, bias, k: int):
    T, d = X.shape
    xq, sx = _check_quant(X)
    wq, sw = _check_quant(Wr)
    logits, idx, gate = moe.moe_route_topk_e4m3(xq, sx, wq, sw, bias, k, renorm=True)
    torch.cuda.synchronize()
    b = None if bias is None else bias.cpu().numpy()
    xq_, sx_, wq_, sw_ = xq.cpu().numpy(), sx.cpu().numpy(), wq.cpu().numpy(), sw.cpu().numpy()
    ref = oq.q_logits(xq_, sx_, wq_, sw_, b)
    got = logits.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    bound = _scores_bound(xq_, sx_, wq_, sw_, b, d)
    worst = np.unravel_index(np.argmax(err - bound), err.shape) if err.size else None
    assert err.size == 0 or np.all(err <= bound), "score %s: err %.3e > bound %.3e" % (
        worst, err[worst], bound[worst])
    ridx, rgate = oracle.topk(got.astype(np.float32), k, renorm=True)
    np.testing.assert_array_equal(idx.cpu().numpy(), ridx)
    close(np32(gate), rgate, GATE_TOL, "gates")
    return idx


SMALL = [  # (T, d, E, k, bias)
    (1, 64, 8, 2, True),
    (77, 256, 60, 4, True),
    (300, 2048, 64, 6, False),
    (33, 128, 256, 8, True),
    (130, 192, 33, 3, True),
    (65, 4096, 8, 2, True),
    (0, 128, 16, 2, True),
    (12300, 256, 130, 5, True),      # >= 192 64-token tiles over > 32 experts: the tiled kernel
    (12290, 128, 40, 3, False),
    (12225, 256, 96, 8, True),
]


@pytest.mark.parametrize("T,d,E,k,use_bias", SMALL)
def test_quantized_scores_and_topk_every_element(T, d, E, k, use_bias):
    say("[qroute]", T, d, E, k, use_bias)
    g = torch.Generator().manual_seed(T * 7 + d + E)
    X = torch.randn(T, d, generator=g).to(torch.bfloat16).cuda()
    Wr = (torch.randn(E, d, generator=g) * 0.02).to(torch.bfloat16).cuda()
    bias = (torch.randn(E, generator=g) * 0.5).cuda() if use_bias else None
    _check_route(X, Wr, bias, k)


FULL = [("mixtral_8x7b", "prefill"), ("deepseek_v2_lite", "prefill"),
        ("qwen15_moe_a27b", "batch"), ("qwen3_30b_a3b", "prefill")]


@pytest.mark.parametrize("name,regime", FULL)
def test_model_shaped_predictor_every_element(name, regime):
    cfg = synth.CONFIGS[name]
    T = cfg.T(regime)
    say("[qroute-full]", name, regime, "T=%d" % T)
    inp = synth.make_layer(cfg, T, seed=0, device="cuda", experts="none")
    idx = _check_route(inp.X, inp.Wr, inp.bias, cfg.k)
    # the predictor ranks like the full-precision gate on most assignments
    _, ref_idx, _ = moe.moe_route_topk(inp.X, inp.Wr, inp.bias, cfg.k, renorm=True,
                                      want_logits=False)
    rate = oq.match_rate(idx.cpu().numpy(), ref_idx.cpu().numpy())
    say("  top-%d match rate vs bf16 routing: %.4f" % (cfg.k, rate))
    assert rate > 0.5
