"""Pins of the quantized-predictor oracle (Sec. V-A; accuracy metric of Sec. VIII).

E4M3 decoding and round-to-nearest-even encoding are checked against torch's
independent float8_e4m3fn conversion over every code and a sweep of fp32
values (ties and subnormals included); the per-row scaling and the gate
scores against closed forms; the match rate against hand counts.
"""
import numpy as np
import pytest
import torch

from oracle import quant as oq


def test_every_code_decodes_like_torch_float8_e4m3fn():
    codes = np.arange(256, dtype=np.uint8)
    ours = oq.e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().double().numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])
    assert oq.e4m3_decode(0x38) == 1.0 and oq.e4m3_decode(0x7E) == 448.0
    assert oq.e4m3_decode(0x01) == 2.0 ** -9 and oq.e4m3_decode(0x08) == 2.0 ** -6


def test_rounding_matches_torch_on_a_sweep_with_ties_and_subnormals():
    rng = np.random.default_rng(0)
    v = np.concatenate([
        rng.uniform(-448, 448, 20000),
        np.ldexp(rng.uniform(-1, 1, 20000), rng.integers(-12, 9, 20000)),
        # exact midpoints between neighbouring codes (ties) and the subnormal range
        (oq.e4m3_decode(np.arange(0, 0x7E)) + oq.e4m3_decode(np.arange(1, 0x7F))) / 2,
        -(oq.e4m3_decode(np.arange(0, 0x7E)) + oq.e4m3_decode(np.arange(1, 0x7F))) / 2,
    ]).astype(np.float32)
    ours = oq.e4m3_decode(oq.e4m3_encode(v))
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).float().double().numpy()
    assert np.array_equal(ours, ref)


@pytest.mark.parametrize("v,want", [(1.0625, 1.0), (1.1875, 1.25), (2.0 ** -10, 0.0),
                                    (3 * 2.0 ** -11, 2.0 ** -9), (460.0, 448.0), (1e6, 448.0),
                                    (-1e6, -448.0), (-2.0 ** -11, 0.0)])
def test_named_roundings(v, want):
    assert oq.e4m3_decode(oq.e4m3_encode(np.float32(v))) == want


def test_row_scale_maps_the_largest_magnitude_to_448_and_zero_rows_to_zero():
    x = np.array([[0.5, -2.0, 1.0], [0.0, 0.0, 0.0], [3.0, 0.75, -0.25]], np.float32)
    q, s = oq.quantize_rows(x)
    assert s.dtype == np.float32
    assert s[0] == np.float32(2.0) / np.float32(448) and s[1] == 1.0
    assert q[0, 1] == 0xFE and q[2, 0] == 0x7E and not q[1].any()
    # the dequantised rows are within half an E4M3 step (relative 1/16) of the input
    back = oq.e4m3_decode(q) * s[:, None]
    assert np.all(np.abs(back - x) <= np.abs(x) / 16 + 1e-12)


def test_gate_scores_of_one_hot_rows_are_the_scale_products_plus_bias():
    xq = np.zeros((2, 4), np.uint8)
    wq = np.zeros((3, 4), np.uint8)
    xq[0, 1] = xq[1, 3] = 0x38            # 1.0
    wq[0, 1] = 0x40                       # 2.0
    wq[2, 3] = 0xB8                       # -1.0
    sx = np.array([0.5, 4.0], np.float32)
    sw = np.array([0.25, 1.0, 2.0], np.float32)
    L = oq.q_logits(xq, sx, wq, sw, bias=np.array([1.0, 2.0, 3.0]))
    assert np.array_equal(L, [[1.0 + 0.5 * 0.25 * 2.0, 2.0, 3.0], [1.0, 2.0, 3.0 - 4.0 * 2.0]])


def test_match_rate_counts_set_overlap():
    assert oq.match_rate([[0, 1], [2, 3]], [[1, 0], [2, 4]]) == 0.75
    assert oq.match_rate([[5, 6, 7]], [[1, 2, 3]]) == 0.0
