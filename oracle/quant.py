"""Plain reference of the quantized routing predictor -- TEST INFRASTRUCTURE.

Only ``tests/`` and the CPU-baseline leg of the benchmark may import this
module; the product never does, and this module imports nothing from it.

Director's quantized predictor (Sec. V-A) is a low-bit replica whose gate
scores rank experts almost as the full-precision model does; its accuracy is
the top-k match rate between predicted and true routing (Sec. VIII, metrics).
The replica here quantizes both the router weights and the token activations
to FP8 E4M3 (the OCP 8-bit float: 1 sign, 4 exponent bits with bias 7, 3
mantissa bits, subnormals, largest finite value 448, no infinities) with one
scale per row, by round-to-nearest-even:

    s_row = max_i |v[row][i]| / 448            (fp32; 1 when the row is zero)
    q[row][i] = E4M3_RNE(v[row][i] / s_row)    (the division in fp32)
    logits_q[t][e] = s_x[t] * s_w[e] * sum_i dec(qx[t][i]) * dec(qw[e][i]) + b[e]

Every step is written out plainly: the E4M3 grid is enumerated, rounding is
to the nearest grid value with ties to the even code, and the dot products
are exact in float64 (E4M3 products and their sums are exact there).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """Value of every E4M3 code (NaN for the two NaN codes)."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    exp = (c >> 3) & 0xF
    man = c & 0x7
    normal = np.ldexp(1.0 + man / 8.0, exp - 7)
    sub = np.ldexp(man / 8.0, -6)
    v = np.where(exp == 0, sub, normal)
    v = np.where((exp == 15) & (man == 7), np.nan, v)
    return sign * v


# the non-negative finite grid, ascending, with its codes
_CODES = np.arange(0x7F, dtype=np.int64)            # 0x00 .. 0x7E (0x7F is NaN)
_GRID = e4m3_decode(_CODES)


def e4m3_encode(v) -> np.ndarray:
    """Round finite values to the nearest E4M3 value, ties to the even code;
    magnitudes beyond 448 saturate to 448."""
    v = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(v), E4M3_MAX)
    hi = np.searchsorted(_GRID, a, side="left")      # first grid value >= a
    hi = np.clip(hi, 0, len(_GRID) - 1)
    lo = np.clip(hi - 1, 0, len(_GRID) - 1)
    d_lo = a - _GRID[lo]
    d_hi = _GRID[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (_CODES[hi] % 2 == 0))
    pick_hi |= (_GRID[hi] == a)
    code = np.where(pick_hi, _CODES[hi], _CODES[lo])
    code = np.where((v < 0) & (code != 0), code | 0x80, code)
    return code.astype(np.uint8)


def quantize_rows(v) -> tuple:
    """Per-row E4M3 codes and fp32 scales of a 2-D array (read as fp32)."""
    v32 = np.asarray(v, dtype=np.float32)
    amax = np.max(np.abs(v32), axis=1) if v32.shape[1] else np.zeros(v32.shape[0], np.float32)
    scale = np.where(amax > 0, (amax / np.float32(E4M3_MAX)).astype(np.float32), np.float32(1.0))
    ratio = (v32 / scale[:, None]).astype(np.float32)      # fp32 division, as the kernel does
    return e4m3_encode(ratio), scale.astype(np.float32)


def q_logits(xq, sx, wq, sw, bias=None) -> np.ndarray:
    """Gate scores of the quantized replica, float64."""
    X = e4m3_decode(xq)
    Wd = e4m3_decode(wq)
    L = (X @ Wd.T) * np.asarray(sx, np.float64)[:, None] * np.asarray(sw, np.float64)[None, :]
    if bias is not None:
        L = L + np.asarray(bias, np.float64)[None, :]
    return L


def match_rate(pred_idx, true_idx) -> float:
    """Mean over tokens of |predicted top-k  intersect  true top-k| / k."""
    p = np.asarray(pred_idx)
    t = np.asarray(true_idx)
    k = t.shape[1]
    hits = [len(set(a.tolist()) & set(b.tolist())) for a, b in zip(p, t)]
    return float(np.mean(hits) / k) if len(hits) else 1.0
