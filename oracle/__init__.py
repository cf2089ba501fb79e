"""CPU oracle for one GPU's share of a Director MoE layer -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never does, and this package never imports the product.

The arithmetic lives in ``moe_oracle.c`` (plain C, double precision, OpenMP
over independent outputs).  This module only compiles it with gcc, loads it
with ctypes and marshals numpy arrays.  The steps follow the paper
(arXiv 2607.08782):

* gate scores and top-k routing, weighted sum of expert outputs  -- Sec. II-A
* packaging tokens for the GPUs that host their experts           -- Sec. II-B
* workload matrix W, per-GPU load (Eq. 1), dispatch volume (Eq. 3),
  placement constraints (Eq. 6d, 6e)                              -- Sec. VI

``oracle.placement`` is the plain reference of the placement model itself
(Eq. 1-5, the LP relaxation's optimum, exhaustive search on tiny inputs).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()


def build(force: bool = True) -> str:
    """Compile moe_oracle.c into liboracle.so with gcc (-O2, IEEE semantics, OpenMP)."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
           "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        i32 = ctypes.c_int
        lib.orc_router_logits.argtypes = [P, P, P, i64, i64, i64, P]
        lib.orc_router_logits.restype = None
        lib.orc_topk.argtypes = [P, i64, i32, i32, i32, P, P]
        lib.orc_topk.restype = i32
        lib.orc_histogram.argtypes = [P, i64, i32, i32, P, P]
        lib.orc_histogram.restype = None
        lib.orc_permute.argtypes = [P, i64, i64, P, P, i32, i32, P, i32, i32,
                                    i64, P, P, P, P, P, P]
        lib.orc_permute.restype = i64
        lib.orc_expert_ffn.argtypes = [P, i64, i64, i64, P, P, P]
        lib.orc_expert_ffn.restype = None
        lib.orc_combine.argtypes = [P, P, P, P, i64, i64, i32, P]
        lib.orc_combine.restype = None
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = i32
        lib.orc_set_num_threads.argtypes = [i32]
        lib.orc_set_num_threads.restype = None
        _lib = lib
        return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's OpenMP loops from now on (n >= 1)."""
    _load().orc_set_num_threads(int(n))


def router_logits(X, Wr, bias=None) -> np.ndarray:
    """logits[t, e] = sum_i X[t, i] * Wr[e, i] + bias[e], in float64 (Sec. II-A)."""
    X = _c(X, np.float32)
    Wr = _c(Wr, np.float32)
    T, d = X.shape
    E = Wr.shape[0]
    assert Wr.shape[1] == d
    b = None if bias is None else _c(bias, np.float32)
    out = np.empty((T, E), np.float64)
    _load().orc_router_logits(_p(X), _p(Wr), _p(b), T, d, E, _p(out))
    return out


def topk(logits_f32, k: int, renorm: bool = True):
    """Top-k on fp32 logits (ties to the lower index), gates in float64 (Sec. II-A).

    Returns (idx int32 [T, k], gate float64 [T, k]).
    """
    L = _c(logits_f32, np.float32)
    T, E = L.shape
    idx = np.empty((T, k), np.int32)
    gate = np.empty((T, k), np.float64)
    rc = _load().orc_topk(_p(L), T, E, k, 1 if renorm else 0, _p(idx), _p(gate))
    if rc != 0:
        raise ValueError("oracle topk: bad k=%d for E=%d" % (k, E))
    return idx, gate


def histogram(idx, E: int, with_coact: bool = False):
    """Per-expert counts (W of Sec. VI-A summed over source GPUs) and co-activation."""
    idx = _c(idx, np.int32)
    T, k = idx.shape
    counts = np.empty(E, np.int64)
    coact = np.empty((E, E), np.int64) if with_coact else None
    _load().orc_histogram(_p(idx), T, k, E, _p(counts), _p(coact))
    return counts, coact


def local_slots(placement, dev: int):
    """Experts hosted on `dev`, ascending id (local slot order)."""
    placement = np.asarray(placement)
    return [int(e) for e in np.nonzero(placement[:, dev])[0]]


def permute(X, idx, gate, E: int, placement, dev: int, cap_rows=None, with_x: bool = True):
    """Package tokens for the experts on GPU `dev` (Sec. II-B, Eq. 1, Eq. 3).

    Returns a dict with rows, group_offsets, row_token, row_gate, token_row,
    send_counts and (if with_x) x_perm.  Raises on an invalid placement.
    """
    idx = _c(idx, np.int32)
    gate = _c(gate, np.float64)
    T, k = idx.shape
    placement = _c(placement, np.uint8)
    assert placement.shape[0] == E
    G = placement.shape[1]
    if X is not None:
        X = _c(X, np.float32)
        d = X.shape[1]
    else:
        d = 0
        with_x = False
    n_local = int(placement[:, dev].sum()) if 0 <= dev < G else 0
    if cap_rows is None:
        cap_rows = T * k
    group_offsets = np.empty(n_local + 1, np.int64)
    row_token = np.empty(max(cap_rows, 1), np.int64)
    row_gate = np.empty(max(cap_rows, 1), np.float64)
    token_row = np.empty((T, k), np.int64)
    send_counts = np.empty(G, np.int64)
    x_perm = np.empty((max(cap_rows, 1), d), np.float32) if with_x else None
    rows = _load().orc_permute(_p(X), T, d, _p(idx), _p(gate), k, E, _p(placement), G, dev,
                               cap_rows, _p(x_perm), _p(group_offsets), _p(row_token),
                               _p(row_gate), _p(token_row), _p(send_counts))
    if rows == -2:
        raise ValueError("oracle permute: an expert has no host GPU")
    if rows == -3:
        raise ValueError("oracle permute: rows exceed cap_rows")
    if rows < 0:
        raise ValueError("oracle permute: bad argument")
    out = dict(rows=int(rows), group_offsets=group_offsets, row_token=row_token[:rows],
               row_gate=row_gate[:rows], token_row=token_row, send_counts=send_counts)
    if with_x:
        out["x_perm"] = x_perm[:rows]
    return out


def expert_ffn(x, W13, W2) -> np.ndarray:
    """SwiGLU expert FFN on rows x [n, d] (Sec. II-A experts), float64 result [n, d]."""
    x = _c(x, np.float32)
    W13 = _c(W13, np.float32)
    W2 = _c(W2, np.float32)
    n, d = x.shape if x.ndim == 2 else (0, W2.shape[0])
    f = W13.shape[0] // 2
    assert W13.shape == (2 * f, d) and W2.shape == (d, f)
    y = np.empty((n, d), np.float64)
    if n:
        _load().orc_expert_ffn(_p(x), n, d, f, _p(W13), _p(W2), _p(y))
    return y


def combine(y_perm, token_row, gate, y_shared, T: int, d: int, k: int) -> np.ndarray:
    """y[t] = sum_r gate[t, r] * y_perm[token_row[t, r]] + y_shared[t] (Sec. II-A)."""
    y_perm = _c(y_perm, np.float64).reshape(-1, d) if d else _c(y_perm, np.float64)
    token_row = _c(token_row, np.int64)
    gate = _c(gate, np.float64)
    ys = None if y_shared is None else _c(y_shared, np.float64)
    y = np.empty((T, d), np.float64)
    _load().orc_combine(_p(y_perm), _p(token_row), _p(gate), _p(ys), T, d, k, _p(y))
    return y


def layer_share(X, Wr, bias, k, placement, dev, w13_local, w2_local,
                shared=(), renorm=True, with_coact=False, logits_f32=None):
    """The whole share of one MoE layer on GPU `dev`, step by step.

    w13_local / w2_local are float arrays in local slot order; shared is a
    sequence of (W13, W2) pairs of always-on experts.  If logits_f32 is given,
    selection uses it instead of the oracle's own logits (rounded to fp32).
    Returns a dict of every intermediate.
    """
    X = _c(X, np.float32)
    T, d = X.shape
    E = np.asarray(Wr).shape[0]
    out = {}
    out["logits"] = router_logits(X, Wr, bias)
    sel = out["logits"].astype(np.float32) if logits_f32 is None else _c(logits_f32, np.float32)
    out["idx"], out["gate"] = topk(sel, k, renorm)
    out["counts"], out["coact"] = histogram(out["idx"], E, with_coact)
    pm = permute(X, out["idx"], out["gate"], E, placement, dev)
    out.update(pm)
    y_perm = np.zeros((pm["rows"], d), np.float64)
    go = pm["group_offsets"]
    for s in range(len(go) - 1):
        a, b = int(go[s]), int(go[s + 1])
        if b > a:
            y_perm[a:b] = expert_ffn(pm["x_perm"][a:b], w13_local[s], w2_local[s])
    out["y_perm"] = y_perm
    ys = None
    for (w13s, w2s) in shared:
        part = expert_ffn(X, w13s, w2s)
        ys = part if ys is None else ys + part
    out["y_shared"] = ys
    out["y"] = combine(y_perm, pm["token_row"], out["gate"], ys, T, d, k)
    return out
