"""Thin Python binding of libmoe.so (the C ABI in include/moe.h).

Argument marshalling only: every function checks that tensors live on the
GPU with the expected dtype and layout, allocates missing outputs with torch
(device memory is all torch is used for), and calls the C entry point of the
same name on torch's current HIP stream.  All arithmetic runs in the HIP
kernels.  If the library is not built this module raises; there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoe.so")

MOE_F32, MOE_BF16 = 0, 1
MOE_OK, MOE_ERR_ARG, MOE_ERR_PLACEMENT, MOE_ERR_SHAPE, MOE_ERR_DEVICE = 0, 1, 2, 3, 4
MOE_RENORM, MOE_LOGITS_IN = 1, 2
MOE_FFN_GATE_UP, MOE_FFN_DOWN, MOE_FFN_SMALL_GROUPS, MOE_FFN_LARGE_GROUPS = 1, 2, 4, 8
MOE_MAX_E, MOE_MAX_K, MOE_MAX_G, MOE_MAX_GROUPS = 256, 16, 64, 128
MOE_PERMUTE_NOALLOC_MAX_WS = 4 << 20

EXPORTS = ("moe_status_string", "moe_route_topk", "moe_route_topk_ws_bytes",
           "moe_expert_histogram", "moe_permute_ws_bytes",
           "moe_permute", "moe_permute_noalloc", "moe_grouped_ffn_ws_bytes", "moe_grouped_ffn",
           "moe_grouped_ffn_products", "moe_grouped_ffn_combine",
           "moe_grouped_ffn_rows", "moe_grouped_ffn_rows_products", "moe_grouped_ffn_rows_shared",
           "moe_combine", "moe_combine_shared",
           "moe_quantize_e4m3", "moe_route_topk_e4m3")

_lib = None


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (status %d)" % (fn, status_string(status), status))


def load_library(path: str = LIB_PATH):
    """Load libmoe.so and declare every exported signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libmoe.so is not built (%s); run __graft_entry__.build()" % path)
    lib = ctypes.CDLL(path)
    P, I, L, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    lib.moe_status_string.argtypes = [I]
    lib.moe_status_string.restype = ctypes.c_char_p
    lib.moe_route_topk.argtypes = [P, I, P, P, L, I, I, I, I, P, P, P, P, S, P]
    lib.moe_route_topk.restype = I
    lib.moe_route_topk_ws_bytes.argtypes = [I, L, I, I, I]
    lib.moe_route_topk_ws_bytes.restype = S
    lib.moe_expert_histogram.argtypes = [P, L, I, I, P, P, P]
    lib.moe_expert_histogram.restype = I
    lib.moe_permute_ws_bytes.argtypes = [L, I, I]
    lib.moe_permute_ws_bytes.restype = S
    lib.moe_permute.argtypes = [P, I, P, P, P, L, I, I, I, P, I, I, I, P, L, P, P, P, P, P, P, S, P]
    lib.moe_permute.restype = I
    lib.moe_permute_noalloc.argtypes = [P, I, P, P, P, L, I, I, I, P, I, I, I, P, L, P, P, P, P, P,
                                        P]
    lib.moe_permute_noalloc.restype = I
    lib.moe_grouped_ffn_ws_bytes.argtypes = [I, L, I, I, I]
    lib.moe_grouped_ffn_ws_bytes.restype = S
    lib.moe_grouped_ffn.argtypes = [P, I, P, I, P, P, I, I, L, P, P, S, P]
    lib.moe_grouped_ffn.restype = I
    lib.moe_grouped_ffn_products.argtypes = [P, I, P, I, P, P, I, I, L, P, P, S, I, P]
    lib.moe_grouped_ffn_products.restype = I
    lib.moe_grouped_ffn_combine.argtypes = [P, I, P, I, P, P, I, I, L, P, P, P, L, I, P, P, S, P]
    lib.moe_grouped_ffn_combine.restype = I
    lib.moe_grouped_ffn_rows.argtypes = [P, L, P, I, P, I, P, P, I, I, L, P, P, S, P]
    lib.moe_grouped_ffn_rows.restype = I
    lib.moe_grouped_ffn_rows_products.argtypes = [P, L, P, I, P, I, P, P, I, I, L, P, P, S, I, P]
    lib.moe_grouped_ffn_rows_products.restype = I
    lib.moe_grouped_ffn_rows_shared.argtypes = [P, L, P, I, P, I, I, P, P, I, I, L, P, P, S, I, P]
    lib.moe_grouped_ffn_rows_shared.restype = I
    lib.moe_combine.argtypes = [P, I, P, P, P, L, I, I, P, P]
    lib.moe_combine.restype = I
    lib.moe_combine_shared.argtypes = [P, I, P, P, P, I, L, I, I, P, P]
    lib.moe_combine_shared.restype = I
    lib.moe_quantize_e4m3.argtypes = [P, I, L, I, P, P, P]
    lib.moe_quantize_e4m3.restype = I
    lib.moe_route_topk_e4m3.argtypes = [P, P, P, P, P, L, I, I, I, I, P, P, P, P]
    lib.moe_route_topk_e4m3.restype = I
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().moe_status_string(int(status)).decode()


def _check(fn: str, status: int):
    if status != MOE_OK:
        raise MoeError(fn, status)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise TypeError("unsupported element type %s (float32 or bfloat16)" % t.dtype)


def _dev(t: Optional[torch.Tensor], name: str, dtype=None):
    """Device pointer of a contiguous GPU tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def moe_route_topk(x: Optional[torch.Tensor], w_router: Optional[torch.Tensor],
                   bias: Optional[torch.Tensor], k: int, *, E: Optional[int] = None,
                   renorm: bool = True, logits: Optional[torch.Tensor] = None,
                   logits_in: bool = False, want_logits: bool = True,
                   topk_idx: Optional[torch.Tensor] = None,
                   topk_gate: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                   stream=None):
    """Gate scores + top-k.  Returns (logits or None, topk_idx, topk_gate)."""
    lib = load_library()
    if logits_in:
        if logits is None:
            raise ValueError("logits_in needs logits")
        T, E_ = logits.shape
        d = 0 if x is None else x.shape[1]
        dtype = MOE_F32 if x is None else _dtype_code(x)
        device = logits.device
    else:
        T, d = x.shape
        E_ = w_router.shape[0]
        dtype = _dtype_code(x)
        if w_router.dtype != x.dtype or w_router.shape[1] != d:
            raise ValueError("w_router must be [E, d] of x's dtype")
        device = x.device
        if logits is None and want_logits:
            logits = _empty((T, E_), torch.float32, device)
    if E is not None and E != E_:
        raise ValueError("E mismatch")
    if topk_idx is None:
        topk_idx = _empty((T, k), torch.int32, device)
    if topk_gate is None:
        topk_gate = _empty((T, k), torch.float32, device)
    flags = (MOE_RENORM if renorm else 0) | (MOE_LOGITS_IN if logits_in else 0)
    need = moe_route_topk_ws_bytes(dtype, T, d, E_, flags)
    if need and ws is None:
        ws = workspace(need, device)
    st = lib.moe_route_topk(_dev(x, "x"), dtype, _dev(w_router, "w_router"),
                            _dev(bias, "bias", torch.float32), T, d, E_, k, flags,
                            _dev(logits, "logits", torch.float32),
                            _dev(topk_idx, "topk_idx", torch.int32),
                            _dev(topk_gate, "topk_gate", torch.float32), _dev(ws, "ws"),
                            0 if ws is None else ws.numel(), _stream(stream))
    _check("moe_route_topk", st)
    return logits, topk_idx, topk_gate


def moe_quantize_e4m3(x: torch.Tensor, *, q: Optional[torch.Tensor] = None,
                      scales: Optional[torch.Tensor] = None, stream=None):
    """Per-row E4M3 codes (uint8 [rows, cols]) and fp32 scales ([rows]) of x."""
    lib = load_library()
    rows, cols = x.shape
    if q is None:
        q = _empty((rows, cols), torch.uint8, x.device)
    if scales is None:
        scales = _empty((rows,), torch.float32, x.device)
    st = lib.moe_quantize_e4m3(_dev(x, "x"), _dtype_code(x), rows, cols, _dev(q, "q", torch.uint8),
                               _dev(scales, "scales", torch.float32), _stream(stream))
    _check("moe_quantize_e4m3", st)
    return q, scales


def moe_route_topk_e4m3(xq: torch.Tensor, x_scale: torch.Tensor, wq: torch.Tensor,
                        w_scale: torch.Tensor, bias: Optional[torch.Tensor], k: int, *,
                        renorm: bool = True, logits: Optional[torch.Tensor] = None,
                        topk_idx: Optional[torch.Tensor] = None,
                        topk_gate: Optional[torch.Tensor] = None, stream=None):
    """Quantized-predictor scores + top-k.  Returns (logits, topk_idx, topk_gate)."""
    lib = load_library()
    T, d = xq.shape
    E = wq.shape[0]
    if wq.shape[1] != d:
        raise ValueError("wq must be [E, d]")
    if logits is None:
        logits = _empty((T, E), torch.float32, xq.device)
    if topk_idx is None:
        topk_idx = _empty((T, k), torch.int32, xq.device)
    if topk_gate is None:
        topk_gate = _empty((T, k), torch.float32, xq.device)
    st = lib.moe_route_topk_e4m3(_dev(xq, "xq", torch.uint8), _dev(x_scale, "x_scale", torch.float32),
                                 _dev(wq, "wq", torch.uint8), _dev(w_scale, "w_scale", torch.float32),
                                 _dev(bias, "bias", torch.float32), T, d, E, k,
                                 MOE_RENORM if renorm else 0,
                                 _dev(logits, "logits", torch.float32),
                                 _dev(topk_idx, "topk_idx", torch.int32),
                                 _dev(topk_gate, "topk_gate", torch.float32), _stream(stream))
    _check("moe_route_topk_e4m3", st)
    return logits, topk_idx, topk_gate


def moe_route_topk_ws_bytes(dtype: int, T: int, d: int, E: int, flags: int) -> int:
    return int(load_library().moe_route_topk_ws_bytes(dtype, T, d, E, flags))


def moe_expert_histogram(topk_idx: torch.Tensor, E: int, *, counts: Optional[torch.Tensor] = None,
                         coact: Optional[torch.Tensor] = None, want_coact: bool = False,
                         stream=None):
    """Per-expert counts (and co-activation).  Returns (counts, coact or None)."""
    lib = load_library()
    T, k = topk_idx.shape
    if counts is None:
        counts = _empty((E,), torch.int32, topk_idx.device)
    if coact is None and want_coact:
        coact = _empty((E, E), torch.int32, topk_idx.device)
    st = lib.moe_expert_histogram(_dev(topk_idx, "topk_idx", torch.int32), T, k, E,
                                  _dev(counts, "counts", torch.int32),
                                  _dev(coact, "coact", torch.int32), _stream(stream))
    _check("moe_expert_histogram", st)
    return counts, coact


def moe_permute_ws_bytes(T: int, k: int, E: int) -> int:
    return int(load_library().moe_permute_ws_bytes(T, k, E))


def moe_grouped_ffn_ws_bytes(dtype: int, cap_rows: int, d: int, f: int, n_groups: int) -> int:
    return int(load_library().moe_grouped_ffn_ws_bytes(dtype, cap_rows, d, f, n_groups))


def workspace(nbytes: int, device) -> torch.Tensor:
    """A 256-byte aligned device workspace (torch's caching allocator aligns to 512 B)."""
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def moe_permute(x: torch.Tensor, topk_idx: torch.Tensor, topk_gate: torch.Tensor,
                counts: torch.Tensor, placement: np.ndarray, dev: int, *, E: int,
                cap_rows: Optional[int] = None, c_max: int = 0, out: Optional[dict] = None,
                ws: Optional[torch.Tensor] = None, want_send_counts: bool = True,
                copy_rows: bool = True, stream=None, noalloc: bool = False):
    """Package tokens for the experts on GPU `dev`.  Returns a dict of device tensors
    (x_perm, group_offsets, row_token, row_gate, token_row, send_counts).  With
    copy_rows=False only the row maps are produced (x_perm is not written; for
    moe_grouped_ffn_rows).  noalloc=True calls moe_permute_noalloc (no workspace:
    the library's own scratch); outputs missing from `out` are still allocated here."""
    lib = load_library()
    T, d = x.shape
    k = topk_idx.shape[1]
    placement = np.ascontiguousarray(placement, dtype=np.uint8)
    if placement.ndim != 2 or placement.shape[0] != E:
        raise ValueError("placement must be a [E, G] array")
    G = placement.shape[1]
    n_local = int((placement[:, dev] != 0).sum()) if 0 <= dev < G else 0
    if cap_rows is None:
        cap_rows = T * min(k, n_local)
    device = x.device
    o = {} if out is None else out
    if "group_offsets" not in o:
        if copy_rows:
            o["x_perm"] = _empty((max(cap_rows, 1), d), x.dtype, device)
        o["group_offsets"] = _empty((n_local + 1,), torch.int32, device)
        o["row_token"] = _empty((max(cap_rows, 1),), torch.int32, device)
        o["row_gate"] = _empty((max(cap_rows, 1),), torch.float32, device)
        o["token_row"] = _empty((T, k), torch.int32, device)
        o["send_counts"] = _empty((G,), torch.int32, device) if want_send_counts else None
    args = [_dev(x, "x") if copy_rows else None, _dtype_code(x),
            _dev(topk_idx, "topk_idx", torch.int32), _dev(topk_gate, "topk_gate", torch.float32),
            _dev(counts, "counts", torch.int32), T, d if copy_rows else 0, k, E,
            placement.ctypes.data_as(ctypes.c_void_p), G, dev, c_max,
            _dev(o["x_perm"], "x_perm", x.dtype) if copy_rows else None, cap_rows,
            _dev(o["group_offsets"], "group_offsets", torch.int32),
            _dev(o["row_token"], "row_token", torch.int32),
            _dev(o["row_gate"], "row_gate", torch.float32),
            _dev(o["token_row"], "token_row", torch.int32),
            _dev(o.get("send_counts"), "send_counts", torch.int32)]
    if noalloc:
        _check("moe_permute_noalloc", lib.moe_permute_noalloc(*args, _stream(stream)))
        return o
    if ws is None:
        ws = workspace(moe_permute_ws_bytes(T, k, E), device)
    _check("moe_permute", lib.moe_permute(*args, _dev(ws, "ws"), ws.numel(), _stream(stream)))
    return o


class WeightTable:
    """Host arrays of per-slot device pointers, as moe_grouped_ffn takes them."""

    def __init__(self, w13: Sequence[torch.Tensor], w2: Sequence[torch.Tensor]):
        if len(w13) != len(w2) or not len(w13):
            raise ValueError("need one (w13, w2) pair per group")
        self.w13 = list(w13)
        self.w2 = list(w2)
        self.f = w13[0].shape[0] // 2
        self.d = w13[0].shape[1]
        self.dtype = w13[0].dtype
        for a, b in zip(self.w13, self.w2):
            _dev(a, "w13", self.dtype)
            _dev(b, "w2", self.dtype)
            if tuple(a.shape) != (2 * self.f, self.d) or tuple(b.shape) != (self.d, self.f):
                raise ValueError("w13 must be [2f, d] and w2 [d, f] for every group")
        n = len(self.w13)
        self.p13 = (ctypes.c_void_p * n)(*[a.data_ptr() for a in self.w13])
        self.p2 = (ctypes.c_void_p * n)(*[b.data_ptr() for b in self.w2])

    def __len__(self):
        return len(self.w13)


def moe_grouped_ffn(x_perm: torch.Tensor, group_offsets: torch.Tensor, weights: WeightTable, *,
                    cap_rows: Optional[int] = None, y_perm: Optional[torch.Tensor] = None,
                    ws: Optional[torch.Tensor] = None, stream=None,
                    products: int = 3) -> torch.Tensor:
    """SwiGLU FFN of every group.  Returns y_perm [cap_rows, d].  products=1 or 2
    runs one product (moe_grouped_ffn_products: gate/up into the workspace, or down
    from it; the down call must follow a gate/up call with the same ws)."""
    lib = load_library()
    if cap_rows is None:
        cap_rows = x_perm.shape[0]
    d, f = weights.d, weights.f
    dtype = _dtype_code(x_perm)
    if x_perm.dtype != weights.dtype or x_perm.shape[1] != d:
        raise ValueError("x_perm must be [rows, d] of the weights' dtype")
    if group_offsets.numel() != len(weights) + 1:
        raise ValueError("group_offsets must hold n_groups + 1 entries")
    if y_perm is None:
        y_perm = _empty((max(cap_rows, 1), d), x_perm.dtype, x_perm.device)
    if ws is None:
        ws = workspace(moe_grouped_ffn_ws_bytes(dtype, cap_rows, d, f, len(weights)), x_perm.device)
    args = [_dev(x_perm, "x_perm"), dtype, _dev(group_offsets, "group_offsets", torch.int32),
            len(weights), ctypes.cast(weights.p13, ctypes.c_void_p),
            ctypes.cast(weights.p2, ctypes.c_void_p), d, f, cap_rows,
            _dev(y_perm, "y_perm", x_perm.dtype), _dev(ws, "ws"), ws.numel()]
    if products == MOE_FFN_GATE_UP | MOE_FFN_DOWN:
        _check("moe_grouped_ffn", lib.moe_grouped_ffn(*args, _stream(stream)))
    else:
        _check("moe_grouped_ffn_products",
               lib.moe_grouped_ffn_products(*args, products, _stream(stream)))
    return y_perm


def moe_grouped_ffn_combine(x_perm: torch.Tensor, group_offsets: torch.Tensor,
                            weights: WeightTable, token_row: torch.Tensor, topk_gate: torch.Tensor,
                            y_shared: Optional[torch.Tensor], *, cap_rows: int, T: int,
                            y: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                            stream=None) -> torch.Tensor:
    """Grouped FFN and weighted combine in one call (every group at most 256 rows).
    Returns y [T, d]."""
    lib = load_library()
    d, f = weights.d, weights.f
    dtype = _dtype_code(x_perm)
    if x_perm.dtype != weights.dtype or x_perm.shape[1] != d:
        raise ValueError("x_perm must be [rows, d] of the weights' dtype")
    k = token_row.shape[1]
    if y is None:
        y = _empty((max(T, 1), d), x_perm.dtype, x_perm.device)
    if ws is None:
        ws = workspace(moe_grouped_ffn_ws_bytes(dtype, cap_rows, d, f, len(weights)), x_perm.device)
    st = lib.moe_grouped_ffn_combine(
        _dev(x_perm, "x_perm"), dtype, _dev(group_offsets, "group_offsets", torch.int32),
        len(weights), ctypes.cast(weights.p13, ctypes.c_void_p),
        ctypes.cast(weights.p2, ctypes.c_void_p), d, f, cap_rows,
        _dev(token_row, "token_row", torch.int32), _dev(topk_gate, "topk_gate", torch.float32),
        _dev(y_shared, "y_shared", x_perm.dtype), T, k, _dev(y, "y", x_perm.dtype),
        _dev(ws, "ws"), ws.numel(), _stream(stream))
    _check("moe_grouped_ffn_combine", st)
    return y


def moe_grouped_ffn_rows(x: torch.Tensor, row_token: torch.Tensor, group_offsets: torch.Tensor,
                         weights: WeightTable, *, cap_rows: int,
                         y_perm: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                         stream=None, products: int = 3) -> torch.Tensor:
    """moe_grouped_ffn reading row p from x[row_token[p]] (no x_perm).  Returns y_perm.
    products other than 3 (single products, hints) call moe_grouped_ffn_rows_products."""
    lib = load_library()
    T = x.shape[0]
    d, f = weights.d, weights.f
    dtype = _dtype_code(x)
    if x.dtype != weights.dtype or x.shape[1] != d:
        raise ValueError("x must be [T, d] of the weights' dtype")
    if group_offsets.numel() != len(weights) + 1:
        raise ValueError("group_offsets must hold n_groups + 1 entries")
    if y_perm is None:
        y_perm = _empty((max(cap_rows, 1), d), x.dtype, x.device)
    if ws is None:
        ws = workspace(moe_grouped_ffn_ws_bytes(dtype, cap_rows, d, f, len(weights)), x.device)
    args = [_dev(x, "x"), T, _dev(row_token, "row_token", torch.int32), dtype,
            _dev(group_offsets, "group_offsets", torch.int32), len(weights),
            ctypes.cast(weights.p13, ctypes.c_void_p), ctypes.cast(weights.p2, ctypes.c_void_p), d, f,
            cap_rows, _dev(y_perm, "y_perm", x.dtype), _dev(ws, "ws"), ws.numel()]
    if products == MOE_FFN_GATE_UP | MOE_FFN_DOWN:
        _check("moe_grouped_ffn_rows", lib.moe_grouped_ffn_rows(*args, _stream(stream)))
    else:
        _check("moe_grouped_ffn_rows_products",
               lib.moe_grouped_ffn_rows_products(*args, products, _stream(stream)))
    return y_perm


def moe_grouped_ffn_rows_shared(x: torch.Tensor, row_token: torch.Tensor,
                                group_offsets: torch.Tensor, weights: WeightTable, n_shared: int, *,
                                cap_rows: int, y_perm: Optional[torch.Tensor] = None,
                                ws: Optional[torch.Tensor] = None, stream=None,
                                products: int = 3) -> torch.Tensor:
    """moe_grouped_ffn_rows_products with n_shared leading groups of T rows each
    (the shared experts, weights[0 .. n_shared-1]); the routed groups follow, their
    rows counted from n_shared * T.  Returns y_perm [n_shared * T + cap_rows, d]."""
    lib = load_library()
    T = x.shape[0]
    d, f = weights.d, weights.f
    dtype = _dtype_code(x)
    if x.dtype != weights.dtype or x.shape[1] != d:
        raise ValueError("x must be [T, d] of the weights' dtype")
    n_groups = len(weights) - n_shared
    if n_shared < 0 or n_groups < 0 or group_offsets.numel() != n_groups + 1:
        raise ValueError("group_offsets must hold n_groups + 1 entries for the routed groups")
    rows = n_shared * T + cap_rows
    if row_token.numel() < rows:
        raise ValueError("row_token must hold n_shared * T + cap_rows entries")
    if y_perm is None:
        y_perm = _empty((max(rows, 1), d), x.dtype, x.device)
    if ws is None:
        ws = workspace(moe_grouped_ffn_ws_bytes(dtype, rows, d, f, len(weights)), x.device)
    st = lib.moe_grouped_ffn_rows_shared(
        _dev(x, "x"), T, _dev(row_token, "row_token", torch.int32), dtype,
        _dev(group_offsets, "group_offsets", torch.int32), n_groups, n_shared,
        ctypes.cast(weights.p13, ctypes.c_void_p), ctypes.cast(weights.p2, ctypes.c_void_p), d, f,
        cap_rows, _dev(y_perm, "y_perm", x.dtype), _dev(ws, "ws"), ws.numel(), products,
        _stream(stream))
    _check("moe_grouped_ffn_rows_shared", st)
    return y_perm


def moe_combine(y_perm: torch.Tensor, token_row: torch.Tensor, topk_gate: torch.Tensor,
                y_shared: Optional[torch.Tensor], *, T: int, d: int,
                y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Gate-weighted sum back in token order (+ shared experts).  Returns y [T, d]."""
    lib = load_library()
    k = token_row.shape[1] if token_row.dim() == 2 else 1
    dtype = _dtype_code(y_perm)
    if y is None:
        y = _empty((T, d), y_perm.dtype, y_perm.device)
    st = lib.moe_combine(_dev(y_perm, "y_perm", y.dtype), dtype,
                         _dev(token_row, "token_row", torch.int32),
                         _dev(topk_gate, "topk_gate", torch.float32),
                         _dev(y_shared, "y_shared", y.dtype), T, d, k,
                         _dev(y, "y", y.dtype), _stream(stream))
    _check("moe_combine", st)
    return y


def moe_combine_shared(y_perm: torch.Tensor, token_row: torch.Tensor, topk_gate: torch.Tensor,
                       y_shared: Optional[torch.Tensor], n_shared: int, *, T: int, d: int,
                       y: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """moe_combine with the shared experts' output in n_shared [T, d] slices
    (y_shared [n_shared, T, d], added in slice order).  Returns y [T, d]."""
    lib = load_library()
    k = token_row.shape[1] if token_row.dim() == 2 else 1
    dtype = _dtype_code(y_perm)
    if y is None:
        y = _empty((T, d), y_perm.dtype, y_perm.device)
    if y_shared is not None and n_shared > 0 and y_shared.numel() < n_shared * T * d:
        raise ValueError("y_shared must hold n_shared slices of [T, d]")
    st = lib.moe_combine_shared(_dev(y_perm, "y_perm", y.dtype), dtype,
                                _dev(token_row, "token_row", torch.int32),
                                _dev(topk_gate, "topk_gate", torch.float32),
                                _dev(y_shared, "y_shared", y.dtype), n_shared, T, d, k,
                                _dev(y, "y", y.dtype), _stream(stream))
    _check("moe_combine_shared", st)
    return y
