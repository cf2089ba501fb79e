"""Host-side checks of the C ABI that need no GPU.

The library must load and export every entry point include/moe.h declares,
and every validation error must be returned before anything touches HIP
(these calls use argument combinations that fail validation, so no kernel is
ever launched and no device pointer is ever dereferenced).
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_08782_amd import moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(moe.LIB_PATH):
        from paper_2607_08782_amd import build
        build.build()
    return moe.load_library()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\*|int|size_t)\s+(moe_\w+)\s*\(", text, re.M)))


def test_header_declares_the_five_steps():
    names = _declared()
    for n in ("moe_route_topk", "moe_expert_histogram", "moe_permute", "moe_grouped_ffn",
              "moe_combine"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(moe.EXPORTS)


def test_status_strings(lib):
    for code in range(5):
        assert moe.status_string(code) != "unknown status"
    assert moe.status_string(99) == "unknown status"


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation


def test_route_topk_validation(lib):
    f = lib.moe_route_topk
    ok = dict(x=FAKE, dtype=1, w=FAKE, b=None, T=4, d=64, E=8, k=2, flags=1, lg=FAKE, idx=FAKE,
              gate=FAKE)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["x"], a["dtype"], a["w"], a["b"], a["T"], a["d"], a["E"], a["k"], a["flags"],
                 a["lg"], a["idx"], a["gate"], a.get("ws"), a.get("ws_bytes", 0), None)
    assert call(k=0) == moe.MOE_ERR_ARG
    assert call(k=9) == moe.MOE_ERR_ARG            # k > E
    assert call(E=300, k=2) == moe.MOE_ERR_ARG      # E > MOE_MAX_E
    assert call(E=64, k=17) == moe.MOE_ERR_ARG      # k > MOE_MAX_K
    assert call(T=-1) == moe.MOE_ERR_ARG
    assert call(dtype=7) == moe.MOE_ERR_ARG
    assert call(flags=8) == moe.MOE_ERR_ARG
    assert call(idx=None) == moe.MOE_ERR_ARG
    assert call(x=None) == moe.MOE_ERR_ARG
    assert call(d=12) == moe.MOE_ERR_SHAPE          # bf16 rows must be 16-byte multiples
    assert call(x=ctypes.c_void_p(0x1002)) == moe.MOE_ERR_ARG   # misaligned bf16 rows
    assert call(flags=3, lg=None) == moe.MOE_ERR_ARG             # logits-in without logits
    assert call(E=256, k=2, d=4194304) == moe.MOE_ERR_SHAPE      # router past 32-bit offsets
    need = lib.moe_route_topk_ws_bytes(1, 4, 4096, 8, 1)
    assert need > 0                                              # a 4-token batch splits K
    assert call(d=4096) == moe.MOE_ERR_SHAPE                     # ... and needs its workspace
    assert call(d=4096, ws=ctypes.c_void_p(0x100000), ws_bytes=need - 1) == moe.MOE_ERR_SHAPE
    assert call(d=4096, ws=ctypes.c_void_p(0x100010), ws_bytes=need) == moe.MOE_ERR_SHAPE
    assert lib.moe_route_topk_ws_bytes(1, 4, 64, 8, 1) == 0      # too short a K to split
    assert lib.moe_route_topk_ws_bytes(1, 4, 64, 8, 3) == 0      # logits-in: none
    assert lib.moe_route_topk_ws_bytes(0, 4, 64, 8, 1) == 0      # fp32 path: none


def test_histogram_validation(lib):
    f = lib.moe_expert_histogram
    assert f(FAKE, 4, 0, 8, FAKE, None, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 4, 2, 0, FAKE, None, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 4, 2, 8, None, None, None) == moe.MOE_ERR_ARG
    assert f(None, 4, 2, 8, FAKE, None, None) == moe.MOE_ERR_ARG


def _permute(lib, placement, T=10, k=2, E=4, cap=None, ws_bytes=None, dev=0, c_max=0, d=64,
             dtype=1):
    pl = np.ascontiguousarray(placement, np.uint8)
    G = pl.shape[1]
    if cap is None:
        cap = T * k
    if ws_bytes is None:
        ws_bytes = lib.moe_permute_ws_bytes(T, k, E)
    return lib.moe_permute(FAKE, dtype, FAKE, FAKE, FAKE, T, d, k, E,
                           pl.ctypes.data_as(ctypes.c_void_p), G, dev, c_max, FAKE, cap, FAKE,
                           FAKE, FAKE, FAKE, FAKE, ctypes.c_void_p(0x100000), ws_bytes, None)


def test_permute_placement_and_capacity_validation(lib):
    pl = np.array([[1, 0], [0, 1], [1, 1], [0, 0]])     # expert 3 has no host
    assert _permute(lib, pl) == moe.MOE_ERR_PLACEMENT
    pl[3, 1] = 1
    assert _permute(lib, pl, dev=2) == moe.MOE_ERR_PLACEMENT          # dev >= G
    assert _permute(lib, pl, c_max=1) == moe.MOE_ERR_PLACEMENT        # 2 local experts > c_max
    assert _permute(lib, pl, cap=10 * 2 - 1) == moe.MOE_ERR_SHAPE     # cap < T*min(k, n_local)
    assert _permute(lib, pl, ws_bytes=16) == moe.MOE_ERR_SHAPE
    assert _permute(lib, pl, d=12) == moe.MOE_ERR_SHAPE
    assert _permute(lib, pl, k=0) == moe.MOE_ERR_ARG
    assert _permute(lib, pl, dtype=5) == moe.MOE_ERR_ARG
    big = np.ones((4, 65), np.uint8)
    assert _permute(lib, big) == moe.MOE_ERR_PLACEMENT                # G > MOE_MAX_G


def test_permute_noalloc_validation(lib):
    """The same checks as moe_permute (nothing touches HIP before they pass), and
    batches whose block counts exceed the library's scratch are refused."""
    f = lib.moe_permute_noalloc

    def call(pl, T=10, d=64, k=2, E=4, dev=0, cap=None, c_max=0):
        pl = np.ascontiguousarray(pl, np.uint8)
        G = pl.shape[1]
        if cap is None:
            cap = T * k
        return f(FAKE, 1, FAKE, FAKE, FAKE, T, d, k, E, pl.ctypes.data_as(ctypes.c_void_p), G,
                 dev, c_max, FAKE, cap, FAKE, FAKE, FAKE, FAKE, None, None)
    pl = np.array([[1, 0], [0, 1], [1, 1], [0, 0]])
    assert call(pl) == moe.MOE_ERR_PLACEMENT                       # expert 3 has no host
    pl[3, 1] = 1
    assert call(pl, dev=2) == moe.MOE_ERR_PLACEMENT
    assert call(pl, c_max=1) == moe.MOE_ERR_PLACEMENT
    assert call(pl, cap=19) == moe.MOE_ERR_SHAPE
    assert call(pl, d=12) == moe.MOE_ERR_SHAPE
    assert call(pl, k=0) == moe.MOE_ERR_ARG
    E = 128
    pl = np.ones((E, 1), np.uint8)
    T = 600000                                                      # 9375 blocks x 128 slots
    assert lib.moe_permute_ws_bytes(T, 8, E) > moe.MOE_PERMUTE_NOALLOC_MAX_WS
    assert call(pl, T=T, k=8, E=E) == moe.MOE_ERR_SHAPE
    T = 500000
    assert lib.moe_permute_ws_bytes(T, 8, E) <= moe.MOE_PERMUTE_NOALLOC_MAX_WS


def test_grouped_ffn_products_validation(lib):
    f = lib.moe_grouped_ffn_products
    arr = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(products=1, x=FAKE, y=FAKE, w13=P, w2=P, d=128, f_=64, ws_bytes=1 << 30):
        return f(x, 1, FAKE, 2, w13, w2, d, f_, 16, y, ctypes.c_void_p(0x100000), ws_bytes,
                 products, None)
    assert call(products=0) == moe.MOE_ERR_ARG
    assert call(products=4) == moe.MOE_ERR_ARG                    # a hint alone runs nothing
    assert call(products=8) == moe.MOE_ERR_ARG
    assert call(products=3 | 4 | 8) == moe.MOE_ERR_ARG            # the two hints contradict
    assert call(products=1 | 16) == moe.MOE_ERR_ARG               # no such flag
    assert call(products=1, x=None) == moe.MOE_ERR_ARG           # gate/up reads x_perm
    assert call(products=1, w13=None) == moe.MOE_ERR_ARG
    assert call(products=2, y=None) == moe.MOE_ERR_ARG           # down writes y_perm
    assert call(products=2, w2=None) == moe.MOE_ERR_ARG
    assert call(products=3, d=100) == moe.MOE_ERR_SHAPE
    assert call(products=3, d=1 << 22) == moe.MOE_ERR_SHAPE          # tile offsets past 32 bits
    assert call(products=3, f_=1 << 22) == moe.MOE_ERR_SHAPE
    assert call(products=2, ws_bytes=10) == moe.MOE_ERR_SHAPE


def test_grouped_ffn_combine_validation(lib):
    f = lib.moe_grouped_ffn_combine
    arr = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(dtype=1, T=8, k=2, y=FAKE, tr=FAKE, d=128, f_=64):
        return f(FAKE, dtype, FAKE, 2, P, P, d, f_, 16, tr, FAKE, None, T, k, y,
                 ctypes.c_void_p(0x100000), 1 << 30, None)
    assert call(dtype=0) == moe.MOE_ERR_ARG                  # bf16 only
    assert call(k=0) == moe.MOE_ERR_ARG
    assert call(k=17) == moe.MOE_ERR_ARG
    assert call(T=-1) == moe.MOE_ERR_ARG
    assert call(y=None) == moe.MOE_ERR_ARG
    assert call(tr=None) == moe.MOE_ERR_ARG
    assert call(y=ctypes.c_void_p(0x1008)) == moe.MOE_ERR_ARG
    assert call(d=100) == moe.MOE_ERR_SHAPE


def test_grouped_ffn_validation(lib):
    f = lib.moe_grouped_ffn
    arr = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    null_arr = (ctypes.c_void_p * 2)(0x1000, None)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(dtype=1, n=2, d=128, f_=64, cap=16, w13=P, ws=0x100000, ws_bytes=1 << 30):
        return f(FAKE, dtype, FAKE, n, w13, P, d, f_, cap, FAKE, ctypes.c_void_p(ws), ws_bytes, None)
    assert call(n=0) == moe.MOE_ERR_ARG
    assert call(n=129) == moe.MOE_ERR_ARG
    assert call(d=100) == moe.MOE_ERR_SHAPE
    assert call(f_=96) == moe.MOE_ERR_SHAPE
    assert call(ws_bytes=10) == moe.MOE_ERR_SHAPE
    assert call(ws=0x100010) == moe.MOE_ERR_SHAPE        # workspace not 256-byte aligned
    assert call(w13=ctypes.cast(null_arr, ctypes.c_void_p)) == moe.MOE_ERR_ARG
    assert call(dtype=3) == moe.MOE_ERR_ARG


def test_grouped_ffn_rows_validation(lib):
    f = lib.moe_grouped_ffn_rows
    arr = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(T=64, rows=FAKE, dtype=1, d=128, f_=64, cap=16, x=FAKE, ws=0x100000, ws_bytes=1 << 30):
        return f(x, T, rows, dtype, FAKE, 2, P, P, d, f_, cap, FAKE, ctypes.c_void_p(ws), ws_bytes,
                 None)
    assert call(rows=None) == moe.MOE_ERR_ARG               # no row map
    assert call(x=None) == moe.MOE_ERR_ARG
    assert call(T=-1) == moe.MOE_ERR_ARG
    assert call(T=0) == moe.MOE_ERR_ARG                     # rows to compute but no token rows
    assert call(T=1 << 24, d=128) == moe.MOE_ERR_SHAPE      # T*d*2 past 32-bit row offsets
    assert call(d=100) == moe.MOE_ERR_SHAPE
    assert call(T=1, f_=1 << 22) == moe.MOE_ERR_SHAPE        # a tile's offsets past 32 bits
    assert call(x=FAKE.value + 8) == moe.MOE_ERR_ARG        # bf16 rows not 16-byte aligned
    assert call(ws_bytes=10) == moe.MOE_ERR_SHAPE
    assert call(dtype=3) == moe.MOE_ERR_ARG


def test_grouped_ffn_rows_products_validation(lib):
    f = lib.moe_grouped_ffn_rows_products
    arr = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(products=3, rows=FAKE, x=FAKE, y=FAKE, d=128, ws_bytes=1 << 30):
        return f(x, 64, rows, 1, FAKE, 2, P, P, d, 64, 16, y, ctypes.c_void_p(0x100000), ws_bytes,
                 products, None)
    assert call(products=0) == moe.MOE_ERR_ARG
    assert call(products=8) == moe.MOE_ERR_ARG                     # a hint alone runs nothing
    assert call(products=3 | 4 | 8) == moe.MOE_ERR_ARG             # the two hints contradict
    assert call(products=1 | 16) == moe.MOE_ERR_ARG
    assert call(products=1, rows=None) == moe.MOE_ERR_ARG          # gate/up reads the row map
    assert call(products=1, x=None) == moe.MOE_ERR_ARG
    assert call(products=2, y=None) == moe.MOE_ERR_ARG             # down writes y_perm
    assert call(products=3 | 8, d=100) == moe.MOE_ERR_SHAPE
    assert call(products=3 | 8, ws_bytes=10) == moe.MOE_ERR_SHAPE


def test_grouped_ffn_rows_shared_validation(lib):
    f = lib.moe_grouped_ffn_rows_shared
    arr = (ctypes.c_void_p * 4)(0x1000, 0x2000, 0x3000, 0x4000)
    P = ctypes.cast(arr, ctypes.c_void_p)

    def call(T=64, n_groups=2, n_shared=2, products=3, rows=FAKE, x=FAKE, y=FAKE, d=128, cap=16,
             offsets=FAKE, ws_bytes=1 << 30):
        return f(x, T, rows, 1, offsets, n_groups, n_shared, P, P, d, 64, cap, y,
                 ctypes.c_void_p(0x100000), ws_bytes, products, None)
    assert call(n_shared=-1) == moe.MOE_ERR_ARG
    assert call(n_groups=-1) == moe.MOE_ERR_ARG
    assert call(n_groups=0, n_shared=0) == moe.MOE_ERR_ARG          # no group at all
    assert call(n_groups=100, n_shared=29) == moe.MOE_ERR_ARG       # past MOE_MAX_GROUPS
    assert call(T=0) == moe.MOE_ERR_ARG                             # shared rows need tokens
    assert call(offsets=None) == moe.MOE_ERR_ARG
    assert call(rows=None) == moe.MOE_ERR_ARG                       # the shared rows' map too
    assert call(products=2, y=None) == moe.MOE_ERR_ARG
    assert call(products=3 | 4 | 8) == moe.MOE_ERR_ARG
    assert call(d=100) == moe.MOE_ERR_SHAPE
    assert call(T=1 << 20, n_shared=2, cap=(1 << 31) - (1 << 20)) == moe.MOE_ERR_ARG   # rows past 2^31
    # the workspace covers the shared rows as well: enough for the routed rows alone fails
    routed_only = lib.moe_grouped_ffn_ws_bytes(1, 16, 128, 64, 4)
    assert call(ws_bytes=routed_only) == moe.MOE_ERR_SHAPE
    assert call(n_shared=0, ws_bytes=routed_only - 1) == moe.MOE_ERR_SHAPE


def test_combine_shared_validation(lib):
    f = lib.moe_combine_shared
    assert f(FAKE, 1, FAKE, FAKE, FAKE, -1, 4, 64, 2, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, FAKE, FAKE, FAKE, 129, 4, 64, 2, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, FAKE, FAKE, ctypes.c_void_p(0x1008), 2, 4, 64, 2, FAKE, None) == \
        moe.MOE_ERR_ARG                                             # slices not 16-byte aligned
    assert f(None, 1, FAKE, FAKE, FAKE, 2, 4, 64, 2, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, FAKE, FAKE, FAKE, 2, 4, 64, 0, FAKE, None) == moe.MOE_ERR_ARG


def test_combine_validation(lib):
    f = lib.moe_combine
    assert f(FAKE, 1, FAKE, FAKE, None, 4, 64, 0, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, FAKE, FAKE, None, 4, 0, 2, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, None, FAKE, None, 4, 64, 2, FAKE, None) == moe.MOE_ERR_ARG
    assert f(FAKE, 1, FAKE, FAKE, None, 4, 64, 2, ctypes.c_void_p(0x1008), None) == moe.MOE_ERR_ARG
    assert f(None, 1, FAKE, FAKE, None, 4, 64, 2, FAKE, None) == moe.MOE_ERR_ARG   # y_perm


def test_workspace_sizes(lib):
    a = lib.moe_permute_ws_bytes(1000, 4, 60)
    b = lib.moe_permute_ws_bytes(2000, 4, 60)
    assert 0 < a < b
    assert lib.moe_grouped_ffn_ws_bytes(1, 100, 256, 128, 4) >= 100 * 128 * 2
    assert lib.moe_grouped_ffn_ws_bytes(0, 100, 256, 128, 4) >= 100 * 128 * 4


def test_quantize_e4m3_validation(lib):
    f = lib.moe_quantize_e4m3
    assert f(FAKE, 2, 4, 64, FAKE, FAKE, None) == moe.MOE_ERR_ARG      # dtype
    assert f(FAKE, 1, -1, 64, FAKE, FAKE, None) == moe.MOE_ERR_ARG     # rows < 0
    assert f(FAKE, 1, 4, 0, FAKE, FAKE, None) == moe.MOE_ERR_ARG       # cols < 1
    assert f(FAKE, 1, 4, 64, None, FAKE, None) == moe.MOE_ERR_ARG      # q
    assert f(FAKE, 1, 4, 64, FAKE, None, None) == moe.MOE_ERR_ARG      # scales


def test_route_topk_e4m3_validation(lib):
    f = lib.moe_route_topk_e4m3

    def call(xq=FAKE, wq=FAKE, T=4, d=128, E=8, k=2, flags=1, lg=FAKE):
        return f(xq, FAKE, wq, FAKE, None, T, d, E, k, flags, lg, FAKE, FAKE, None)
    assert call(d=96) == moe.MOE_ERR_SHAPE                  # d % 64
    assert call(d=0) == moe.MOE_ERR_SHAPE
    assert call(E=0) == moe.MOE_ERR_ARG
    assert call(E=257) == moe.MOE_ERR_ARG
    assert call(k=9) == moe.MOE_ERR_ARG                     # k > E
    assert call(k=17, E=64) == moe.MOE_ERR_ARG              # k > MOE_MAX_K
    assert call(flags=2) == moe.MOE_ERR_ARG                 # scores are computed here
    assert call(lg=None) == moe.MOE_ERR_ARG                 # logits are required
    assert call(wq=ctypes.c_void_p(0x1008)) == moe.MOE_ERR_ARG   # 16-byte alignment
    assert call(xq=None) == moe.MOE_ERR_ARG
