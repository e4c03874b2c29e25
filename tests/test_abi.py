"""C-ABI surface checks that need no GPU: every symbol declared in
include/sscater.h is exported by the built library, and host-side argument
validation rejects bad calls before any HIP work."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2512_08557_amd as ssc
from paper_2512_08557_amd import engine as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "sscater.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(sscater_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_binding_surface():
    assert _declared() == sorted(E.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ssc.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name


def test_strerror_texts():
    lib = ssc.lib()
    for code in (0, -1, -2, -3, -4, -5, -99):
        assert isinstance(lib.sscater_strerror(code), bytes)
    assert b"max_pillars" in lib.sscater_strerror(ssc.E_OVERFLOW)


def _create(grid, layers, weights=True):
    lib = ssc.lib()
    n = len(layers)
    larr = (E.Layer * max(n, 1))(*layers) if n else None
    bufs = [np.zeros((l.cout, l.cin, 3, 3), np.float32) for l in layers]
    wp = (ctypes.c_void_p * max(n, 1))(*[b.ctypes.data for b in bufs]) if weights else None
    h = ctypes.c_void_p()
    return lib.sscater_create(ctypes.byref(grid) if grid is not None else None, larr, n, wp, ctypes.byref(h))


@pytest.mark.parametrize("case", [
    "null_grid", "no_layers", "k5", "pad0", "stride3", "chain", "unsupported_cout", "bad_c0", "bad_dtype",
    "relu2", "too_many_layers", "huge_grid", "tall_grid", "null_weights"])
def test_create_rejects_invalid_arguments(case):
    g = E.Grid(32, 32, 64, 100, E.F32)
    L = [E.Layer(64, 64, 3, 2, 1, 1), E.Layer(64, 64, 3, 1, 1, 1)]
    weights = True
    if case == "null_grid":
        g = None
    elif case == "no_layers":
        L = []
    elif case == "k5":
        L[0].k = 5
    elif case == "pad0":
        L[1].pad = 0
    elif case == "stride3":
        L[0].stride = 3
    elif case == "chain":
        L[1].cin = 32
    elif case == "unsupported_cout":
        L[1].cout = 24
    elif case == "bad_c0":
        g.C0 = 48
    elif case == "bad_dtype":
        g.dtype = 7
    elif case == "relu2":
        L[0].relu = 2
    elif case == "too_many_layers":
        L = [E.Layer(64, 64, 3, 1, 1, 1)] * 33
    elif case == "huge_grid":
        g.H, g.W = 1 << 16, 1 << 16
    elif case == "tall_grid":               # 32768 x 1 cells is small, but a coordinate needs 16 bits
        g.H, g.W = 1 << 15, 1
    elif case == "null_weights":
        weights = False
    assert _create(g, L, weights) == ssc.E_INVALID_ARG


def test_calls_reject_null_handle():
    lib = ssc.lib()
    p = E.Pillars(None, None, 0)
    assert lib.sscater_step(None, ctypes.byref(p), None) == ssc.E_INVALID_ARG
    assert lib.sscater_step_sorted(None, ctypes.byref(p), None) == ssc.E_INVALID_ARG
    assert lib.sscater_step_sorted(None, None, None) == ssc.E_INVALID_ARG
    assert lib.sscater_read(None, 0, None, 0, None) == ssc.E_INVALID_ARG
    assert lib.sscater_reset(None, None) == ssc.E_INVALID_ARG
    assert lib.sscater_destroy(None) == ssc.E_INVALID_ARG
    n = ctypes.c_int32()
    assert lib.sscater_changed(None, 0, None, 0, ctypes.byref(n), None) == ssc.E_INVALID_ARG
    st = E.Stats()
    assert lib.sscater_stats(None, ctypes.byref(st), None) == ssc.E_INVALID_ARG


def test_weight_marshalling_for_bf16():
    w = np.array([1.0, -2.5, 0.15625], np.float32)
    b = E.weights_to_dtype_bytes(w, "bf16")
    assert b.dtype == np.uint16 and b.tolist() == [0x3F80, 0xC020, 0x3E20]
    with pytest.raises(ValueError):
        E.weights_to_dtype_bytes(np.array([0.1], np.float32), "bf16")


def _create_neck(grid, layers, ups, up_w=True):
    lib = ssc.lib()
    n = len(layers)
    larr = (E.Layer * n)(*layers)
    bufs = [np.zeros((l.cout, l.cin, 3, 3), np.float32) for l in layers]
    wp = (ctypes.c_void_p * n)(*[b.ctypes.data for b in bufs])
    nu = len(ups)
    uarr = (E.Upsampler * max(nu, 1))(*ups)
    cins = [layers[u.src_layer - 1].cout if 1 <= u.src_layer <= n else 16 for u in ups]
    ubufs = [np.zeros((ci, u.cout, max(u.stride, 1), max(u.stride, 1)), np.float32) for ci, u in zip(cins, ups)]
    up = (ctypes.c_void_p * max(nu, 1))(*[b.ctypes.data for b in ubufs]) if up_w else None
    h = ctypes.c_void_p()
    rc = lib.sscater_create_neck(ctypes.byref(grid), larr, n, wp, uarr, nu, up, ctypes.byref(h))
    if rc == ssc.OK:
        lib.sscater_destroy(h)
    return rc


@pytest.mark.parametrize("case", ["src0", "src_beyond", "stride3", "unsupported", "grid_mismatch", "null_weights",
                                  "too_many"])
def test_create_neck_rejects_invalid_arguments(case):
    g = E.Grid(32, 32, 64, 100, E.F32)
    L = [E.Layer(64, 64, 3, 2, 1, 1), E.Layer(64, 128, 3, 2, 1, 1)]     # 16x16x64, then 8x8x128
    ups = [E.Upsampler(1, 128, 1, 1), E.Upsampler(2, 128, 2, 1)]        # both onto 16x16
    up_w = True
    if case == "src0":
        ups[0].src_layer = 0
    elif case == "src_beyond":
        ups[1].src_layer = 3
    elif case == "stride3":
        ups[1].stride = 3
    elif case == "unsupported":
        ups[0].cout = 48
    elif case == "grid_mismatch":
        ups[1].stride = 4                                                 # 8x8 -> 32x32, not 16x16
    elif case == "null_weights":
        up_w = False
    elif case == "too_many":
        ups = ups * 3
    assert _create_neck(g, L, ups, up_w) == ssc.E_INVALID_ARG


def _create_pfn(grid, layers, pfn, pfn_w=True):
    lib = ssc.lib()
    n = len(layers)
    larr = (E.Layer * n)(*layers)
    bufs = [np.zeros((l.cout, l.cin, 3, 3), np.float32) for l in layers]
    wp = (ctypes.c_void_p * n)(*[b.ctypes.data for b in bufs])
    pw = np.zeros((max(grid.C0, 1), 9), np.float32)
    ptr = pw.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if pfn_w else None
    h = ctypes.c_void_p()
    rc = lib.sscater_create_pfn(ctypes.byref(grid), larr, n, wp, ctypes.byref(pfn) if pfn is not None else None,
                                ptr, ctypes.byref(h))
    if rc == ssc.OK:
        lib.sscater_destroy(h)
    return rc


@pytest.mark.parametrize("case", ["no_spec", "no_weights", "res0", "res_nan", "corner_inf", "points0",
                                  "points129", "window0", "window65", "new_neg", "c0_wide", "bad_layers"])
def test_create_pfn_rejects_invalid_arguments(case):
    """Every check runs on the host before any HIP call."""
    g = E.Grid(16, 16, 64, 0, E.F32)
    L = [E.Layer(64, 64, 3, 1, 1, 1)]
    p = E.Pfn(-1.28, -1.28, 0.16, 100, 10, 2400)
    w = True
    if case == "no_spec":
        p = None
    elif case == "no_weights":
        w = False
    elif case == "res0":
        p.res = 0.0
    elif case == "res_nan":
        p.res = float("nan")
    elif case == "corner_inf":
        p.x_min = float("inf")
    elif case == "points0":
        p.max_points = 0
    elif case == "points129":
        p.max_points = 129
    elif case == "window0":
        p.window = 0
    elif case == "window65":
        p.window = 65
    elif case == "new_neg":
        p.max_new_points = -1
    elif case == "c0_wide":
        g = E.Grid(16, 16, 128, 0, E.F32)
        L = [E.Layer(128, 64, 3, 1, 1, 1)]
    elif case == "bad_layers":
        L = [E.Layer(32, 64, 3, 1, 1, 1)]
    assert _create_pfn(g, L, p, w) == ssc.E_INVALID_ARG


def test_points_calls_reject_null_handle():
    assert ssc.lib().sscater_step_points(None, None, 0, None) == ssc.E_INVALID_ARG


@pytest.mark.parametrize("case", ["null_flags", "first_sub", "sub_stride2", "flag2", "bad_layers"])
def test_create_sparse_rejects_invalid_arguments(case):
    """Every check runs on the host before any HIP call."""
    lib = ssc.lib()
    g = E.Grid(16, 16, 64, 100, E.F32)
    L = [E.Layer(64, 64, 3, 2, 1, 1), E.Layer(64, 64, 3, 1, 1, 1), E.Layer(64, 64, 3, 1, 1, 1)]
    flags = [0, 1, 1]
    if case == "first_sub":
        flags = [1, 1, 1]
    elif case == "sub_stride2":
        L[2].stride = 2
    elif case == "flag2":
        flags = [0, 2, 1]
    elif case == "bad_layers":
        L[1].cin = 32
    n = len(L)
    larr = (E.Layer * n)(*L)
    bufs = [np.zeros((l.cout, l.cin, 3, 3), np.float32) for l in L]
    wp = (ctypes.c_void_p * n)(*[b.ctypes.data for b in bufs])
    fl = None if case == "null_flags" else (ctypes.c_int32 * n)(*flags)
    h = ctypes.c_void_p()
    rc = lib.sscater_create_sparse(ctypes.byref(g), larr, n, wp, fl, ctypes.byref(h))
    if rc == ssc.OK:
        lib.sscater_destroy(h)
    assert rc == ssc.E_INVALID_ARG


@pytest.mark.parametrize("batch,hw", [(0, 16), (-1, 16), (1 << 11, 1 << 10)])
def test_create_batched_rejects_invalid_batch(batch, hw):
    """batch < 1, and a batch whose cells exceed 2^30 (host-side checks made
    before any HIP call)."""
    lib = ssc.lib()
    g = E.Grid(hw, hw, 64, 100, E.F32)
    L = [E.Layer(64, 64, 3, 1, 1, 1)]
    larr = (E.Layer * 1)(*L)
    buf = np.zeros((64, 64, 3, 3), np.float32)
    wp = (ctypes.c_void_p * 1)(buf.ctypes.data)
    h = ctypes.c_void_p()
    assert lib.sscater_create_batched(ctypes.byref(g), batch, larr, 1, wp, ctypes.byref(h)) == ssc.E_INVALID_ARG


def test_noalloc_change_list_rejects_bad_arguments_on_the_host():
    lib = ssc.lib()
    cnt = ctypes.c_void_p(8)   # never dereferenced: every case fails validation first
    assert lib.sscater_changed_noalloc(None, 0, None, 0, cnt, None) == ssc.E_INVALID_ARG
    assert b"scratch" in lib.sscater_strerror(E.E_SCRATCH)
