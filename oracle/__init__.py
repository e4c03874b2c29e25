"""CPU oracle for the delta-scatter backbone -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The GPU library never loads it and shares no code
with it.

What it computes (SSCATeR, arXiv 2512.08557):

* ``forward``: every backbone layer recomputed densely from the window's input
  canvas in float64 (``sscater_oracle.c``).  The paper states that the recycled
  maps are identical to recomputation (abstract; Sec. IV-G), so recomputation is
  the reference for the maps.
* ``changed_lists``: the per-layer changed-cell sets.  The input set A_0 is the
  set of cells whose input feature vector differs bit for bit from the previous
  window (a pillar whose points changed, Sec. III-B and Alg. 1, PFN part).  For
  each convolution layer the set is derived in the *gather* direction: an
  output cell is changed iff one of its 3x3 input taps lies in the grid and in
  the previous layer's set (Alg. 1, backbone part: an output site touched by
  the scatter of a changed site is marked, and for stride > 1 a downsampled
  site is marked when any site under its kernel is changed).  The GPU path
  builds the same sets in the scatter direction.
* ``conv_transpose`` / ``forward_neck`` / ``upsample_mask``: the neck that
  upsamples block outputs by a transposed convolution with kernel = stride and
  concatenates them (Sec. III-B, backbone paragraph).  Upsampled change sets
  follow Alg. 1's deconvolution rule: every upsampled site under a changed
  site is changed.
* ``value_changed``: the cells whose layer output value actually differs
  between two windows (used for the locality invariant: a value can only change
  where the structural set says so).

``method_model.DeltaScatterModel`` is a float64 CPU model of the method itself
(Eq. 2 plus the change-map rules), used only to pin that recycling equals
recomputation.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"oracle library not built: {LIB_PATH} (run __graft_entry__.build())")
        lib = ctypes.CDLL(LIB_PATH)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int)
        lib.oracle_conv3x3_f64.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, dp,
                                           ctypes.c_int, ctypes.c_int, dp]
        lib.oracle_conv3x3_f64.restype = ctypes.c_int
        lib.oracle_round_bf16.argtypes = [dp, ctypes.c_size_t]
        lib.oracle_round_bf16.restype = None
        lib.oracle_backbone_f64.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ip, ip, ip, ip, ctypes.POINTER(dp), ctypes.c_int,
                                            ctypes.POINTER(dp)]
        lib.oracle_backbone_f64.restype = ctypes.c_int
        lib.oracle_convT_f64.argtypes = [dp, ctypes.c_int, ctypes.c_int, ctypes.c_int, dp,
                                         ctypes.c_int, ctypes.c_int, dp]
        lib.oracle_convT_f64.restype = ctypes.c_int
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """Threads the oracle's OpenMP loops run on."""
    return int(_load().oracle_threads())


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def out_extent(n: int, stride: int) -> int:
    """3x3 conv, zero padding 1: floor((n + 2 - 3) / s) + 1."""
    return (n + 2 - 3) // stride + 1


def conv3x3(x: np.ndarray, w: np.ndarray, stride: int) -> np.ndarray:
    """Dense 3x3 conv, zero padding 1. x: [H, W, cin] float64; w: OIHW."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    H, W, cin = x.shape
    cout = w.shape[0]
    assert w.shape == (cout, cin, 3, 3)
    out = np.empty((out_extent(H, stride), out_extent(W, stride), cout), dtype=np.float64)
    rc = _load().oracle_conv3x3_f64(_dptr(x), H, W, cin, _dptr(w), cout, stride, _dptr(out))
    if rc != 0:
        raise ValueError("oracle_conv3x3_f64 rejected its arguments")
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float64 -> float32 (RNE) -> bfloat16 (RNE), returned as float64."""
    y = np.array(x, dtype=np.float64, copy=True, order="C")
    _load().oracle_round_bf16(_dptr(y), y.size)
    return y


def forward(x0: np.ndarray, weights: Sequence[np.ndarray], layers: Sequence[Tuple[int, int, int, bool]],
            bf16_storage: bool = False) -> List[np.ndarray]:
    """All layer outputs Y_1..Y_L recomputed from scratch (float64).

    x0: [H0, W0, C0] canvas holding the exact values of the stored dtype.
    layers: (cin, cout, stride, relu) per layer.
    """
    x0 = np.ascontiguousarray(x0, dtype=np.float64)
    H, W, C = x0.shape
    L = len(layers)
    ws = [np.ascontiguousarray(w, dtype=np.float64) for w in weights]
    ys = []
    h, wd = H, W
    for (cin, cout, s, _r) in layers:
        h, wd = out_extent(h, s), out_extent(wd, s)
        ys.append(np.empty((h, wd, cout), dtype=np.float64))
    arr = lambda vals, t: (t * L)(*vals)
    dp = ctypes.POINTER(ctypes.c_double)
    rc = _load().oracle_backbone_f64(
        _dptr(x0), H, W, C, L,
        arr([l[0] for l in layers], ctypes.c_int), arr([l[1] for l in layers], ctypes.c_int),
        arr([l[2] for l in layers], ctypes.c_int), arr([int(bool(l[3])) for l in layers], ctypes.c_int),
        (dp * L)(*[_dptr(w) for w in ws]), int(bool(bf16_storage)), (dp * L)(*[_dptr(y) for y in ys]))
    if rc != 0:
        raise ValueError("oracle_backbone_f64 rejected its arguments")
    return ys


def conv_transpose(x: np.ndarray, w: np.ndarray, stride: int) -> np.ndarray:
    """Transposed conv, kernel = stride, no padding. x: [H, W, cin] float64;
    w: [cin, cout, s, s] (ConvTranspose2d layout). Returns [H*s, W*s, cout]."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    H, W, cin = x.shape
    cout = w.shape[1]
    assert w.shape == (cin, cout, stride, stride)
    out = np.empty((H * stride, W * stride, cout), dtype=np.float64)
    rc = _load().oracle_convT_f64(_dptr(x), H, W, cin, _dptr(w), cout, stride, _dptr(out))
    if rc != 0:
        raise ValueError("oracle_convT_f64 rejected its arguments")
    return out


def forward_neck(ys: Sequence[np.ndarray], up_weights: Sequence[np.ndarray],
                 ups: Sequence[Tuple[int, int, int, bool]], bf16_storage: bool = False) -> np.ndarray:
    """The neck output: for each upsampler (src_layer 1..L, cout, stride,
    relu), phi(conv_transpose(Y_src)), bf16-rounded for bf16 storage, all
    concatenated along the channels in order.  ys: Y_1..Y_L from forward()."""
    outs = []
    for (src, _cout, s, relu), w in zip(ups, up_weights):
        z = conv_transpose(ys[src - 1], w, s)
        if relu:
            z = np.maximum(z, 0.0)
        if bf16_storage:
            z = round_bf16(z)
        outs.append(z)
    shapes = {o.shape[:2] for o in outs}
    assert len(shapes) == 1, "upsampled maps must share one grid"
    return np.concatenate(outs, axis=-1)


def upsample_mask(mask: np.ndarray, stride: int) -> np.ndarray:
    """Alg. 1, deconvolution rule: output (y, x) is changed iff its one input
    cell (y // s, x // s) is changed."""
    H, W = mask.shape
    ys = np.arange(H * stride) // stride
    xs = np.arange(W * stride) // stride
    return mask[np.ix_(ys, xs)]


def neck_changed(lists: Sequence[np.ndarray], layer_shapes: Sequence[Tuple[int, int]],
                 ups: Sequence[Tuple[int, int, int, bool]]) -> np.ndarray:
    """Sorted cell list of the neck's change set: the union of the upsampled
    sets of the source layers.  lists: A_0..A_L as from changed_lists();
    layer_shapes: (H_l, W_l) for l = 1..L."""
    out = None
    for (src, _cout, s, _relu) in ups:
        H, W = layer_shapes[src - 1]
        m = np.zeros(H * W, dtype=bool)
        m[lists[src]] = True
        up = upsample_mask(m.reshape(H, W), s)
        out = up if out is None else (out | up)
    return np.flatnonzero(out)


# ---------------------------------------------------------------------------
# changed-cell sets
# ---------------------------------------------------------------------------
def input_changed_mask(prev_bits: np.ndarray, new_bits: np.ndarray) -> np.ndarray:
    """A_0 as a [H, W] bool mask: any channel's bit pattern differs."""
    assert prev_bits.shape == new_bits.shape and prev_bits.dtype == new_bits.dtype
    return np.any(prev_bits != new_bits, axis=-1)


def propagate_gather(mask: np.ndarray, stride: int) -> np.ndarray:
    """Next layer's changed mask by the receptive-field rule: output (y, x) is
    changed iff some tap (s*y+m-1, s*x+n-1), m, n in 0..2, is in the grid and
    changed."""
    H, W = mask.shape
    Ho, Wo = out_extent(H, stride), out_extent(W, stride)
    out = np.zeros((Ho, Wo), dtype=bool)
    ys = np.arange(Ho)
    xs = np.arange(Wo)
    for m in range(3):
        iy = stride * ys + m - 1
        oky = (iy >= 0) & (iy < H)
        for n in range(3):
            ix = stride * xs + n - 1
            okx = (ix >= 0) & (ix < W)
            sub = np.zeros((Ho, Wo), dtype=bool)
            sub[np.ix_(oky, okx)] = mask[np.ix_(iy[oky], ix[okx])]
            out |= sub
    return out


def changed_lists(prev_bits: np.ndarray, new_bits: np.ndarray, strides: Sequence[int]) -> List[np.ndarray]:
    """Sorted row-major cell lists A_0..A_L (int64)."""
    m = input_changed_mask(prev_bits, new_bits)
    out = [np.flatnonzero(m)]
    for s in strides:
        m = propagate_gather(m, s)
        out.append(np.flatnonzero(m))
    return out


def value_changed(y_prev: np.ndarray, y_new: np.ndarray) -> np.ndarray:
    """Cells whose output vector differs in value between two windows."""
    return np.flatnonzero(np.any(y_prev != y_new, axis=-1))


def exact_canvas(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Stored canvas (float32 values, or uint16 bf16 bit patterns) -> exact float64."""
    if dtype == "bf16":
        f = (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
        return f.astype(np.float64)
    return np.asarray(bits, dtype=np.float32).astype(np.float64)


def canvas_bits(bits_or_values: np.ndarray, dtype: str) -> np.ndarray:
    """Bit patterns of a stored canvas for the bitwise change test."""
    if dtype == "bf16":
        return np.ascontiguousarray(bits_or_values, dtype=np.uint16)
    return np.ascontiguousarray(bits_or_values, dtype=np.float32).view(np.uint32)


def pair_counts(mask: np.ndarray, stride: int) -> int:
    """Number of (changed input cell, output cell) pairs joined by one kernel
    tap, counted in the gather direction: for every output cell, its in-grid
    taps that fall on a changed input cell.  This is the number of per-tap
    contractions the scatter of Eq. 2 performs for the layer."""
    H, W = mask.shape
    Ho, Wo = out_extent(H, stride), out_extent(W, stride)
    total = 0
    ys, xs = np.arange(Ho), np.arange(Wo)
    for m in range(3):
        iy = stride * ys + m - 1
        oky = (iy >= 0) & (iy < H)
        for n in range(3):
            ix = stride * xs + n - 1
            okx = (ix >= 0) & (ix < W)
            total += int(mask[np.ix_(iy[oky], ix[okx])].sum())
    return total
