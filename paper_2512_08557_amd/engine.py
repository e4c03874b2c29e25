"""ctypes binding of libsscater.so (argument marshalling only).

Every step of the hot path runs in the library's HIP kernels; this module
only converts Python/torch arguments into the C ABI of include/sscater.h:
device pointers come from ``tensor.data_ptr()`` and the HIP stream from
``torch.cuda.current_stream().cuda_stream``.  There is no fallback: if the
library is missing, importing the binding raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsscater.so")

MAX_LAYERS = 32
MAX_UPSAMPLERS = 4
OK, E_INVALID_ARG, E_OUT_OF_MEMORY, E_HIP, E_OVERFLOW, E_DEVICE, E_SCRATCH = 0, -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1

# every function declared in include/sscater.h
EXPORTS = ("sscater_create", "sscater_create_neck", "sscater_create_pfn", "sscater_create_sparse",
           "sscater_create_batched", "sscater_step", "sscater_step_sorted",
           "sscater_step_points",
           "sscater_read", "sscater_reset", "sscater_destroy", "sscater_changed", "sscater_changed_noalloc",
           "sscater_stats", "sscater_profile", "sscater_profile_read", "sscater_strerror")


class Grid(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("W", ctypes.c_int32), ("C0", ctypes.c_int32),
                ("max_pillars", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Layer(ctypes.Structure):
    _fields_ = [("cin", ctypes.c_int32), ("cout", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("relu", ctypes.c_int32)]


class Upsampler(ctypes.Structure):
    _fields_ = [("src_layer", ctypes.c_int32), ("cout", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("relu", ctypes.c_int32)]


class Pfn(ctypes.Structure):
    _fields_ = [("x_min", ctypes.c_float), ("y_min", ctypes.c_float), ("res", ctypes.c_float),
                ("max_points", ctypes.c_int32), ("window", ctypes.c_int32), ("max_new_points", ctypes.c_int32)]


class Pillars(ctypes.Structure):
    _fields_ = [("idx", ctypes.c_void_p), ("feats", ctypes.c_void_p), ("count", ctypes.c_int32)]


class Stats(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("pillars", ctypes.c_int32), ("steps", ctypes.c_int64),
                ("active", ctypes.c_int64 * (MAX_LAYERS + 1)), ("pairs", ctypes.c_int64 * (MAX_LAYERS + 1)),
                ("active_total", ctypes.c_int64 * (MAX_LAYERS + 1)),
                ("pairs_total", ctypes.c_int64 * (MAX_LAYERS + 1)),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double), ("n_ups", ctypes.c_int32),
                ("up_pairs", ctypes.c_int64 * MAX_UPSAMPLERS)]


class SscaterError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {lib().sscater_strerror(code).decode()} ({code})")


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"HIP library not built: {LIB_PATH} (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.sscater_create.argtypes = [ctypes.POINTER(Grid), ctypes.POINTER(Layer), i32,
                                     ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(vp)]
        L.sscater_create_neck.argtypes = [ctypes.POINTER(Grid), ctypes.POINTER(Layer), i32,
                                          ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(Upsampler), i32,
                                          ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(vp)]
        L.sscater_create_pfn.argtypes = [ctypes.POINTER(Grid), ctypes.POINTER(Layer), i32,
                                         ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(Pfn),
                                         ctypes.POINTER(ctypes.c_float), ctypes.POINTER(vp)]
        L.sscater_create_sparse.argtypes = [ctypes.POINTER(Grid), ctypes.POINTER(Layer), i32,
                                            ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(i32), ctypes.POINTER(vp)]
        L.sscater_create_batched.argtypes = [ctypes.POINTER(Grid), i32, ctypes.POINTER(Layer), i32,
                                             ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(vp)]
        L.sscater_step.argtypes = [vp, ctypes.POINTER(Pillars), vp]
        L.sscater_step_sorted.argtypes = [vp, ctypes.POINTER(Pillars), vp]
        L.sscater_step_points.argtypes = [vp, vp, i32, vp]
        L.sscater_read.argtypes = [vp, i32, vp, ctypes.c_size_t, vp]
        L.sscater_reset.argtypes = [vp, vp]
        L.sscater_destroy.argtypes = [vp]
        L.sscater_changed.argtypes = [vp, i32, ctypes.POINTER(i32), i32, ctypes.POINTER(i32), vp]
        L.sscater_changed_noalloc.argtypes = [vp, i32, vp, i32, vp, vp]
        L.sscater_stats.argtypes = [vp, ctypes.POINTER(Stats), vp]
        L.sscater_profile.argtypes = [vp, i32]
        L.sscater_profile_read.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), i32,
                                           vp]
        L.sscater_strerror.argtypes = [ctypes.c_int]
        L.sscater_strerror.restype = ctypes.c_char_p
        for f in EXPORTS[:-1]:
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int, where: str) -> None:
    if rc != OK:
        raise SscaterError(rc, where)


def out_extent(n: int, stride: int) -> int:
    return (n - 1) // stride + 1


def weights_to_dtype_bytes(w: np.ndarray, dtype: str) -> np.ndarray:
    """OIHW weights as the grid dtype's bytes: float32, or the bf16 bit
    patterns of values that are exactly representable in bf16."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    if dtype == "f32":
        return w
    u = w.view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("bf16 weights must be exactly representable in bfloat16")
    return np.ascontiguousarray((u >> 16).astype(np.uint16))


class Engine:
    """One handle of the delta-scatter backbone state (one sensor stream)."""

    def __init__(self, H: int, W: int, C0: int, layers: Sequence[Tuple[int, int, int, bool]],
                 weights: Sequence[np.ndarray], dtype: str = "f32", max_pillars: int = 16000,
                 ups: Sequence[Tuple[int, int, int, bool]] = (), up_weights: Sequence[np.ndarray] = (),
                 pfn=None, pfn_weights: Optional[np.ndarray] = None, submanifold: Optional[Sequence[bool]] = None,
                 batch: int = 1):
        """layers: (cin, cout, stride, relu); weights: OIHW per layer.  ups:
        optional neck, (src_layer, cout, stride, relu) per upsampler with
        [cin, cout, s, s] weights; the neck map is layer len(layers) + 1.
        pfn: optional points mode, (x_min, y_min, res, max_points, window,
        max_new_points) with [C0, 9] float32 pfn_weights; strides are then
        given to step_points.  submanifold: optional per-layer flags of a
        sparse backbone (regular sparse layers where False).  batch: several
        independent images of H x W in one handle (cell b*H*W + r*W + c);
        read() then returns [batch, H, W, C]."""
        import torch  # device memory and streams only
        self._torch = torch
        self.H, self.W, self.C0 = H, W, C0
        self.dtype = dtype
        self.layers = [tuple(l) for l in layers]
        self.shapes = [(H, W, C0)]
        h, w = H, W
        for (cin, cout, s, _r) in self.layers:
            h, w = out_extent(h, s), out_extent(w, s)
            self.shapes.append((h, w, cout))
        grid = Grid(H, W, C0, max_pillars, BF16 if dtype == "bf16" else F32)
        n = len(self.layers)
        larr = (Layer * n)(*[Layer(ci, co, 3, s, 1, int(bool(r))) for (ci, co, s, r) in self.layers])
        self._wbufs = [weights_to_dtype_bytes(wt, dtype) for wt in weights]
        if len(self._wbufs) != n:
            raise ValueError("one weight tensor per layer")
        wptrs = (ctypes.c_void_p * n)(*[b.ctypes.data for b in self._wbufs])
        handle = ctypes.c_void_p()
        self.ups = [tuple(u) for u in ups]
        self.pfn = tuple(pfn) if pfn is not None else None
        self.submanifold = [bool(x) for x in submanifold] if submanifold is not None else None
        self.batch = int(batch)
        if self.batch != 1:
            if self.ups or self.pfn is not None or self.submanifold is not None:
                raise ValueError("a batched handle takes no neck, points mode or sparse layers")
            _check(lib().sscater_create_batched(ctypes.byref(grid), self.batch, larr, n, wptrs, ctypes.byref(handle)),
                   "sscater_create_batched")
        elif self.submanifold is not None:
            if self.ups or self.pfn is not None:
                raise ValueError("a sparse backbone takes no neck and no points mode")
            if len(self.submanifold) != n:
                raise ValueError("one submanifold flag per layer")
            flags = (ctypes.c_int32 * n)(*[int(x) for x in self.submanifold])
            _check(lib().sscater_create_sparse(ctypes.byref(grid), larr, n, wptrs, flags, ctypes.byref(handle)),
                   "sscater_create_sparse")
        elif self.pfn is not None:
            if self.ups:
                raise ValueError("points mode takes no neck")
            pw = np.ascontiguousarray(pfn_weights, dtype=np.float32)
            if pw.shape != (C0, 9):
                raise ValueError("pfn_weights must be [C0, 9]")
            spec = Pfn(float(self.pfn[0]), float(self.pfn[1]), float(self.pfn[2]), int(self.pfn[3]),
                       int(self.pfn[4]), int(self.pfn[5]))
            _check(lib().sscater_create_pfn(ctypes.byref(grid), larr, n, wptrs, ctypes.byref(spec),
                                            pw.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                            ctypes.byref(handle)), "sscater_create_pfn")
        elif self.ups:
            nu = len(self.ups)
            if len(up_weights) != nu:
                raise ValueError("one weight tensor per upsampler")
            self._ubufs = [weights_to_dtype_bytes(wt, dtype) for wt in up_weights]
            uarr = (Upsampler * nu)(*[Upsampler(src, co, s, int(bool(r))) for (src, co, s, r) in self.ups])
            uptrs = (ctypes.c_void_p * nu)(*[b.ctypes.data for b in self._ubufs])
            _check(lib().sscater_create_neck(ctypes.byref(grid), larr, n, wptrs, uarr, nu, uptrs,
                                             ctypes.byref(handle)), "sscater_create_neck")
            src0, _co, s0, _r = self.ups[0]
            hs, ws_, _c = self.shapes[src0]
            self.shapes.append((hs * s0, ws_ * s0, sum(u[1] for u in self.ups)))
            self._ubufs = None
        else:
            _check(lib().sscater_create(ctypes.byref(grid), larr, n, wptrs, ctypes.byref(handle)), "sscater_create")
        self._h = handle
        self._wbufs = None   # copied by the library

    # -- helpers ---------------------------------------------------------------
    def _stream(self, stream=None, tensors=()) -> ctypes.c_void_p:
        """The HIP stream handle of a call.  A stream other than the current
        one first waits for the current stream (where the caller's tensors
        were produced), and every tensor the call reads or writes is recorded
        on it, so the caching allocator does not hand the memory out again
        before the library's kernels on that stream are done with it."""
        t = self._torch
        cur = t.cuda.current_stream()
        s = stream if stream is not None else cur
        if s != cur:
            s.wait_stream(cur)
            for x in tensors:
                if x is not None:
                    x.record_stream(s)
        return ctypes.c_void_p(s.cuda_stream)

    @property
    def torch_dtype(self):
        return self._torch.float32 if self.dtype == "f32" else self._torch.bfloat16

    # -- C ABI calls -------------------------------------------------------------
    def step(self, idx, feats, stream=None, sorted=False) -> None:
        """idx: int32 cuda tensor [P] (or None for a dense [H, W, C0] canvas);
        feats: cuda tensor [P, C0] of the grid dtype (float32, or bf16 bits as
        int16/uint16/bfloat16).  sorted: idx increases strictly
        (sscater_step_sorted)."""
        if idx is not None:
            if idx.dtype != self._torch.int32 or not idx.is_cuda or not idx.is_contiguous():
                raise ValueError("idx must be a contiguous int32 cuda tensor")
            count = idx.numel()
        else:
            count = self.H * self.W * self.batch
        if count and (not feats.is_cuda or not feats.is_contiguous() or feats.element_size() !=
                      (4 if self.dtype == "f32" else 2) or feats.numel() != count * self.C0):
            raise ValueError("feats must be a contiguous cuda tensor [count, C0] of the grid dtype")
        p = Pillars(idx.data_ptr() if idx is not None else None, feats.data_ptr() if count else None, count)
        fn = lib().sscater_step_sorted if sorted else lib().sscater_step
        _check(fn(self._h, ctypes.byref(p), self._stream(stream, (idx, feats if count else None))),
               "sscater_step_sorted" if sorted else "sscater_step")

    def step_points(self, points, stream=None) -> None:
        """points: contiguous float32 cuda tensor [n, 4] = (x, y, z, intensity)
        of one stride (points mode)."""
        n = 0
        if points is not None:
            if points.dtype != self._torch.float32 or not points.is_cuda or not points.is_contiguous() or \
                    points.dim() != 2 or points.shape[1] != 4:
                raise ValueError("points must be a contiguous float32 cuda tensor [n, 4]")
            n = points.shape[0]
        ptr = ctypes.c_void_p(points.data_ptr() if n else None)
        _check(lib().sscater_step_points(self._h, ptr, n, self._stream(stream, (points if n else None,))),
               "sscater_step_points")

    def read(self, layer: int, out=None, stream=None):
        h, w, c = self.shapes[layer]
        if out is None:
            shape = (h, w, c) if self.batch == 1 else (self.batch, h, w, c)
            out = self._torch.empty(shape, dtype=self.torch_dtype, device="cuda")
        _check(lib().sscater_read(self._h, layer, ctypes.c_void_p(out.data_ptr()),
                                  out.numel() * out.element_size(), self._stream(stream, (out,))), "sscater_read")
        return out

    def reset(self, stream=None) -> None:
        _check(lib().sscater_reset(self._h, self._stream(stream)), "sscater_reset")

    def changed(self, layer: int, stream=None) -> np.ndarray:
        h, w, _ = self.shapes[layer]
        cap = h * w * self.batch
        buf = np.empty(cap, dtype=np.int32)
        cnt = ctypes.c_int32(0)
        _check(lib().sscater_changed(self._h, layer, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cap,
                                     ctypes.byref(cnt), self._stream(stream)), "sscater_changed")
        return buf[:cnt.value].copy()

    def changed_noalloc(self, layer: int, dst, count, stream=None) -> None:
        """The last stride's sorted change list of `layer` into the int32 cuda
        tensor dst (its capacity is dst.numel()) and its length into the
        one-element int32 cuda tensor count, enqueued on the stream; the
        library allocates nothing."""
        for t in (dst, count):
            if t.dtype != self._torch.int32 or not t.is_cuda or not t.is_contiguous():
                raise ValueError("dst and count must be contiguous int32 cuda tensors")
        if count.numel() < 1:
            raise ValueError("count needs one element")
        _check(lib().sscater_changed_noalloc(self._h, layer, ctypes.c_void_p(dst.data_ptr()), dst.numel(),
                                             ctypes.c_void_p(count.data_ptr()), self._stream(stream, (dst, count))),
               "sscater_changed_noalloc")

    def stats(self, stream=None) -> Dict:
        st = Stats()
        _check(lib().sscater_stats(self._h, ctypes.byref(st), self._stream(stream)), "sscater_stats")
        L = st.n_layers
        return dict(steps=st.steps, pillars=st.pillars, active=list(st.active[:L + 1]),
                    pairs=list(st.pairs[:L + 1]), active_total=list(st.active_total[:L + 1]),
                    pairs_total=list(st.pairs_total[:L + 1]), flops=st.flops, bytes=st.bytes,
                    up_pairs=list(st.up_pairs[:st.n_ups]))

    def profile(self, enable: bool) -> None:
        _check(lib().sscater_profile(self._h, int(bool(enable))), "sscater_profile")

    def profile_read(self, stream=None):
        """(ms per slot, launches per slot); slot 0 detect, 1 vanished, 1+l layer l
        (for a layer contracted in two launches: its tap sum), L+2+u upsampler u,
        L+1+n_ups+l the contraction launch of layer l when it has one."""
        n = 2 * len(self.layers) + 2 + len(self.ups)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check(lib().sscater_profile_read(self._h, ms, cnt, n, self._stream(stream)), "sscater_profile_read")
        return list(ms), list(cnt)

    def close(self) -> None:
        if getattr(self, "_h", None):
            _check(lib().sscater_destroy(self._h), "sscater_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
