"""Helpers for the GPU parity tests: marshal seeded streams to the device,
read the library's maps and lists back, and compare them with the oracle."""
import sys

import numpy as np

import oracle
import streams as S


def layers_of(wl):
    return [(l.cin, l.cout, l.stride, bool(l.relu)) for l in wl.layers]


def make_engine(wl, ws, **kw):
    from paper_2512_08557_amd import Engine
    return Engine(wl.H, wl.W, wl.C0, layers_of(wl), ws, dtype=wl.dtype,
                  max_pillars=kw.pop("max_pillars", wl.max_pillars), **kw)


def to_device(stride, dtype):
    import torch
    idx = torch.from_numpy(np.ascontiguousarray(stride.idx, dtype=np.int32)).cuda()
    f = stride.feats.view(np.int16) if dtype == "bf16" else stride.feats
    return idx, torch.from_numpy(np.ascontiguousarray(f)).cuda()


def canvas_bits(stride, wl):
    return oracle.canvas_bits(S.canvas(stride, wl.H, wl.W, wl.C0), wl.dtype)


def read_map(eng, layer):
    """Layer map as exact float64 values (bf16 maps decoded from their bits)."""
    import torch
    t = eng.read(layer)
    torch.cuda.synchronize()
    if eng.dtype == "bf16":
        b = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return oracle.exact_canvas(b, "bf16")
    return t.cpu().numpy().astype(np.float64)


def check_lists(eng, ref_lists, where=""):
    for l, ref in enumerate(ref_lists):
        got = eng.changed(l)
        if not np.array_equal(got, ref):
            extra = np.setdiff1d(got, ref)[:10]
            miss = np.setdiff1d(ref, got)[:10]
            raise AssertionError(f"{where} A_{l}: |gpu|={len(got)} |ref|={len(ref)} extra={extra} missing={miss}")


def map_errors(eng, ys_ref):
    out = []
    for l, ref in enumerate(ys_ref, start=1):
        got = read_map(eng, l)
        assert got.shape == ref.shape
        out.append((float(np.abs(got - ref).max()), float(np.abs(ref).max())))
    return out


def check_maps(eng, ys_ref, tol, where=""):
    for l, (err, scale) in enumerate(map_errors(eng, ys_ref), start=1):
        if scale == 0.0:
            assert err <= 1e-6, f"{where} layer {l}: reference is zero, max|gpu| = {err}"
        else:
            assert err <= tol * scale, f"{where} layer {l}: max err {err:.3e} > {tol} * {scale:.3e}"


def note(msg):
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()
