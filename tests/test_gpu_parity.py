"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Lists and counts must match bit for bit; maps within max|err| <= tol * max|ref|
per layer (fp32: 1e-4, bf16: 2e-2), relative to the oracle's dense float64
recomputation of the same window.
"""
import numpy as np
import pytest

import oracle
import streams as S
from gpu_util import (canvas_bits, check_lists, check_maps, layers_of, make_engine, note, oracle_maps, read_map,
                      run_stream, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu-test] start {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def test_c1_single_layer_all_strides():
    run_stream("c1", map_every=1)


def test_c2_block1_100_strides():
    run_stream("c2", map_every=10)


def test_c3_backbone_100_strides():
    run_stream("c3", map_every=25)


def test_c4_backbone_bf16_200_strides():
    run_stream("c4", map_every=50)


@pytest.mark.parametrize("name,n", [("c3", 20), ("c4", 30)])
def test_one_launch_wide_layers(name, n, monkeypatch):
    """The wide stride-1 layers in the one-launch output-stationary kernel
    (SSCATER_FUSED_WIDE=1, read when a handle is created) instead of the
    contraction and tap sum: its tap groups over the nine stride-1 taps."""
    monkeypatch.setenv("SSCATER_FUSED_WIDE", "1")
    run_stream(name, n_strides=n, map_every=10)


def test_c5_four_concurrent_streams():
    name = "c5"
    wl = S.workload(name)
    ws = S.weights(name)
    n = 100
    gens = [iter(S.Stream(name, seed=S.SCENE_SEED + k, n_strides=n)) for k in range(4)]
    engs = [make_engine(wl, ws) for _ in range(4)]
    hip_streams = [torch.cuda.Stream() for _ in range(4)]
    prev = [np.zeros((wl.H, wl.W, wl.C0), dtype=np.uint32) for _ in range(4)]
    strides_l = [l.stride for l in wl.layers]
    for t in range(n + 1):
        sts = [next(g) for g in gens]
        devs = [to_device(s, wl.dtype) for s in sts]
        torch.cuda.synchronize()
        for k in range(4):
            with torch.cuda.stream(hip_streams[k]):
                engs[k].step(*devs[k], stream=hip_streams[k])
        if t % 10 == 0 or t == n:
            note(f"[gpu-test] c5 check stride {t}")
            for k in range(4):
                hip_streams[k].synchronize()
                bits = canvas_bits(sts[k], wl)
                check_lists(engs[k], oracle.changed_lists(prev[k], bits, strides_l), f"c5[{k}] stride {t}")
                check_maps(engs[k], oracle_maps(sts[k], wl, ws), TOL["f32"], f"c5[{k}] stride {t}")
        else:
            for k in range(4):
                hip_streams[k].synchronize()
        for k in range(4):
            prev[k] = canvas_bits(sts[k], wl)
    for e in engs:
        e.close()


# ---------------------------------------------------------------- invariants
def _c2_engine_and_strides(n=6):
    wl = S.workload("c2")
    ws = S.weights("c2")
    return wl, ws, S.make_stream("c2", n_strides=n), make_engine(wl, ws)


def test_zero_change_stride_leaves_everything_bitwise():
    wl, ws, strides, eng = _c2_engine_and_strides(3)
    for st in strides:
        eng.step(*to_device(st, wl.dtype))
    before = [eng.read(l).clone() for l in range(len(wl.layers) + 1)]
    eng.step(*to_device(strides[-1], wl.dtype))
    st = eng.stats()
    assert st["active"] == [0] * (len(wl.layers) + 1)
    assert st["pairs"] == [0] * (len(wl.layers) + 1) and st["flops"] == 0.0
    for l in range(len(wl.layers) + 1):
        assert torch.equal(before[l].view(torch.int32), eng.read(l).view(torch.int32))
    eng.close()


def test_reset_equivalence_and_full_pass_list():
    wl, ws, strides, eng = _c2_engine_and_strides(8)
    for st in strides:
        eng.step(*to_device(st, wl.dtype))
    acc = [read_map(eng, l) for l in range(1, len(wl.layers) + 1)]
    eng.reset()
    eng.step(*to_device(strides[-1], wl.dtype))
    full = [read_map(eng, l) for l in range(1, len(wl.layers) + 1)]
    for a, b in zip(acc, full):
        assert np.abs(a - b).max() <= 1e-4 * np.abs(b).max()
    nz = np.flatnonzero(np.any(S.canvas(strides[-1], wl.H, wl.W, wl.C0) != 0, axis=-1))
    np.testing.assert_array_equal(eng.changed(0), nz)
    assert eng.stats()["steps"] == 1
    eng.close()


def test_round_trip_returns_to_the_same_maps():
    wl, ws, strides, eng = _c2_engine_and_strides(3)
    a, b = strides[1], strides[3]
    eng.step(*to_device(a, wl.dtype))
    ref = [read_map(eng, l) for l in range(1, len(wl.layers) + 1)]
    eng.step(*to_device(b, wl.dtype))
    eng.step(*to_device(a, wl.dtype))
    for l, r in enumerate(ref, start=1):
        assert np.abs(read_map(eng, l) - r).max() <= 1e-4 * np.abs(r).max()
    eng.close()


def test_two_runs_are_bitwise_identical():
    wl, ws, strides, e1 = _c2_engine_and_strides(5)
    e2 = make_engine(wl, ws)
    for st in strides:
        d = to_device(st, wl.dtype)
        e1.step(*d)
        e2.step(*d)
        for l in range(len(wl.layers) + 1):
            np.testing.assert_array_equal(e1.changed(l), e2.changed(l))
    for l in range(1, len(wl.layers) + 1):
        assert torch.equal(e1.read(l).view(torch.int32), e2.read(l).view(torch.int32))
    e1.close()
    e2.close()


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_maps_do_not_depend_on_the_pillar_order(name):
    """One handle fed every stride's pillars in cell order, one fed them in a
    fresh random order: the change lists then come out of the atomics in
    different orders (and the tiles of every layer hold different cells), yet
    every list and every map must be bit-identical, the full backbone's
    stride-2 wide layer included (its tap groups must not depend on which
    cells share a tile pair)."""
    wl = S.workload(name)
    ws = S.weights(name)
    strides = S.make_stream(name, n_strides=8)
    e1, e2 = make_engine(wl, ws), make_engine(wl, ws)
    rng = np.random.default_rng(11)
    for t, st in enumerate(strides):
        idx, feats = to_device(st, wl.dtype)
        perm = torch.from_numpy(rng.permutation(len(st.idx))).cuda()
        e1.step(idx, feats)
        e2.step(idx[perm].contiguous(), feats[perm].contiguous())
        for l in range(len(wl.layers) + 1):
            np.testing.assert_array_equal(e1.changed(l), e2.changed(l), err_msg=f"stride {t} A_{l}")
        for l in range(len(wl.layers) + 1):
            x1, x2 = e1.read(l), e2.read(l)
            v1 = x1.view(torch.int32) if x1.element_size() == 4 else x1.view(torch.int16)
            v2 = x2.view(torch.int32) if x2.element_size() == 4 else x2.view(torch.int16)
            assert torch.equal(v1, v2), f"stride {t}: map {l} differs"
    e1.close()
    e2.close()


def test_dense_mode_matches_pillar_mode():
    wl, ws, strides, e1 = _c2_engine_and_strides(3)
    e2 = make_engine(wl, ws)
    for st in strides:
        e1.step(*to_device(st, wl.dtype))
        canvas = torch.from_numpy(S.canvas(st, wl.H, wl.W, wl.C0)).cuda()
        e2.step(None, canvas)
        for l in range(len(wl.layers) + 1):
            np.testing.assert_array_equal(e1.changed(l), e2.changed(l))
    # back to pillar mode after a dense stride: vanished pillars are found
    st = strides[-1]
    keep = np.arange(len(st.idx)) % 7 != 0
    sub = S.Stride(st.index, st.idx[keep], st.feats[keep])
    e1.step(*to_device(sub, wl.dtype))
    e2.step(*to_device(sub, wl.dtype))
    for l in range(len(wl.layers) + 1):
        np.testing.assert_array_equal(e1.changed(l), e2.changed(l))
    for l in range(1, len(wl.layers) + 1):
        assert torch.equal(e1.read(l).view(torch.int32), e2.read(l).view(torch.int32))
    e1.close()
    e2.close()


def test_error_paths():
    from paper_2512_08557_amd import E_DEVICE, E_OVERFLOW, SscaterError
    wl = S.workload("c1")
    ws = S.weights("c1")
    eng = make_engine(wl, ws, max_pillars=500)
    st = S.make_stream("c1", n_strides=0)[0]
    # more pillars than the budget: refused before any device work
    big_idx = torch.arange(501, dtype=torch.int32, device="cuda")
    big_f = torch.zeros((501, wl.C0), dtype=torch.float32, device="cuda")
    with pytest.raises(SscaterError) as ei:
        eng.step(big_idx, big_f)
    assert ei.value.code == E_OVERFLOW
    # a cell index outside the grid: the kernel's bounds check flags it
    idx, feats = to_device(st, "f32")
    bad = idx.clone()
    bad[5] = wl.H * wl.W + 3
    eng.step(bad, feats)
    torch.cuda.synchronize()
    with pytest.raises(SscaterError) as ei:
        eng.step(idx, feats)
    assert ei.value.code == E_DEVICE
    eng.reset()
    eng.step(idx, feats)
    torch.cuda.synchronize()
    # duplicate indices within one stride
    dup = idx.clone()
    dup[3] = dup[4]
    eng.step(dup, feats)
    torch.cuda.synchronize()
    with pytest.raises(SscaterError) as ei:
        eng.read(1)
    assert ei.value.code == E_DEVICE
    eng.reset()
    eng.step(idx, feats)
    x = oracle.exact_canvas(S.canvas(st, wl.H, wl.W, wl.C0), "f32")
    check_maps(eng, oracle.forward(x, ws, layers_of(wl)), 1e-4, "after reset")
    eng.close()


def test_empty_stride_and_empty_grid_regions():
    wl = S.workload("c1")
    ws = S.weights("c1")
    eng = make_engine(wl, ws)
    empty_i = torch.zeros(0, dtype=torch.int32, device="cuda")
    empty_f = torch.zeros((0, wl.C0), dtype=torch.float32, device="cuda")
    eng.step(empty_i, empty_f)
    assert eng.stats()["active"] == [0, 0]
    st = S.make_stream("c1", n_strides=0)[0]
    eng.step(*to_device(st, "f32"))
    eng.step(empty_i, empty_f)       # every pillar vanishes
    assert eng.stats()["active"][0] == len(st.idx)
    assert np.abs(read_map(eng, 1)).max() <= 1e-6
    eng.close()


# ---------------------------------------------------------------- random stacks
STACKS = [
    (9, 11, 16, [(16, 32, 1, True), (32, 16, 2, True), (16, 16, 1, False)], "f32"),
    (17, 5, 32, [(32, 64, 2, False), (64, 64, 2, True)], "f32"),
    (23, 31, 64, [(64, 128, 2, True), (128, 256, 2, True), (256, 256, 1, True)], "f32"),
    (1, 1, 16, [(16, 16, 1, True), (16, 16, 2, True)], "f32"),
    (40, 3, 16, [(16, 16, 2, True)] * 4, "f32"),
    (13, 21, 16, [(16, 32, 1, True), (32, 32, 2, True), (32, 64, 1, False)], "bf16"),
    (33, 29, 64, [(64, 64, 2, True), (64, 128, 1, True)], "bf16"),
    (19, 23, 32, [(32, 8, 1, True)], "f32"),
    (21, 17, 128, [(128, 8, 2, False)], "f32"),
    (15, 26, 16, [(16, 8, 1, True)], "bf16"),
]


@pytest.mark.parametrize("H,W,C0,layers,dtype", STACKS)
def test_random_stacks_with_toggles(H, W, C0, layers, dtype):
    rng = np.random.default_rng(H * 1000 + W)
    ws = []
    for (ci, co, s, r) in layers:
        w = (rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2.0 / (9 * ci))).astype(np.float32)
        if dtype == "bf16":
            w = S.bf16_bits_to_f32(S.round_to_bf16_bits(w)).reshape(w.shape)
        ws.append(w)
    from paper_2512_08557_amd import Engine
    eng = Engine(H, W, C0, layers, ws, dtype=dtype, max_pillars=H * W)
    occ = rng.random(H * W) < 0.3
    feat = np.zeros((H * W, C0), np.float32)
    feat[occ] = rng.standard_normal((int(occ.sum()), C0))
    prev = None
    for t in range(25):
        if t:
            r = occ & (rng.random(H * W) < 0.1)
            feat[r] = rng.standard_normal((int(r.sum()), C0))
            tog = rng.random(H * W) < 0.03
            feat[tog & occ] = 0.0
            on = tog & ~occ
            feat[on] = rng.standard_normal((int(on.sum()), C0))
            occ = occ ^ tog
        idx = np.flatnonzero(occ).astype(np.int32)
        perm = rng.permutation(len(idx))          # unsorted pillar order is allowed
        idx = idx[perm]
        f = feat[idx]
        if dtype == "bf16":
            fb = S.round_to_bf16_bits(f).reshape(f.shape)
            feat[idx] = S.bf16_bits_to_f32(fb).reshape(f.shape)
            st = S.Stride(t, idx, fb)
        else:
            st = S.Stride(t, idx, f.copy())
        eng.step(*to_device(st, dtype))
        canvas = S.canvas(st, H, W, C0)
        bits = oracle.canvas_bits(canvas, dtype)
        pb = np.zeros_like(bits) if prev is None else prev
        check_lists(eng, oracle.changed_lists(pb, bits, [l[2] for l in layers]), f"stride {t}")
        prev = bits
    x = oracle.exact_canvas(canvas, dtype)
    check_maps(eng, oracle.forward(x, ws, layers, bf16_storage=(dtype == "bf16")), TOL[dtype], "final")
    eng.close()
