"""GPU tests of batched handles (several independent images advanced by one
launch chain): every image's maps and change lists equal those of a handle of
its own exactly, on the four-stream 1024x1024 workload and on random stacks
with ragged grids, stride-2 layers and toggles; one image is also checked
against the CPU oracle."""
import numpy as np
import pytest

import oracle
import streams as S
from gpu_util import canvas_bits, check_lists, check_maps, layers_of, make_engine, note, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu-test] start {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _batched(H, W, C0, layers, ws, dtype, B, max_pillars):
    from paper_2512_08557_amd import Engine
    return Engine(H, W, C0, layers, ws, dtype=dtype, max_pillars=max_pillars, batch=B)


def _stack(strides, H, W):
    """One batched stride from per-image strides: cell b*H*W + p."""
    idx = np.concatenate([s.idx.astype(np.int64) + b * H * W for b, s in enumerate(strides)]).astype(np.int32)
    feats = np.concatenate([s.feats for s in strides])
    return S.Stride(strides[0].index, idx, np.ascontiguousarray(feats))


def _compare(beng, sengs, L, where):
    for l in range(L + 1):
        got = beng.read(l)
        for b, e in enumerate(sengs):
            ref = e.read(l)
            assert torch.equal(got[b], ref), f"{where}: layer {l} image {b} differs"
        lists = []
        for b, e in enumerate(sengs):
            h, w, _c = e.shapes[l]
            lists.append(e.changed(l).astype(np.int64) + b * h * w)
        np.testing.assert_array_equal(beng.changed(l), np.concatenate(lists), err_msg=f"{where}: A_{l}")


def test_four_stream_drone_grid_in_one_handle():
    """The four 1024x1024 streams in one batched handle with the one-launch
    detection of its sorted pillar list (the bench's default launch
    configuration for this workload; ~160k pillars, so the multi-pass chunks)
    over the full 100 delta strides, against handles of their own that take
    the two detection passes:
    every 10th stride each image equals a handle of its own bit for bit, and
    every 20th stride and the last one image (in turn) is checked against the
    oracle."""
    wl = S.workload("c5")
    ws = S.weights("c5")
    B, n = 4, 100
    gens = [S.make_stream("c5", seed=S.SCENE_SEED + k, n_strides=n) for k in range(B)]
    beng = _batched(wl.H, wl.W, wl.C0, layers_of(wl), ws, wl.dtype, B, B * wl.max_pillars)
    sengs = [make_engine(wl, ws) for _ in range(B)]
    for t in range(n + 1):
        note(f"[gpu-test] c5 batched stride {t}")
        for b in range(B):
            sengs[b].step(*to_device(gens[b][t], wl.dtype))
        beng.step(*to_device(_stack([g[t] for g in gens], wl.H, wl.W), wl.dtype), sorted=True)
        if t % 10 == 0 or t == n:
            _compare(beng, sengs, len(wl.layers), f"stride {t}")
        if t % 20 == 0 or t == n:
            img = (t // 20) % B
            x = oracle.exact_canvas(S.canvas(gens[img][t], wl.H, wl.W, wl.C0), wl.dtype)
            ys = oracle.forward(x, ws, layers_of(wl))
            for l, y in enumerate(ys, start=1):
                got = beng.read(l)[img].cpu().numpy().astype(np.float64)
                err, scale = float(np.abs(got - y).max()), float(np.abs(y).max())
                assert err <= 1e-4 * scale, f"stride {t} image {img} layer {l}: {err:.3e} vs {scale:.3e}"
    for e in sengs + [beng]:
        e.close()


STACKS = [
    (13, 21, 16, [(16, 32, 2, True), (32, 32, 1, True), (32, 64, 2, False)], "f32", 3),
    (9, 7, 64, [(64, 64, 1, True), (64, 128, 2, True), (128, 128, 1, True)], "f32", 2),
    (17, 11, 32, [(32, 32, 2, True), (32, 16, 1, True)], "bf16", 5),
]


@pytest.mark.parametrize("H,W,C0,layers,dtype,B", STACKS)
def test_random_batched_stacks_equal_separate_handles(H, W, C0, layers, dtype, B):
    from paper_2512_08557_amd import Engine
    rng = np.random.default_rng(H * 31 + W * 7 + B)
    ws = []
    for (ci, co, _s, _r) in layers:
        w = (rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2.0 / (9 * ci))).astype(np.float32)
        if dtype == "bf16":
            w = S.bf16_bits_to_f32(S.round_to_bf16_bits(w)).reshape(w.shape)
        ws.append(w)
    beng = _batched(H, W, C0, layers, ws, dtype, B, B * H * W)
    sengs = [Engine(H, W, C0, layers, ws, dtype=dtype, max_pillars=H * W) for _ in range(B)]
    occ = rng.random((B, H * W)) < 0.3
    feat = np.zeros((B, H * W, C0), np.float32)
    feat[occ] = rng.standard_normal((int(occ.sum()), C0))
    for t in range(15):
        if t:
            tog = rng.random((B, H * W)) < 0.05
            feat[tog & occ] = 0.0
            on = tog & ~occ
            feat[on] = rng.standard_normal((int(on.sum()), C0))
            occ = occ ^ tog
            r = occ & (rng.random((B, H * W)) < 0.1)
            feat[r] = rng.standard_normal((int(r.sum()), C0))
        per = []
        for b in range(B):
            idx = np.flatnonzero(occ[b]).astype(np.int32)
            idx = idx[rng.permutation(len(idx))]
            f = feat[b][idx]
            if dtype == "bf16":
                fb = S.round_to_bf16_bits(f).reshape(f.shape)
                feat[b][idx] = S.bf16_bits_to_f32(fb).reshape(f.shape)
                per.append(S.Stride(t, idx, fb))
            else:
                per.append(S.Stride(t, idx, f.copy()))
            sengs[b].step(*to_device(per[-1], dtype))
        st = _stack(per, H, W)
        order = rng.permutation(len(st.idx))                 # pillars of all images interleaved
        beng.step(*to_device(S.Stride(t, st.idx[order], np.ascontiguousarray(st.feats[order])), dtype))
        _compare(beng, sengs, len(layers), f"stride {t}")
    for e in sengs + [beng]:
        e.close()


def test_batched_reset_empty_image_and_zero_change():
    """A batch whose middle image never holds a pillar: its maps stay exactly
    zero and its lists empty; a repeated stride changes nothing anywhere; after
    reset the next stride is the full pass of every image again."""
    rng = np.random.default_rng(77)
    H, W, C0, B = 11, 13, 32, 3
    layers = [(32, 32, 1, True), (32, 64, 2, True), (64, 64, 1, True)]
    ws = [(rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2.0 / (9 * ci))).astype(np.float32)
          for (ci, co, _s, _r) in layers]
    beng = _batched(H, W, C0, layers, ws, "f32", B, B * H * W)
    seng = [make_engine_like(H, W, C0, layers, ws) for _ in (0, 2)]

    def stride(t):
        per = []
        for b in (0, 2):
            r = np.random.default_rng((t, b))
            idx = np.flatnonzero(r.random(H * W) < 0.4).astype(np.int32)
            per.append(S.Stride(t, idx, r.standard_normal((len(idx), C0)).astype(np.float32)))
        return per

    def run(t, per):
        for e, st in zip(seng, per):
            e.step(*to_device(st, "f32"))
        empty = S.Stride(t, np.zeros(0, np.int32), np.zeros((0, C0), np.float32))
        st = _stack([per[0], empty, per[1]], H, W)
        beng.step(*to_device(st, "f32"))

    def check(where):
        for l in range(len(layers) + 1):
            got = beng.read(l)
            assert torch.equal(got[0], seng[0].read(l)), f"{where}: layer {l} image 0"
            assert torch.equal(got[2], seng[1].read(l)), f"{where}: layer {l} image 2"
            assert int(torch.count_nonzero(got[1])) == 0, f"{where}: layer {l} empty image not zero"
            h, w, _c = seng[0].shapes[l]
            ref = np.concatenate([seng[0].changed(l).astype(np.int64), seng[1].changed(l).astype(np.int64) + 2 * h * w])
            np.testing.assert_array_equal(beng.changed(l), ref, err_msg=f"{where}: A_{l}")

    for t in range(4):
        per = stride(t)
        run(t, per)
        check(f"stride {t}")
    before = [beng.read(l).clone() for l in range(len(layers) + 1)]
    run(4, per)                                   # the same input again
    for l in range(len(layers) + 1):
        assert torch.equal(beng.read(l), before[l]), f"zero-change stride moved layer {l}"
        assert len(beng.changed(l)) == 0, f"zero-change stride listed cells in A_{l}"
    beng.reset()
    for e in seng:
        e.reset()
    run(5, stride(5))
    check("after reset")
    for e in seng + [beng]:
        e.close()


def make_engine_like(H, W, C0, layers, ws):
    from paper_2512_08557_amd import Engine
    return Engine(H, W, C0, layers, ws, dtype="f32", max_pillars=H * W)
