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
    wl = S.workload("c5")
    ws = S.weights("c5")
    B, n = 4, 12
    gens = [S.make_stream("c5", seed=S.SCENE_SEED + k, n_strides=n) for k in range(B)]
    beng = _batched(wl.H, wl.W, wl.C0, layers_of(wl), ws, wl.dtype, B, B * wl.max_pillars)
    sengs = [make_engine(wl, ws) for _ in range(B)]
    for t in range(n + 1):
        note(f"[gpu-test] c5 batched stride {t}")
        for b in range(B):
            sengs[b].step(*to_device(gens[b][t], wl.dtype))
        beng.step(*to_device(_stack([g[t] for g in gens], wl.H, wl.W), wl.dtype))
        if t % 4 == 0 or t == n:
            _compare(beng, sengs, len(wl.layers), f"stride {t}")
    x = oracle.exact_canvas(S.canvas(gens[2][n], wl.H, wl.W, wl.C0), wl.dtype)
    ys = oracle.forward(x, ws, layers_of(wl))
    for l, y in enumerate(ys, start=1):
        got = beng.read(l)[2].cpu().numpy().astype(np.float64)
        assert np.abs(got - y).max() <= 1e-4 * np.abs(y).max()
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
