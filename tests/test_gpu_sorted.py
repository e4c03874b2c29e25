"""The one-launch change detection for pillar lists sorted by cell
(sscater_step_sorted) through the C ABI: against the CPU oracle on the
backbone streams (lists bit for bit, maps within 1e-4 * max|ref| for fp32 and
2e-2 for bf16), and bit for bit against the two-pass detection of
sscater_step on random grids whose pillars appear and vanish: regions that
empty or fill at once (a previous chunk against a long stretch of the new
list), an empty list, a stride after a dense one and a stride after an
unsorted sscater_step call (both take the two passes)."""
import numpy as np
import pytest

import oracle
import streams as S
from gpu_util import check_lists, check_maps, layers_of, make_engine, note, run_stream, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu-test] start {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def test_c2_sorted_100_strides():
    run_stream("c2", map_every=10, sorted=True)


def test_c3_sorted_40_strides():
    run_stream("c3", n_strides=40, map_every=20, sorted=True)


def test_c4_sorted_60_strides():
    run_stream("c4", n_strides=60, map_every=30, sorted=True)


def _same(e1, e2, n_layers, where):
    for l in range(n_layers + 1):
        a, b = e1.changed(l), e2.changed(l)
        assert np.array_equal(a, b), f"{where}: A_{l} differs ({len(a)} vs {len(b)})"
    s1, s2 = e1.stats(), e2.stats()
    assert s1["active"] == s2["active"] and s1["pairs"] == s2["pairs"], where
    for l in range(n_layers + 1):
        x1, x2 = e1.read(l), e2.read(l)
        v1 = x1.view(torch.int32) if x1.element_size() == 4 else x1.view(torch.int16)
        v2 = x2.view(torch.int32) if x2.element_size() == 4 else x2.view(torch.int16)
        assert torch.equal(v1, v2), f"{where}: map {l} differs"


# (H, W, C0, layers, dtype): chunks of 48 rows (fp32 C0 = 16), 12 (fp32 C0 = 64)
# and 64 (bf16 C0 = 16) pillars.  The two large grids hold more pillars than
# 2048 one-pass chunks (24,576 fp32 rows of 64 channels, 49,152 bf16 ones), so
# their strides take the multi-pass chunks (60 and 48 rows), except where most
# pillars vanish
GRIDS = [
    (37, 23, 16, [(16, 32, 1, True), (32, 32, 2, True)], "f32"),
    (29, 31, 64, [(64, 64, 2, True), (64, 128, 1, True), (128, 128, 1, True)], "f32"),
    (40, 40, 16, [(16, 16, 1, True), (16, 32, 2, False)], "bf16"),
    (5, 300, 64, [(64, 64, 1, True)], "bf16"),
    (300, 300, 64, [(64, 64, 1, True)], "f32"),
    (420, 420, 64, [(64, 64, 2, True)], "bf16"),
]


@pytest.mark.parametrize("H,W,C0,layers,dtype", GRIDS)
def test_sorted_matches_two_pass_bitwise(H, W, C0, layers, dtype):
    rng = np.random.default_rng(H * 1000 + W + C0)
    ws = []
    for (ci, co, _s, _r) in layers:
        w = (rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2.0 / (9 * ci))).astype(np.float32)
        if dtype == "bf16":
            w = S.bf16_bits_to_f32(S.round_to_bf16_bits(w)).reshape(w.shape)
        ws.append(w)
    from paper_2512_08557_amd import Engine
    e1 = Engine(H, W, C0, layers, ws, dtype=dtype, max_pillars=H * W)
    e2 = Engine(H, W, C0, layers, ws, dtype=dtype, max_pillars=H * W)
    strides_l = [l[2] for l in layers]
    occ = rng.random(H * W) < 0.3
    feat = rng.standard_normal((H * W, C0)).astype(np.float32)
    prev_bits = np.zeros((H, W, C0), dtype=np.uint16 if dtype == "bf16" else np.uint32)

    def stride(t, occ, dense=False):
        nonlocal prev_bits
        idx = np.flatnonzero(occ).astype(np.int32)
        f = feat[idx]
        fb = S.round_to_bf16_bits(f).reshape(f.shape) if dtype == "bf16" else f.copy()
        st = S.Stride(t, idx, fb)
        if dense:
            c = S.canvas(st, H, W, C0)
            canvas = torch.from_numpy(c.view(np.int16) if dtype == "bf16" else c).cuda()
            e1.step(None, canvas, sorted=True)
            e2.step(None, canvas)
        else:
            d = to_device(st, dtype)
            e1.step(*d, sorted=True)
            e2.step(*d)
        _same(e1, e2, len(layers), f"stride {t} P={len(idx)}")
        bits = oracle.canvas_bits(S.canvas(st, H, W, C0), dtype)
        check_lists(e1, oracle.changed_lists(prev_bits, bits, strides_l), f"stride {t}")
        prev_bits = bits
        return st

    t = 0
    stride(t, occ)
    for t in range(1, 9):                              # refreshes and toggles, both ends of the grid included
        tog = rng.random(H * W) < 0.1
        tog[:3] = True
        tog[-3:] = True
        occ = occ ^ tog
        r = rng.random(H * W) < 0.15
        feat[r] = rng.standard_normal((int(r.sum()), C0))
        stride(t, occ)
    keep = occ & (rng.random(H * W) < 0.1)             # most pillars vanish
    stride(9, keep)
    stride(10, occ)                                    # they come back
    stride(11, np.zeros(H * W, bool))                  # an empty list
    stride(12, occ)
    stride(13, occ, dense=True)                        # a dense stride, then the previous list is all cells
    occ = occ ^ (rng.random(H * W) < 0.1)
    stride(14, occ)
    occ = occ ^ (rng.random(H * W) < 0.1)
    stride(15, occ)
    stride(16, occ)                                    # nothing changed
    assert e1.stats()["active"][0] == 0
    grid = occ.reshape(H, W).copy()
    r0, r1 = H // 4, max(H // 4 + 1, 3 * H // 4)
    grid[r0:r1, :] = False                             # a band empties at once
    occ = grid.reshape(-1)
    stride(17, occ)
    grid[r0:r1, :] = True                              # and fills completely: a long stretch of new cells
    occ = grid.reshape(-1)                             # between two previous ones
    r = rng.random(H * W) < 0.5
    feat[r] = rng.standard_normal((int(r.sum()), C0))
    stride(18, occ)
    occ = occ ^ (rng.random(H * W) < 0.05)
    st = stride(19, occ)
    x = oracle.exact_canvas(S.canvas(st, H, W, C0), dtype)
    check_maps(e1, oracle.forward(x, ws, layers, bf16_storage=(dtype == "bf16")),
               1e-4 if dtype == "f32" else 2e-2, "end")
    e1.close()
    e2.close()


def test_sorted_after_an_unsorted_step():
    """A stride through sscater_step with a shuffled list, then sorted strides:
    the first of them takes the two passes (its previous list is not
    sorted), the next ones the one launch; all equal the two passes."""
    wl = S.workload("c4")
    ws = S.weights("c4")
    strides = S.make_stream("c4", n_strides=5)
    e1, e2 = make_engine(wl, ws), make_engine(wl, ws)
    rng = np.random.default_rng(3)
    for t, st in enumerate(strides):
        idx, feats = to_device(st, wl.dtype)
        if t == 1:
            perm = torch.from_numpy(rng.permutation(len(st.idx))).cuda()
            e1.step(idx[perm].contiguous(), feats[perm].contiguous())
        else:
            e1.step(idx, feats, sorted=True)
        e2.step(idx, feats)
        _same(e1, e2, len(wl.layers), f"stride {t}")
    e1.close()
    e2.close()


def test_sorted_batched_images():
    """A batched handle: cells b*H*W + r*W + c, sorted over the whole batch."""
    from paper_2512_08557_amd import Engine
    H, W, C0, B = 24, 19, 64, 3
    layers = [(64, 64, 2, True), (64, 64, 1, True)]
    rng = np.random.default_rng(7)
    ws = [(rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2.0 / (9 * ci))).astype(np.float32)
          for (ci, co, _s, _r) in layers]
    e1 = Engine(H, W, C0, layers, ws, max_pillars=B * H * W, batch=B)
    e2 = Engine(H, W, C0, layers, ws, max_pillars=B * H * W, batch=B)
    occ = rng.random(B * H * W) < 0.25
    feat = rng.standard_normal((B * H * W, C0)).astype(np.float32)
    for t in range(8):
        if t:
            occ = occ ^ (rng.random(B * H * W) < 0.1)
            if t == 4:
                occ[H * W:2 * H * W] = False             # image 1 empties
            r = rng.random(B * H * W) < 0.2
            feat[r] = rng.standard_normal((int(r.sum()), C0))
        idx = torch.from_numpy(np.flatnonzero(occ).astype(np.int32)).cuda()
        f = torch.from_numpy(feat[np.flatnonzero(occ)]).cuda()
        e1.step(idx, f, sorted=True)
        e2.step(idx, f)
        _same(e1, e2, len(layers), f"batched stride {t}")
    e1.close()
    e2.close()


def test_unsorted_list_passed_as_sorted_is_flagged():
    from paper_2512_08557_amd import E_DEVICE, SscaterError
    wl = S.workload("c1")
    ws = S.weights("c1")
    eng = make_engine(wl, ws)
    st = S.make_stream("c1", n_strides=0)[0]
    idx, feats = to_device(st, "f32")
    eng.step(idx, feats, sorted=True)
    perm = torch.from_numpy(np.random.default_rng(1).permutation(len(st.idx))).cuda()
    eng.step(idx[perm].contiguous(), feats[perm].contiguous(), sorted=True)
    torch.cuda.synchronize()
    with pytest.raises(SscaterError) as ei:
        eng.step(idx, feats, sorted=True)
    assert ei.value.code == E_DEVICE
    eng.reset()
    eng.step(idx, feats, sorted=True)
    x = oracle.exact_canvas(S.canvas(st, wl.H, wl.W, wl.C0), "f32")
    check_maps(eng, oracle.forward(x, ws, layers_of(wl)), 1e-4, "after reset")
    eng.close()
