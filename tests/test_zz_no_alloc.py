"""GPU test of the allocation-free change list (sscater_changed_noalloc):
called through the C ABI, its device-built sorted list and count equal those
of sscater_changed exactly, on two calls in a row with the second over a
smaller list, after every stride of the block-1 stream, with a truncating
capacity, on a sparse handle (restricted lists), before the first stride,
and a grid above the fixed scratch's 64 Mi cells is refused."""
import numpy as np
import pytest

import streams as S
from gpu_util import make_engine, note, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

SENTINEL = -7


def _device_list(eng, layer, cap):
    dst = torch.full((cap + 8,), SENTINEL, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), SENTINEL, dtype=torch.int32, device="cuda")
    eng.changed_noalloc(layer, dst[:cap], cnt)
    torch.cuda.synchronize()
    return dst.cpu().numpy(), int(cnt.item())


def _check(eng, layer, cap=None):
    ref = eng.changed(layer)
    h, w, _c = eng.shapes[layer]
    cap = h * w * eng.batch if cap is None else cap
    got, n = _device_list(eng, layer, cap)
    assert n == len(ref), f"layer {layer}: count {n} != {len(ref)}"
    k = min(n, cap)
    np.testing.assert_array_equal(got[:k], ref[:k], err_msg=f"layer {layer}")
    assert np.all(got[k:] == SENTINEL), f"layer {layer}: wrote past the list"
    return n


def test_block1_stream_two_calls_in_a_row_second_smaller():
    wl = S.workload("c2")
    eng = make_engine(wl, S.weights("c2"))
    strides = S.make_stream("c2", n_strides=4)
    _, n = _device_list(eng, 1, 16)
    assert n == 0                                     # nothing stepped yet
    for t, st in enumerate(strides):
        note(f"[gpu-test] no-alloc list, c2 stride {t}")
        eng.step(*to_device(st, wl.dtype))
        # the largest list first, then every smaller one in turn
        sizes = {l: len(eng.changed(l)) for l in range(len(wl.layers) + 1)}
        order = sorted(sizes, key=lambda l: -sizes[l])
        last = None
        for l in order:
            n = _check(eng, l)
            assert last is None or n <= last
            last = n
        # a capacity below the list length writes a prefix and reports the length
        _check(eng, order[0], cap=max(1, sizes[order[0]] // 3))
        _check(eng, order[0], cap=0)
    eng.reset()
    assert _device_list(eng, 2, 16)[1] == 0
    eng.close()


def test_sparse_handle_lists_are_restricted_like_the_host_list():
    wl = S.workload("s2")
    eng = make_engine(wl, S.weights("s2"), submanifold=[l.sub for l in wl.layers])
    for t, st in enumerate(S.make_stream("s2", n_strides=3)):
        note(f"[gpu-test] no-alloc list, s2 stride {t}")
        eng.step(*to_device(st, wl.dtype))
        for l in range(len(wl.layers) + 1):
            _check(eng, l)
    eng.close()


def test_grid_above_the_scratch_limit_is_refused():
    from paper_2512_08557_amd import Engine, SscaterError
    from paper_2512_08557_amd.engine import E_SCRATCH
    H, W, C0, B = 1025, 1024, 16, 64                 # 64 x 1025 x 1024 cells > 64 Mi
    rng = np.random.default_rng(5)
    w = (rng.standard_normal((16, 16, 3, 3)) * 0.1).astype(np.float32)
    eng = Engine(H, W, C0, [(16, 16, 2, True)], [w], max_pillars=256, batch=B)
    cells = rng.choice(B * H * W, 200, replace=False).astype(np.int32)
    feats = rng.standard_normal((200, C0)).astype(np.float32)
    eng.step(torch.from_numpy(cells).cuda(), torch.from_numpy(feats).cuda())
    dst = torch.zeros(16, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(SscaterError) as ei:
        eng.changed_noalloc(0, dst, cnt)
    assert ei.value.code == E_SCRATCH
    _check(eng, 1)                                   # 64 x 513 x 512 cells fit
    eng.close()
