"""Synthetic input streams: determinism and the workload shapes they stand for."""
import numpy as np
import pytest

import streams as S


def test_deterministic_and_sorted():
    a = S.make_stream("c1")
    b = S.make_stream("c1")
    assert len(a) == 11
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x.idx, y.idx)
        np.testing.assert_array_equal(x.feats.view(np.uint32), y.feats.view(np.uint32))
        assert np.all(np.diff(x.idx) > 0)
        assert x.idx.dtype == np.int32 and x.feats.dtype == np.float32


@pytest.mark.parametrize("name,target", [("c2", 12000), ("c5", 40000)])
def test_occupancy_near_target(name, target):
    st = S.Stream(name, n_strides=2)
    first = next(iter(st))
    assert abs(len(first.idx) - target) <= 0.05 * target


def test_c2_sector_refresh_fraction():
    strides = S.make_stream("c2", n_strides=3)
    for prev, cur in zip(strides, strides[1:]):
        np.testing.assert_array_equal(prev.idx, cur.idx)       # static scene
        changed = np.any(prev.feats != cur.feats, axis=1).mean()
        assert 0.03 < changed < 0.2                             # about one 36 degree wedge


def test_bf16_stream_bits():
    strides = S.make_stream("c4", n_strides=2)
    for s in strides:
        assert s.feats.dtype == np.uint16
        f = S.bf16_bits_to_f32(s.feats)
        assert np.all(np.isfinite(f)) and not np.any(s.feats == 0x8000)   # no -0.0
    w = S.weights("c4")
    for wl in w:
        np.testing.assert_array_equal(S.bf16_bits_to_f32(S.round_to_bf16_bits(wl)).reshape(wl.shape), wl)


def test_weights_shapes_and_family():
    w2, w3 = S.weights("c2"), S.weights("c3")
    assert len(w2) == 4 and len(w3) == 16
    for a, b in zip(w2, w3):
        np.testing.assert_array_equal(a, b)
    assert w3[-1].shape == (256, 256, 3, 3)


def _changed_count(prev, cur):
    """Cells whose pillar appeared, vanished or carries a different vector."""
    a = dict(zip(prev.idx.tolist(), range(len(prev.idx))))
    n = len(set(prev.idx.tolist()) ^ set(cur.idx.tolist()))
    for i, p in enumerate(cur.idx.tolist()):
        j = a.get(p)
        if j is not None and not np.array_equal(prev.feats[j], cur.feats[i]):
            n += 1
    return n


def test_drone_scan_stream_has_the_paper_sparsity():
    """Sweep stream on 504 x 504: the paper reports 1,781 active and 483
    changed cells per 10 ms stride on average (27 % of active), with active
    between 1,552 and 2,533 and changed between 169 and 1,154."""
    st = S.make_stream("l64x64")
    assert len(st) == 101
    act = np.array([len(s.idx) for s in st[1:]])
    chg = np.array([_changed_count(a, b) for a, b in zip(st, st[1:])])
    assert 1600 < act.mean() < 2050 and act.min() > 1000 and act.max() < 2700
    assert 420 < chg.mean() < 550 and chg.min() > 150 and chg.max() < 1200
    assert 0.22 < (chg / act).mean() < 0.32
    for s in st:
        assert np.all(np.diff(s.idx) > 0) and np.all(np.any(s.feats != 0.0, axis=1))


def test_sweep_streams_share_cells_and_differ_in_width():
    a = S.make_stream("l16x8", n_strides=5)
    b = S.make_stream("l128x64", n_strides=5)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x.idx, y.idx)
        assert x.feats.shape[1] == 16 and y.feats.shape[1] == 128
    assert len(S.SWEEP_CIN) * len(S.SWEEP_COUT) == 20
    w = S.weights("l32x8")
    assert len(w) == 1 and w[0].shape == (8, 32, 3, 3)
    assert not np.array_equal(S.weights("l32x16")[0][:8], w[0])


def test_point_stream_bins_to_the_paper_sparsity():
    """Points of the drone scan binned into 0.16 m pillars: ~1,800 occupied and
    ~480 event-changed pillars per 10 ms stride over 100 ms windows, far below
    N = 100 points per pillar; the stream is deterministic."""
    from oracle import pfn as P
    sp, wl = S.pfn_spec("p2"), S.workload("p2")
    b = S.make_point_stream("p2", n_strides=40)
    assert len(b) == 40 + sp.window
    again = S.make_point_stream("p2", n_strides=40)
    for x, y in zip(b, again):
        np.testing.assert_array_equal(x, y)
        assert x.dtype == np.float32 and x.shape[1] == 4 and len(x) <= sp.max_new_points
    act, chg = [], []
    for k in range(sp.window, len(b)):
        occ, cnt = P.occupancy(b[k - sp.window + 1:k + 1], wl.H, wl.W, sp.x_min, sp.y_min, sp.res)
        act.append(len(occ))
        assert cnt.max() < sp.max_points
        chg.append(len(P.changed_cells(b[k], b[k - sp.window], wl.H, wl.W, sp.x_min, sp.y_min, sp.res)))
    assert 1400 < np.mean(act) < 2200 and 380 < np.mean(chg) < 600
