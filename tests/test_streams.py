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
