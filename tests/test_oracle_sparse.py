"""Pins of the sparse-backbone oracle (regular sparse and submanifold
convolutions) against brute force written from the operators' definitions,
the dense special case and invariants."""
import numpy as np
import pytest

import oracle
from oracle import sparse as SP


def _brute(x, occ, ws, layers, sub):
    """Direct loops: active sets from their definitions, outputs at active
    sites only, zeros elsewhere."""
    y, s_in = x.astype(np.float64), occ.astype(bool)
    outs = []
    for (ci, co, st, relu), w, is_sub in zip(layers, ws, sub):
        H, W = s_in.shape
        Ho, Wo = (H - 1) // st + 1, (W - 1) // st + 1
        s_out = np.zeros((Ho, Wo), bool)
        z = np.zeros((Ho, Wo, co))
        for r in range(Ho):
            for c in range(Wo):
                any_in = False
                for m in range(3):
                    for n in range(3):
                        i, j = st * r + m - 1, st * c + n - 1
                        if 0 <= i < H and 0 <= j < W:
                            any_in = any_in or s_in[i, j]
                            z[r, c] += w[:, :, m, n] @ y[i, j]
                s_out[r, c] = s_in[r, c] if is_sub else any_in
        yo = np.maximum(z, 0) if relu else z
        yo[~s_out] = 0.0
        outs.append(yo)
        y, s_in = yo, s_out
    return outs


def _case(rng, H, W, C, layers, p_occ):
    occ = rng.random((H, W)) < p_occ
    x = np.where(occ[..., None], rng.standard_normal((H, W, C)), 0.0)
    ws = [rng.standard_normal((co, ci, 3, 3)) * 0.3 for (ci, co, _s, _r) in layers]
    return x, occ, ws


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    layers = [(3, 4, 2, True), (4, 4, 1, True), (4, 5, 1, False), (5, 3, 2, True), (3, 3, 1, True)]
    sub = [False, True, True, False, True]
    x, occ, ws = _case(rng, 11, 9, 3, layers, 0.15)
    got = SP.forward(x, occ, ws, layers, sub)
    want = _brute(x, occ, ws, layers, sub)
    for g, w_ in zip(got, want):
        np.testing.assert_allclose(g, w_, rtol=1e-12, atol=1e-12)


def test_all_active_equals_the_dense_backbone():
    rng = np.random.default_rng(4)
    layers = [(4, 4, 1, True), (4, 4, 1, True), (4, 6, 2, True), (6, 6, 1, False)]
    x, _occ, ws = _case(rng, 8, 10, 4, layers, 1.0)
    occ = np.ones((8, 10), bool)
    got = SP.forward(x, occ, ws, layers, [False, True, False, True])
    for g, d in zip(got, oracle.forward(x, ws, layers)):
        np.testing.assert_allclose(g, d, rtol=1e-12, atol=1e-12)


def test_worked_example_submanifold_keeps_empty_sites_empty():
    """One pillar at (2, 2) of a 5 x 5 grid, all-ones 1-channel weights, no
    ReLU: the regular layer's active set is the 3 x 3 block around it, whose
    sites all hold 1.  The submanifold layer sums 3 x 3 neighbourhoods only
    at those 9 sites (centre 9, edge midpoints 6, corners 4); the dense
    convolution would also give (0, 0) the value 1."""
    x = np.zeros((5, 5, 1))
    x[2, 2, 0] = 1.0
    occ = np.zeros((5, 5), bool)
    occ[2, 2] = True
    w = np.ones((1, 1, 3, 3))
    layers = [(1, 1, 1, False), (1, 1, 1, False)]
    y1, y2 = SP.forward(x, occ, [w, w], layers, [False, True])
    np.testing.assert_array_equal(y1[..., 0], np.pad(np.ones((3, 3)), 1))
    want = np.zeros((5, 5))
    want[1:4, 1:4] = [[4, 6, 4], [6, 9, 6], [4, 6, 4]]
    np.testing.assert_array_equal(y2[..., 0], want)
    assert oracle.forward(x, [w, w], layers)[1][0, 0, 0] == 1.0


def test_change_lists_cover_every_value_change_and_stay_in_the_active_sets():
    rng = np.random.default_rng(8)
    layers = [(3, 3, 2, True), (3, 3, 1, True), (3, 4, 1, True), (4, 4, 2, True), (4, 4, 1, True)]
    sub = [False, True, True, False, True]
    x, occ, ws = _case(rng, 16, 14, 3, layers, 0.2)
    x2, occ2 = x.copy(), occ.copy()
    flip = rng.random((16, 14)) < 0.05                 # pillars appear and vanish
    occ2 ^= flip
    x2[~occ2] = 0.0
    new = occ2 & (flip | (rng.random((16, 14)) < 0.1))
    x2[new] = rng.standard_normal((int(new.sum()), 3))
    lists = SP.changed_lists(oracle.canvas_bits(x.astype(np.float32), "f32"),
                             oracle.canvas_bits(x2.astype(np.float32), "f32"), occ, occ2, layers, sub)
    ya, yb = SP.forward(x, occ, ws, layers, sub), SP.forward(x2, occ2, ws, layers, sub)
    sa, sb = SP.active_sets(occ, layers, sub), SP.active_sets(occ2, layers, sub)
    for l in range(len(layers)):
        moved = np.flatnonzero(np.any(ya[l] != yb[l], axis=-1))
        assert np.all(np.isin(moved, lists[l + 1])), l
        assert np.all((sa[l] | sb[l]).reshape(-1)[lists[l + 1]]), l
    # A_0 holds the toggled pillars even when their features are all zero
    assert np.all(np.isin(np.flatnonzero(flip), lists[0]))


def test_submanifold_requires_stride_one():
    with pytest.raises(AssertionError):
        SP.active_sets(np.ones((4, 4), bool), [(1, 1, 2, True)], [True])


def _value_changed_lists(ys_a, ys_b, x_a, x_b):
    """Cells whose value differs between two windows, per layer (layer 0 the
    canvas): the value semantics the change sets must reproduce."""
    out = [np.flatnonzero(np.any(x_a != x_b, axis=-1))]
    for a, b in zip(ys_a, ys_b):
        out.append(np.flatnonzero(np.any(a != b, axis=-1)))
    return out


def _unmasked_variant(prev_bits, new_bits, prev_occ, new_occ, layers, sub):
    """A plausible misreading kept here only to show the pin rejects it: the
    receptive-field rule propagates the unmasked set, and only each layer's
    reported set is restricted to the active sites."""
    m = np.any(prev_bits != new_bits, axis=-1) | (prev_occ ^ new_occ)
    out = [np.flatnonzero(m)]
    s_old, s_new = SP.active_sets(prev_occ, layers, sub), SP.active_sets(new_occ, layers, sub)
    for (_ci, _co, stride, _r), so, sn in zip(layers, s_old, s_new):
        m = oracle.propagate_gather(m, stride)
        out.append(np.flatnonzero(m & (so | sn)))
    return out


def _lists_of(x_a, x_b, occ_a, occ_b, layers, sub, fn=SP.changed_lists):
    return fn(oracle.canvas_bits(x_a.astype(np.float32), "f32"), oracle.canvas_bits(x_b.astype(np.float32), "f32"),
              occ_a, occ_b, layers, sub)


def test_worked_example_change_sets_stop_at_inactive_sites():
    """Pillars at (2, 2) and (2, 6) of a 5 x 9 grid, one channel, all-ones
    weights, no ReLU; a regular stride-1 layer and two submanifold layers.
    The regular layer's active set is the two 3 x 3 blocks (columns 1-3 and
    5-7); column 4 is empty in both windows.  Refreshing the pillar at (2, 2)
    changes the 3 x 3 block around it in layer 1, and the submanifold layers
    cannot leave their active set, so layers 2 and 3 change exactly the same
    block: rows 1-3, columns 1-3.  Propagating through the empty column 4
    (reading the rule without the restriction) would also mark rows 1-3 of
    column 5 in layer 3, whose values do not move."""
    x = np.zeros((5, 9, 1))
    occ = np.zeros((5, 9), bool)
    for c in (2, 6):
        occ[2, c] = True
        x[2, c, 0] = 1.0
    x2 = x.copy()
    x2[2, 2, 0] = 2.0
    layers = [(1, 1, 1, False)] * 3
    sub = [False, True, True]
    block = sorted(r * 9 + c for r in (1, 2, 3) for c in (1, 2, 3))
    lists = _lists_of(x, x2, occ, occ, layers, sub)
    assert list(lists[0]) == [2 * 9 + 2]
    for l in (1, 2, 3):
        assert list(lists[l]) == block, l
    # the value semantics agree
    w = np.ones((1, 1, 3, 3))
    ya, yb = SP.forward(x, occ, [w] * 3, layers, sub), SP.forward(x2, occ, [w] * 3, layers, sub)
    for l, v in enumerate(_value_changed_lists(ya, yb, x, x2)):
        np.testing.assert_array_equal(v, lists[l])
    # the misreading does not
    bad = _lists_of(x, x2, occ, occ, layers, sub, _unmasked_variant)
    assert sorted(set(bad[3]) - set(block)) == [r * 9 + 5 for r in (1, 2, 3)]


_STACKS = [
    ([(3, 3, 1, False), (3, 3, 1, False), (3, 3, 1, False), (3, 4, 2, False), (4, 4, 1, False)],
     [False, True, True, False, True]),
    ([(2, 3, 2, False), (3, 3, 1, False), (3, 3, 1, False), (3, 2, 1, False)],
     [False, True, True, True]),
    ([(3, 3, 1, False), (3, 3, 1, False), (3, 3, 2, False), (3, 3, 1, False), (3, 3, 1, False)],
     [False, False, False, True, True]),
]


@pytest.mark.parametrize("case", range(len(_STACKS)))
def test_change_sets_equal_value_changes_without_relu(case):
    """The sparse analogue of the locality pin: with the identity activation,
    generic weights and generic (never zero) features, a site's value changes
    exactly when the change rule marks it, at every layer and stride, through
    refreshes and pillars that appear and vanish.  (ReLU or an all-zero
    pillar can only make the value set smaller.)  Small sparse grids put
    submanifold sites next to sites that are empty in both windows, where a
    wrong restriction of the rule shows."""
    layers, sub = _STACKS[case]
    rng = np.random.default_rng(100 + case)
    H, W, C = 13, 11, layers[0][0]
    ws = [rng.standard_normal((co, ci, 3, 3)) for (ci, co, _s, _r) in layers]
    occ = rng.random((H, W)) < 0.12
    x = np.where(occ[..., None], rng.uniform(0.5, 1.5, (H, W, C)) * rng.choice([-1.0, 1.0], (H, W, C)), 0.0)
    x = x.astype(np.float32).astype(np.float64)
    y = SP.forward(x, occ, ws, layers, sub)
    variant_differs = False
    for t in range(12):
        occ2 = occ ^ (rng.random((H, W)) < 0.03)
        x2 = np.where(occ2[..., None], x, 0.0)
        fresh = occ2 & ((rng.random((H, W)) < 0.08) | ~occ)
        x2[fresh] = rng.uniform(0.5, 1.5, (int(fresh.sum()), C)) * rng.choice([-1.0, 1.0], (int(fresh.sum()), C))
        x2 = x2.astype(np.float32).astype(np.float64)
        y2 = SP.forward(x2, occ2, ws, layers, sub)
        lists = _lists_of(x, x2, occ, occ2, layers, sub)
        vals = _value_changed_lists(y, y2, x, x2)
        for l in range(len(layers) + 1):
            np.testing.assert_array_equal(lists[l], vals[l], err_msg=f"stack {case} stride {t} layer {l}")
        bad = _lists_of(x, x2, occ, occ2, layers, sub, _unmasked_variant)
        variant_differs |= any(not np.array_equal(b, v) for b, v in zip(bad, vals))
        x, occ, y = x2, occ2, y2
    if case == 0:
        assert variant_differs, "the seeded strides must include a case the unrestricted rule gets wrong"
