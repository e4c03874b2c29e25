"""Pins of the pillar feature net oracle (Sec. III-B; Alg. 1, PFN part)
against worked values, a library reference and properties that hold by
definition, none of which reuse the oracle's own formulas."""
import numpy as np
import pytest

from oracle import pfn as P

torch = pytest.importorskip("torch")


def test_worked_example_two_points_identity_weights():
    """Grid corner (0, 0), 1 m pillars, W = I (C0 = 9): two points in the pillar
    of row 1, column 2 (centre (2.5, 1.5)); mean (2.3, 1.55, 0.5).  The feature
    is the channelwise max of ReLU(decoration) over the two points."""
    pts = np.array([[2.1, 1.2, 0.0, 0.5],
                    [2.5, 1.9, 1.0, 0.25]], dtype=np.float32)
    cells = P.bin_points(pts, 4, 4, 0.0, 0.0, 1.0)
    assert list(cells) == [1 * 4 + 2, 1 * 4 + 2]
    f = P.pillar_feature(pts, 6, 4, 0.0, 0.0, 1.0, np.eye(9))
    # point 1: x y z r = 2.1 1.2 0 0.5; x_p y_p = -0.4 -0.3; x_c y_c z_c = -0.2 -0.35 -0.5
    # point 2: 2.5 1.9 1 0.25; x_p y_p = 0 0.4; x_c y_c z_c = 0.2 0.35 0.5
    want = [2.5, 1.9, 1.0, 0.5, 0.0, 0.4, 0.2, 0.35, 0.5]
    np.testing.assert_allclose(f, want, rtol=0, atol=1e-6)


def test_linear_relu_max_matches_torch():
    rng = np.random.default_rng(7)
    pts = rng.standard_normal((37, 4)).astype(np.float32) * 0.05
    pts[:, 0] += 3.3
    pts[:, 1] += -1.7
    w = rng.standard_normal((64, 9)).astype(np.float32)
    cell = int(P.bin_points(pts[:1], 8, 8, -4.0, -4.0, 1.0)[0])
    got = P.pillar_feature(pts, cell, 8, -4.0, -4.0, 1.0, w)
    dec = torch.from_numpy(P.decorate(pts, cell, 8, -4.0, -4.0, 1.0))
    lin = torch.nn.Linear(9, 64, bias=False).double()
    with torch.no_grad():
        lin.weight.copy_(torch.from_numpy(w.astype(np.float64)))
        ref = torch.relu(lin(dec)).max(dim=0).values.numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_cluster_offsets_sum_to_zero_and_centre_offsets_bounded():
    rng = np.random.default_rng(3)
    pts = np.column_stack([rng.uniform(1.0, 1.16, 50), rng.uniform(2.0, 2.16, 50),
                           rng.standard_normal(50), rng.random(50)]).astype(np.float32)
    cells = P.bin_points(pts, 32, 32, 0.0, 0.0, 0.16)
    c = int(cells[0])
    sel = pts[cells == c]
    d = P.decorate(sel, c, 32, 0.0, 0.0, 0.16)
    np.testing.assert_allclose(d[:, 6:9].sum(axis=0), 0.0, atol=1e-9)
    assert np.all(np.abs(d[:, 4:6]) <= 0.08 + 1e-6)


def test_binning_edges_in_float32():
    """Exactly representable edges with 0.25 m pillars from corner (-2, -2) on
    a 16 x 16 grid: the corner is column 0, just below it is outside, the far
    edge is outside, NaN is outside, cell boundaries go to the upper cell."""
    pts = np.array([[-2.0, -2.0, 0, 0],       # cell (0, 0)
                    [-2.0000002, 0.0, 0, 0],   # x below the corner
                    [2.0, 0.0, 0, 0],          # x at the far edge
                    [1.75, 1.9, 0, 0],         # last row, last column
                    [0.25, -1.5, 0, 0],        # boundary: column 9, row 2
                    [np.nan, 0.0, 0, 0]], dtype=np.float32)
    got = P.bin_points(pts, 16, 16, -2.0, -2.0, 0.25)
    assert list(got) == [0, -1, -1, 15 * 16 + 15, 2 * 16 + 9, -1]


def test_canvas_ignores_point_order_and_batch_split():
    rng = np.random.default_rng(11)
    pts = np.column_stack([rng.uniform(-1, 1, 300), rng.uniform(-1, 1, 300), rng.standard_normal(300),
                           rng.random(300)]).astype(np.float32)
    w = rng.standard_normal((16, 9)).astype(np.float32)
    a = P.canvas([pts], 12, 12, -1.0, -1.0, 2.0 / 12, w)
    perm = pts[rng.permutation(300)]
    b = P.canvas([perm[:100], perm[100:250], perm[250:]], 12, 12, -1.0, -1.0, 2.0 / 12, w)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    assert np.all(a >= 0.0)
    occ, _ = P.occupancy([pts], 12, 12, -1.0, -1.0, 2.0 / 12)
    empty = np.setdiff1d(np.arange(144), occ)
    assert np.all(a.reshape(144, 16)[empty] == 0.0)


def test_event_change_map_equals_brute_force_multiset_difference():
    """Window of 3 strides: a pillar is changed exactly when the multiset of
    its points differs between consecutive windows."""
    rng = np.random.default_rng(5)
    H = W = 10
    batches = [np.column_stack([rng.uniform(0, 1, 40), rng.uniform(0, 1, 40), rng.standard_normal(40),
                                rng.random(40)]).astype(np.float32) for _ in range(8)]
    batches.append(np.zeros((0, 4), np.float32))          # a stride without points
    win = 3

    def cell_sets(k):
        out = {}
        for b in batches[max(0, k - win + 1):k + 1]:
            for p, c in zip(b, P.bin_points(b, H, W, 0.0, 0.0, 0.1)):
                if c >= 0:
                    out.setdefault(int(c), []).append(tuple(p.tolist()))
        return {c: sorted(v) for c, v in out.items()}

    for k in range(1, len(batches)):
        old = batches[k - win] if k - win >= 0 else None
        got = P.changed_cells(batches[k], old, H, W, 0.0, 0.0, 0.1)
        a, b = cell_sets(k - 1), cell_sets(k)
        want = sorted(c for c in set(a) | set(b) if a.get(c) != b.get(c))
        assert list(got) == want, k
