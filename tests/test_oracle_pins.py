"""Pins of the CPU oracle against facts fixed independently of it.

Each test ties one part of the oracle to something other than its own code:
brute force, a library routine computing the same special case, a closed form,
a hand-derived table in tests/golden, or an invariant the paper states.
"""
import itertools
import os

import numpy as np
import pytest

import oracle
from oracle.method_model import DeltaScatterModel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_conv(x, w, s):
    """Seven nested loops straight from the definition (cross-correlation,
    zero padding 1): Z[y,x,co] = sum_{m,n,ci} X[s*y+m-1, s*x+n-1, ci] W[co,ci,m,n]."""
    H, W, cin = x.shape
    cout = w.shape[0]
    Ho, Wo = (H - 1) // s + 1, (W - 1) // s + 1
    z = np.zeros((Ho, Wo, cout))
    for yy in range(Ho):
        for xx in range(Wo):
            for co in range(cout):
                acc = 0.0
                for m in range(3):
                    for n in range(3):
                        for ci in range(cin):
                            iy, ix = s * yy + m - 1, s * xx + n - 1
                            if 0 <= iy < H and 0 <= ix < W:
                                acc += float(x[iy, ix, ci]) * float(w[co, ci, m, n])
                z[yy, xx, co] = acc
    return z


# -------------------------------------------------------------------- P-a
@pytest.mark.parametrize("H,W", [(5, 7), (8, 8), (9, 11), (1, 1), (2, 3)])
@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("cin,cout", [(1, 1), (3, 3), (3, 2)])
def test_conv_matches_brute_force(H, W, s, cin, cout):
    rng = np.random.default_rng(H * 100 + W * 10 + s + cin)
    x = rng.standard_normal((H, W, cin))
    x[rng.random((H, W)) < 0.3] = 0.0          # some empty cells
    w = rng.standard_normal((cout, cin, 3, 3))
    ref = brute_conv(x, w, s)
    got = oracle.conv3x3(x, w, s)
    assert got.shape == ref.shape
    scale = max(np.abs(ref).max(), 1e-300)
    assert np.abs(got - ref).max() <= 1e-12 * scale


# -------------------------------------------------------------------- P-b
@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("H,W,cin,cout", [(16, 13, 8, 5), (31, 20, 16, 16), (7, 9, 64, 8)])
def test_conv_matches_torch(s, H, W, cin, cout):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7 + H + s)
    x = rng.standard_normal((H, W, cin))
    w = rng.standard_normal((cout, cin, 3, 3))
    ref = torch.nn.functional.conv2d(torch.from_numpy(x).permute(2, 0, 1)[None], torch.from_numpy(w),
                                     stride=s, padding=1)[0].permute(1, 2, 0).numpy()
    got = oracle.conv3x3(x, w, s)
    assert got.shape == ref.shape
    assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()


def test_forward_chain_matches_torch_with_relu_and_bf16():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    layers = [(4, 8, 2, True), (8, 8, 1, True), (8, 6, 1, False)]
    ws = [rng.standard_normal((co, ci, 3, 3)) * 0.3 for (ci, co, _, _) in layers]
    x = rng.standard_normal((13, 10, 4))
    for bf16 in (False, True):
        ys = oracle.forward(x, ws, layers, bf16_storage=bf16)
        t = torch.from_numpy(x).permute(2, 0, 1)[None]
        for l, (ci, co, s, relu) in enumerate(layers):
            t = torch.nn.functional.conv2d(t, torch.from_numpy(ws[l]), stride=s, padding=1)
            if relu:
                t = torch.relu(t)
            if bf16:
                t = t.to(torch.float32).to(torch.bfloat16).to(torch.float64)
            ref = t[0].permute(1, 2, 0).numpy()
            if bf16:
                # identical rounding decisions except where fp64 summation order
                # differs across a bf16 rounding boundary
                bad = np.abs(ys[l] - ref) > 1e-12 * np.abs(ref).max()
                assert bad.mean() < 0.01
            else:
                assert np.abs(ys[l] - ref).max() <= 1e-12 * np.abs(ref).max()
            t = torch.from_numpy(ys[l]).permute(2, 0, 1)[None]   # continue from the oracle's own maps


def test_round_bf16_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [0.0, 1.0, -1.0, 1.00390625, 1.005859375, 3.0e38, -2.5e-30]])
    ref = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.round_bf16(x)
    np.testing.assert_array_equal(got, ref)


# -------------------------------------------------------------------- P-c
@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("i,j", [(4, 5), (5, 4), (5, 5), (4, 4)])
def test_impulse_gives_flipped_stencil(s, i, j):
    H, W, cin, cout, ci = 11, 12, 3, 4, 1
    rng = np.random.default_rng(5)
    w = rng.standard_normal((cout, cin, 3, 3))
    x = np.zeros((H, W, cin))
    x[i, j, ci] = 1.0
    z = oracle.conv3x3(x, w, s)
    Ho, Wo = z.shape[:2]
    expect = np.zeros_like(z)
    for m in range(3):
        for n in range(3):
            if (i - m + 1) % s or (j - n + 1) % s:
                continue
            r, c = (i - m + 1) // s, (j - n + 1) // s
            if 0 <= r < Ho and 0 <= c < Wo:
                expect[r, c, :] = w[:, ci, m, n]
    np.testing.assert_array_equal(z, expect)
    # which taps contribute at stride 2: m = 1 for even i, m in {0, 2} for odd i
    if s == 2:
        rows = set(np.flatnonzero(np.any(z != 0, axis=(1, 2))))
        assert rows == ({i // 2} if i % 2 == 0 else {(i - 1) // 2, (i + 1) // 2})


# ---------------------------------------------------------- footprint table
def _footprint_table():
    rows = []
    with open(os.path.join(GOLDEN, "footprints.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split(":")
            s, n, i = map(int, lhs.split())
            rows.append((s, n, i, sorted(map(int, rhs.split()))))
    return rows


@pytest.mark.parametrize("s,n,i,outs", _footprint_table())
def test_gather_rule_matches_footprint_table(s, n, i, outs):
    mask = np.zeros((1, n), dtype=bool)
    mask[0, i] = True
    got = np.flatnonzero(oracle.propagate_gather(mask, s)[0])
    assert got.tolist() == outs
    mask = np.zeros((n, 1), dtype=bool)
    mask[i, 0] = True
    assert np.flatnonzero(oracle.propagate_gather(mask, s)[:, 0]).tolist() == outs


@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("H,W", [(7, 9), (8, 8), (6, 11)])
def test_gather_rule_equals_dependency_of_dense_conv(s, H, W):
    """Perturbing one input cell changes exactly the outputs the gather rule
    lists (generic weights, no activation): the lists describe the true
    dependency structure of the convolution."""
    rng = np.random.default_rng(H * W + s)
    w = rng.standard_normal((3, 2, 3, 3))
    x = rng.standard_normal((H, W, 2))
    z0 = oracle.conv3x3(x, w, s)
    for (i, j) in itertools.product(range(H), range(W)):
        x1 = x.copy()
        x1[i, j] += rng.standard_normal(2)
        diff = np.any(oracle.conv3x3(x1, w, s) != z0, axis=-1)
        mask = np.zeros((H, W), dtype=bool)
        mask[i, j] = True
        np.testing.assert_array_equal(oracle.propagate_gather(mask, s), diff)


# -------------------------------------------------------------------- P-d
def test_dilation_counts():
    table = {}
    with open(os.path.join(GOLDEN, "impulse_counts.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                case, l, c = line.split()
                table[(case, int(l))] = int(c)
    H = W = 21
    cells = {"interior": (10, 10), "corner": (0, 0), "edge": (0, 7)}
    for (case, l), count in table.items():
        prev = np.zeros((H, W, 1), dtype=np.uint32)
        new = prev.copy()
        new[cells[case]] = 1
        lists = oracle.changed_lists(prev, new, [1] * l)
        assert len(lists[0]) == 1
        assert len(lists[l]) == count
        if case == "interior":
            for k in range(1, l + 1):
                assert len(lists[k]) == (2 * k + 1) ** 2


# -------------------------------------------------------------------- P-e
def test_linearity_of_delta_scatter():
    """Eq. 2's fused form rests on conv(X_new) - conv(X_old) = conv(X_new - X_old)."""
    rng = np.random.default_rng(21)
    w = rng.standard_normal((16, 16, 3, 3)) / 12
    a = rng.standard_normal((64, 64, 16))
    b = a.copy()
    sel = rng.random((64, 64)) < 0.05
    b[sel] = rng.standard_normal((int(sel.sum()), 16))
    for s in (1, 2):
        lhs = oracle.conv3x3(b, w, s) - oracle.conv3x3(a, w, s)
        rhs = oracle.conv3x3(b - a, w, s)
        assert np.abs(lhs - rhs).max() <= 1e-12 * np.abs(oracle.conv3x3(b, w, s)).max()


# ------------------------------------------------------------ P-f, P-g, P-h
def _toy_stream(H, W, C0, n, seed, toggles=True, refresh=0.05):
    rng = np.random.default_rng(seed)
    occ = rng.random((H, W)) < 0.15
    x = np.zeros((H, W, C0), dtype=np.float32)
    x[occ] = rng.standard_normal((int(occ.sum()), C0)).astype(np.float32)
    out = [x.copy()]
    for _ in range(n):
        r = (rng.random((H, W)) < refresh) & occ
        x[r] = rng.standard_normal((int(r.sum()), C0)).astype(np.float32)
        if toggles:
            t = rng.random((H, W)) < 0.01
            off = t & occ
            on = t & ~occ
            x[off] = 0.0
            x[on] = rng.standard_normal((int(on.sum()), C0)).astype(np.float32)
            occ = (occ & ~off) | on
        out.append(x.copy())
    return out


@pytest.mark.parametrize("layers", [
    [(4, 4, 1, False)],
    [(4, 6, 2, True), (6, 6, 1, True), (6, 5, 1, True)],
    [(4, 5, 1, True), (5, 5, 2, True), (5, 4, 2, False)],
])
def test_method_model_equals_recompute(layers):
    """The recycling claim (abstract; Sec. IV-G): after many delta strides with
    refreshes and toggles, the recycled maps equal recomputation."""
    H, W, C0 = 13, 11, 4
    rng = np.random.default_rng(99)
    ws = [rng.standard_normal((co, ci, 3, 3)) * 0.4 for (ci, co, _, _) in layers]
    model = DeltaScatterModel(H, W, C0, layers, ws)
    frames = _toy_stream(H, W, C0, 50, 5)
    prev_bits = np.zeros((H, W, C0), dtype=np.uint32)
    for x in frames:
        bits = x.view(np.uint32)
        lists = model.step(x.astype(np.float64), bits)
        ref_lists = oracle.changed_lists(prev_bits, bits, [l[2] for l in layers])
        for a, b in zip(lists, ref_lists):
            np.testing.assert_array_equal(a, b)
        prev_bits = bits.copy()
    ys = oracle.forward(frames[-1].astype(np.float64), ws, layers)
    for got, ref in zip(model.maps(), ys):
        assert np.abs(got - ref).max() <= 1e-10 * max(np.abs(ref).max(), 1e-300)


def test_method_model_equals_recompute_bf16_storage():
    layers = [(4, 6, 2, True), (6, 6, 1, True)]
    H, W, C0 = 12, 12, 4
    rng = np.random.default_rng(4)
    ws = [oracle.round_bf16(rng.standard_normal((co, ci, 3, 3)) * 0.4) for (ci, co, _, _) in layers]
    model = DeltaScatterModel(H, W, C0, layers, ws, bf16_storage=True)
    frames = [oracle.round_bf16(f.astype(np.float64)).astype(np.float32) for f in _toy_stream(H, W, C0, 30, 8)]
    for x in frames:
        model.step(x.astype(np.float64), x.view(np.uint32))
    ys = oracle.forward(frames[-1].astype(np.float64), ws, layers, bf16_storage=True)
    for got, ref in zip(model.maps(), ys):
        # same rounding decisions up to the float64 summation-order residue
        assert np.abs(got - ref).max() <= 1e-2 * np.abs(ref).max()
        assert (np.abs(got - ref) > 1e-9 * np.abs(ref).max()).mean() < 0.02


def test_locality_value_changes_lie_in_structural_sets():
    """V_l (cells whose value changed) is a subset of A_l; without ReLU and with
    generic data the two coincide for the first layer."""
    layers = [(4, 4, 1, False), (4, 4, 2, True), (4, 4, 1, True)]
    H, W, C0 = 16, 15, 4
    rng = np.random.default_rng(8)
    ws = [rng.standard_normal((co, ci, 3, 3)) for (ci, co, _, _) in layers]
    frames = _toy_stream(H, W, C0, 12, 17)
    prev = None
    for x in frames:
        ys = oracle.forward(x.astype(np.float64), ws, layers)
        if prev is not None:
            px, pys = prev
            lists = oracle.changed_lists(px.view(np.uint32), x.view(np.uint32), [l[2] for l in layers])
            for l in range(len(layers)):
                v = oracle.value_changed(pys[l], ys[l])
                assert set(v.tolist()) <= set(lists[l + 1].tolist())
            np.testing.assert_array_equal(oracle.value_changed(pys[0], ys[0]), lists[1])
        prev = (x, ys)


def test_zero_change_stride_does_no_work():
    layers = [(4, 6, 2, True), (6, 6, 1, True)]
    H, W, C0 = 10, 9, 4
    rng = np.random.default_rng(2)
    ws = [rng.standard_normal((co, ci, 3, 3)) for (ci, co, _, _) in layers]
    model = DeltaScatterModel(H, W, C0, layers, ws)
    x = _toy_stream(H, W, C0, 0, 3)[0]
    model.step(x.astype(np.float64), x.view(np.uint32))
    before = [m.copy() for m in model.maps()]
    lists = model.step(x.astype(np.float64), x.view(np.uint32))
    assert all(len(a) == 0 for a in lists)
    for a, b in zip(before, model.maps()):
        np.testing.assert_array_equal(a, b)
    ref = oracle.changed_lists(x.view(np.uint32), x.view(np.uint32), [2, 1])
    assert all(len(a) == 0 for a in ref)


def test_full_pass_lists_are_nonzero_cells():
    """The first window after a cold start changes exactly the non-empty cells."""
    x = _toy_stream(9, 9, 3, 0, 12)[0]
    lists = oracle.changed_lists(np.zeros_like(x.view(np.uint32)), x.view(np.uint32), [1])
    np.testing.assert_array_equal(lists[0], np.flatnonzero(np.any(x != 0, axis=-1)))


@pytest.mark.parametrize("s", [1, 2])
def test_pair_counts_equal_sum_of_single_cell_footprints(s):
    """Pairs counted in the gather direction equal the sum over changed cells of
    their individual footprints (each pinned above by the dependency test)."""
    rng = np.random.default_rng(30 + s)
    for H, W in [(7, 9), (8, 8), (5, 12)]:
        mask = rng.random((H, W)) < 0.3
        expect = 0
        for p in np.flatnonzero(mask):
            single = np.zeros((H, W), dtype=bool)
            single.flat[p] = True
            expect += int(oracle.propagate_gather(single, s).sum())
        assert oracle.pair_counts(mask, s) == expect


# ------------------------------------------------------------ neck (upsampling + concat)
@pytest.mark.parametrize("s", [1, 2, 4])
def test_conv_transpose_matches_torch(s):
    """Library special case: torch's ConvTranspose2d (kernel = stride, no
    padding) in float64."""
    import torch
    rng = np.random.default_rng(10 + s)
    x = rng.standard_normal((5, 6, 3))
    w = rng.standard_normal((3, 4, s, s))
    got = oracle.conv_transpose(x, w, s)
    ref = torch.nn.functional.conv_transpose2d(torch.from_numpy(x).permute(2, 0, 1)[None], torch.from_numpy(w),
                                               stride=s)[0].permute(1, 2, 0).numpy()
    assert got.shape == (5 * s, 6 * s, 4)
    assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()


def test_conv_transpose_brute_force():
    """Every output cell is one input cell's row times one kernel position."""
    rng = np.random.default_rng(3)
    s, H, W, cin, cout = 2, 3, 2, 2, 3
    x = rng.standard_normal((H, W, cin))
    w = rng.standard_normal((cin, cout, s, s))
    ref = np.zeros((H * s, W * s, cout))
    for i in range(H):
        for j in range(W):
            for a in range(s):
                for b in range(s):
                    for co in range(cout):
                        for ci in range(cin):
                            ref[s * i + a, s * j + b, co] += x[i, j, ci] * w[ci, co, a, b]
    assert np.abs(oracle.conv_transpose(x, w, s) - ref).max() <= 1e-13


@pytest.mark.parametrize("s", [1, 2, 4])
def test_upsample_rule_is_the_dependency_of_conv_transpose(s):
    """Alg. 1, deconvolution branch: perturbing one input cell changes exactly
    the upsampled sites under it, which upsample_mask names."""
    rng = np.random.default_rng(20 + s)
    H, W = 4, 5
    x = rng.standard_normal((H, W, 2))
    w = rng.standard_normal((2, 3, s, s))
    base = oracle.conv_transpose(x, w, s)
    for (i, j) in [(0, 0), (2, 3), (3, 4)]:
        y = x.copy()
        y[i, j] += 1.0
        diff = np.any(oracle.conv_transpose(y, w, s) != base, axis=-1)
        m = np.zeros((H, W), dtype=bool)
        m[i, j] = True
        np.testing.assert_array_equal(diff, oracle.upsample_mask(m, s))
        assert diff.sum() == s * s


def test_neck_concat_and_union():
    """The neck output is the channel concatenation of the upsampled maps in
    order, and its change set is the union of the upsampled sets."""
    rng = np.random.default_rng(7)
    # sources on 8x4, 4x2 and 2x1 grids, all upsampled to 8x4
    ys = [rng.standard_normal((8, 4, 2)), rng.standard_normal((4, 2, 3)), rng.standard_normal((2, 1, 4))]
    ups = [(1, 2, 1, True), (2, 3, 2, False), (3, 1, 4, True)]
    ws = [rng.standard_normal((2, 2, 1, 1)), rng.standard_normal((3, 3, 2, 2)), rng.standard_normal((4, 1, 4, 4))]
    out = oracle.forward_neck(ys, ws, ups)
    assert out.shape == (8, 4, 6)
    np.testing.assert_array_equal(out[..., :2], np.maximum(oracle.conv_transpose(ys[0], ws[0], 1), 0))
    np.testing.assert_array_equal(out[..., 2:5], oracle.conv_transpose(ys[1], ws[1], 2))
    np.testing.assert_array_equal(out[..., 5:], np.maximum(oracle.conv_transpose(ys[2], ws[2], 4), 0))
    # A_1 = {0, 31} on 8x4, A_2 = {5} on 4x2 (cell (2, 1)), A_3 = {1} on 2x1 (cell (1, 0))
    lists = [np.zeros(0, np.int64), np.array([0, 31]), np.array([5]), np.array([1])]
    got = oracle.neck_changed(lists, [(8, 4), (4, 2), (2, 1)], ups)
    want = {0, 31}
    want |= {(2 * 2 + a) * 4 + (2 * 1 + b) for a in range(2) for b in range(2)}
    want |= {(4 * 1 + a) * 4 + b for a in range(4) for b in range(4)}
    np.testing.assert_array_equal(got, np.array(sorted(want)))


def test_neck_recycling_equals_recompute():
    """The delta form for the neck: Z_up(new) = Z_up(old) + convT(Y_src(new) -
    Y_src(old)), with the source delta nonzero only on the source's change set,
    so updating the upsampled blocks of the changed cells reproduces the
    recomputed map."""
    rng = np.random.default_rng(11)
    w = rng.standard_normal((3, 2, 2, 2))
    y_old = rng.standard_normal((5, 4, 3))
    y_new = y_old.copy()
    changed = [(0, 1), (3, 3), (4, 0)]
    for (i, j) in changed:
        y_new[i, j] = rng.standard_normal(3)
    z = oracle.conv_transpose(y_old, w, 2)
    d = oracle.conv_transpose(y_new - y_old, w, 2)
    m = np.zeros((5, 4), dtype=bool)
    for (i, j) in changed:
        m[i, j] = True
    up = oracle.upsample_mask(m, 2)
    assert not np.any(d[~up])                 # no change outside the upsampled set
    z[up] += d[up]
    ref = oracle.conv_transpose(y_new, w, 2)
    assert np.abs(z - ref).max() <= 1e-12 * np.abs(ref).max()


def test_delta_form_model_pair_equals_recompute_and_rounding_drifts():
    """The delta-form model: with the exact pair delta and float64 maps it
    follows recomputation with bf16 storage (the same rounding decisions up
    to float64 summation order, as for the loop model); rounding the delta to
    bf16 before the scatter makes the recycled maps leave recomputation."""
    from oracle.method_model import DeltaFormModel
    layers = [(4, 6, 2, True), (6, 6, 1, True), (6, 4, 1, True)]
    H, W, C0 = 14, 12, 4
    rng = np.random.default_rng(21)
    ws = [oracle.round_bf16(rng.standard_normal((co, ci, 3, 3)) * 0.4) for (ci, co, _, _) in layers]
    frames = [oracle.round_bf16(f.astype(np.float64)) for f in _toy_stream(H, W, C0, 40, 8)]
    exact = DeltaFormModel(layers, ws, delta="pair", z32=False)
    rounded = DeltaFormModel(layers, ws, delta="rounded", z32=False)
    worst_rounded = 0.0
    for x in frames:
        ys_e, ys_r = exact.step(x), rounded.step(x)
        ref = oracle.forward(x, ws, layers, bf16_storage=True)
        for got, r in zip(ys_e, ref):
            assert np.abs(got - r).max() <= 1e-2 * np.abs(r).max()
            assert (np.abs(got - r) > 1e-9 * np.abs(r).max()).mean() < 0.02
        worst_rounded = max(worst_rounded, max(np.abs(g - r).max() / np.abs(r).max() for g, r in zip(ys_r, ref)))
    assert worst_rounded > 1e-3
