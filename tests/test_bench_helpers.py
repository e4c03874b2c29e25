"""Host-side helpers of bench.py: the whole-stride roofline model and the
stacking of several streams' strides into one batched stride."""
import numpy as np
import pytest

import bench
import streams as S


def test_stride_roofline_single_layer_by_hand():
    wl = S.workload("c1")          # 64x64, one 16->16 stride-1 layer, fp32
    K = 2
    act = [2 * 50, 2 * 300]        # |A_0| = 50, |A_1| = 300 per stride
    pairs = [0, 2 * 400]           # 400 (changed input, in-grid tap) pairs per stride
    r = bench.stride_roofline(wl, act, pairs, K, mean_pillars=400.0, t_us=10.0, copy_gbs=4000.0)
    flops = 2.0 * 16 * 16 * 400
    b_a1 = 400 * (4 + 16 * 4) + 400 * 16 * 4 + 50 * 16 * 8 + 8 * 400
    b_1 = 50 * 16 * 4 + 300 * 16 * 8 + 9 * 16 * 16 * 4 + 8 * (50 + 300)   # last layer: no deltas out
    assert r["alg_flops"] == pytest.approx(flops)
    assert r["alg_bytes"] == pytest.approx(b_a1 + b_1)
    t_spec = b_a1 / 8e12 + max(flops / 157.3e12, b_1 / 8e12)
    t_copy = b_a1 / 4e12 + max(flops / 157.3e12, b_1 / 4e12)
    assert r["t_roof_us_spec"] == pytest.approx(t_spec * 1e6)
    assert r["t_roof_us_copy"] == pytest.approx(t_copy * 1e6)
    assert r["frac_spec"] == pytest.approx(t_spec * 1e6 / 10.0)


def test_stride_roofline_bf16_uses_bf16_peak_and_element_sizes():
    wl = S.workload("c4")
    L = len(wl.layers)
    act = [1000] * (L + 1)
    pairs = [0] + [9000] * L
    r = bench.stride_roofline(wl, act, pairs, 1, 12000.0, 100.0, 5000.0)
    # bf16: canvas and weights 2 bytes, deltas carried as the 4-byte pair
    sp = wl.layers[0]
    b1 = 1000 * sp.cin * 4 + 1000 * sp.cout * 8 + 1000 * sp.cout * 4 + 9 * sp.cin * sp.cout * 2 + 8 * 2000
    f1 = 2.0 * sp.cin * sp.cout * 9000
    assert r["alg_flops"] == pytest.approx(sum(2.0 * l.cin * l.cout * 9000 for l in wl.layers))
    assert r["t_roof_us_spec"] >= max(f1 / 2500e12, b1 / 8e12) * 1e6


def test_stack_strides_offsets_every_image():
    H, W = 5, 7
    a = S.Stride(3, np.array([0, 34], np.int32), np.ones((2, 4), np.float32))
    b = S.Stride(3, np.array([5], np.int32), 2 * np.ones((1, 4), np.float32))
    st = bench.stack_strides([a, b], H, W)
    np.testing.assert_array_equal(st.idx, [0, 34, 35 + 5])
    assert st.feats.shape == (3, 4) and st.feats[2, 0] == 2.0 and st.idx.dtype == np.int32


def test_kernel_names_of_the_two_launch_layers():
    """c3: the 128- and 256-channel stride-1 layers after the first run as a
    contraction launch plus a tap sum; every other layer keeps one launch."""
    wl = S.workload("c3")
    L = len(wl.layers)
    names = [bench.kernel_name(1 + l, wl) for l in range(1, L + 1)]
    assert names[0] == "layer_kernel<64,64,2,f32>"
    assert names[4] == "layer_kernel<64,128,2,f32>"
    assert names[5:10] == ["tap_sum_kernel<128,f32>"] * 5
    assert names[10] == "layer_kernel_wide<128,256,2,f32>"
    assert names[11:] == ["tap_sum_kernel<256,f32>"] * 5
    split = [l for l in range(1, L + 1) if bench.layer_split(l, wl)]
    assert split == list(range(6, 11)) + list(range(12, 17))
    assert bench.kernel_name(L + 1 + 12, wl) == "contract_kernel<256,256,f32>"
    assert bench.launches_per_stride("contract_kernel<256,256,f32>", wl) == 5
    assert bench.launches_per_stride("tap_sum_kernel<128,f32>", wl) == 5
    assert bench.launches_per_stride("layer_kernel<64,64,1,f32>", wl) == 3
    assert not any(bench.layer_split(l, S.workload("c2")) for l in range(1, 5))


def test_block_times_split_at_stride_two_layers():
    wl = S.workload("c3")
    L = len(wl.layers)
    K = 2
    ms = [0.0] * (2 * L + 2)
    ms[0], ms[1] = 0.010, 0.004                       # detection, ms over K strides
    for l in range(1, L + 1):
        ms[1 + l] = 0.001 * l                         # layer (or tap sum) l
        if bench.layer_split(l, wl):
            ms[L + 1 + l] = 0.002                     # its contraction launch
    b = bench.block_times(wl, ms, K)
    assert b["detect"] == pytest.approx(7.0)
    assert b["block 1"] == pytest.approx(sum(0.001 * l for l in range(1, 5)) / K * 1e3)
    assert b["block 2"] == pytest.approx((sum(0.001 * l for l in range(5, 11)) + 5 * 0.002) / K * 1e3)
    assert b["block 3"] == pytest.approx((sum(0.001 * l for l in range(11, 17)) + 5 * 0.002) / K * 1e3)
    assert b["all blocks"] == pytest.approx(b["block 1"] + b["block 2"] + b["block 3"])


def test_detection_slot_names_follow_the_detection_form(monkeypatch):
    wl = S.workload("c3")
    monkeypatch.setattr(bench, "SORTED", True)
    assert bench.kernel_name(0, wl) == "detect_sorted_kernel"
    monkeypatch.setattr(bench, "SORTED", False)
    assert bench.kernel_name(0, wl) == "detect_kernel<present>"
    assert bench.kernel_name(1, wl) == "detect_kernel<vanished>"
    assert bench.short_kernel("void ssc::detect_sorted_kernel<256, false, false>(ssc::DetectArgs)") == \
        "detect_sorted_kernel<256,f32>"
    assert bench.short_kernel("void ssc::detect_sorted_kernel<256, false, true, 1>(ssc::DetectArgs)") == \
        "detect_sorted_kernel<256,f32>"
    assert bench.short_kernel("void ssc::detect_sorted_kernel<128, true, false, 2>(ssc::DetectArgs)") == \
        "detect_sorted_kernel<128,bf16,2 passes>"
    assert bench.short_kernel("void ssc::detect_kernel<128, true, true, false>(ssc::DetectArgs)") == \
        "detect_kernel<128,bf16,vanished>"
    assert bench.launches_per_stride("detect_sorted_kernel<256,f32>", wl) == 1
    assert bench.short_kernel("void ssc::layer_kernel<64, 64, 2, false, true, true>(int const*, int const*, int, "
                              "ssc::LayerArgs)") == "layer_kernel<64,64,2,f32>"
    assert bench.short_kernel("void ssc::layer_kernel_wide<128, 256, 2, true, false>(int const*, int const*, int, "
                              "ssc::LayerArgs)") == "layer_kernel_wide<128,256,2,bf16>"
