#!/usr/bin/env python3
"""Throughput of the delta-scatter backbone on one MI355X.

One "step" is one sliding-window stride through the whole hot path: changed
cell detection on the pillar canvas, then for every layer the delta
contraction on the matrix cores, the update of the persistent map, the
activation-delta epilogue and the change-list propagation.

Workload (default): the full 3-block PointPillars backbone -- blocks of
4/6/6 3x3 convs with 64/128/256 channels, each block opened by a stride-2
conv, ReLU, fp32 -- on the 432x496 grid, fed by a seeded synthetic sweep
stream of ~12k occupied pillars whose 36 degree sector is refreshed each
stride (~10% of the pillars).  All strides are uploaded to
HBM before timing; the full window (stride 0) and `warmup` delta strides run
untimed, then exactly `steps` delta strides are timed.

Printed: one JSON line with
  value        changed-cell conv updates per second, sum_l |A_{l-1}| per stride
               (one changed input cell pushed through one layer's 3x3 filter bank)
  ms_per_step  wall-clock ms per stride over the timed region
  roofline     the dominant kernel's algorithmic flops (or bytes) per launch over
               its duration from HIP events stamped by the kernel's dispatch,
               against the MI355X peak
  cpu_baseline the CPU oracle (dense float64 recompute) on a bounded sample of the
               same strides
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import streams as S  # noqa: E402

PEAK_TFLOPS = {"f32": 157.3, "bf16": 2500.0}   # dense MFMA peaks of MI355X
PEAK_HBM_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.txt")
# change detection through sscater_step_sorted (one launch; the synthetic
# pillar lists are in row-major cell order), or sscater_step with --two-pass
SORTED = True
METRIC = "ms per stride and changed-cell conv updates/s; fraction of HBM/MFMA roofline"
PAPER_CONTEXT = {
    "hardware": "NVIDIA Jetson AGX Orin 32 GB (2048 Ampere cores) and AGX Xavier; real drone LiDAR, 504x504 grid",
    "single_layer": "up to 6.61x less processing time than scatter-based sparse convolution "
                    "(Cin 128, Cout 8, Orin, Table II)",
    "backbone_all_blocks_ms": {"sscater": 7.994378, "scatter_sparse": 27.821631, "table": "III (Orin, NC)"},
}


def log(msg: str) -> None:
    sys.stderr.write(msg + "\n")
    sys.stderr.flush()


def layers_of(wl):
    return [(l.cin, l.cout, l.stride, bool(l.relu)) for l in wl.layers]


def upload(strides, dtype):
    import torch
    out = []
    for st in strides:
        f = st.feats.view(np.int16) if dtype == "bf16" else st.feats
        out.append((torch.from_numpy(np.ascontiguousarray(st.idx)).cuda(),
                    torch.from_numpy(np.ascontiguousarray(f)).cuda()))
    torch.cuda.synchronize()
    return out


def layer_kernel_name(cin: int, cout: int, stride: int, dtype: str) -> str:
    """The library's kernel for a layer: the wide-layer kernel takes more than
    8 input chunks of 16 channels with cout >= 32, or more than 4 with
    cout >= 128; every other layer the narrow one."""
    nch = cin // 16
    wide = (nch > 8 and cout >= 32) or (nch > 4 and cout >= 128)
    return f"layer_kernel{'_wide' if wide else ''}<{cin},{cout},{stride},{dtype}>"


CONTRACT_SHAPES = {(128, 128), (128, 256), (256, 128), (256, 256)}


def layer_split(l: int, wl) -> bool:
    """Whether layer l (1-based) runs in two launches, the contraction of its
    changed input rows with all nine taps and the tap sum: the wide stride-1
    layers after the first."""
    sp = wl.layers[l - 1]
    return (l >= 2 and sp.stride == 1 and (sp.cin, sp.cout) in CONTRACT_SHAPES
            and not int(os.environ.get("SSCATER_FUSED_WIDE", "0") or 0))


def kernel_name(slot: int, wl, ups=(), points=False) -> str:
    """Slots: 0/1 detection, 1 + l layer l (its tap sum when split), then the
    upsamplers, then L + 1 + n_ups + l the contraction launch of layer l."""
    L, nu = len(wl.layers), len(ups)
    if slot == 0:
        if points:
            return "pillar_update_kernel"
        return "detect_sorted_kernel" if SORTED else "detect_kernel<present>"
    if slot == 1:
        return f"pfn_kernel<{wl.dtype}>" if points else "detect_kernel<vanished>"
    if slot >= L + 2 + nu:
        sp = wl.layers[slot - (L + 1 + nu) - 1]
        return f"contract_kernel<{sp.cin},{sp.cout},{wl.dtype}>"
    if slot >= L + 2:
        u = ups[slot - L - 2]
        cin = wl.layers[u.src - 1].cout
        return f"upsample_kernel<{cin},{u.cout},{u.stride},{wl.dtype}>"
    l = slot - 1
    sp = wl.layers[l - 1]
    if layer_split(l, wl):
        return f"tap_sum_kernel<{sp.cout},{wl.dtype}>"
    return layer_kernel_name(sp.cin, sp.cout, sp.stride, wl.dtype)


def layer_work(wl, l: int, act, pairs, launches: int):
    """Algorithmic work of layer l (1-based) over a run: flops, the bytes of
    the contraction's operands (input delta rows, weights once per launch,
    input list) and the bytes of the update (Z read + write, emitted deltas,
    output list and stamps)."""
    sp = wl.layers[l - 1]
    L = len(wl.layers)
    e_d = 4.0                                   # fp32 delta, or the bf16 pair
    e_w = 2.0 if wl.dtype == "bf16" else 4.0
    flops = 2.0 * sp.cin * sp.cout * pairs[l]
    b_c = act[l - 1] * sp.cin * e_d + launches * 9.0 * sp.cin * sp.cout * e_w + 8.0 * act[l - 1]
    b_s = act[l] * sp.cout * 8.0 + (act[l] * sp.cout * e_d if l < L else 0.0) + 8.0 * act[l]
    return flops, b_c, b_s


def block_times(wl, ms, K: int, n_ups: int = 0) -> dict:
    """Per-stride kernel time (us) of change detection, of each backbone block
    (a block starts at every stride-2 layer, as the PointPillars blocks do),
    of all blocks together and of the neck, from the per-slot sums of the
    profile pass (slot 0/1 detection, 1 + l layer l, then the upsamplers,
    then the contraction launches of layers that take two)."""
    L = len(wl.layers)
    out = {"detect": (ms[0] + ms[1]) / K * 1e3}
    b, tot = 0, 0.0
    for l in range(1, L + 1):
        if l == 1 or wl.layers[l - 1].stride == 2:
            b += 1
            out[f"block {b}"] = 0.0
        t = ms[1 + l] + (ms[L + 1 + n_ups + l] if len(ms) > L + 1 + n_ups + l else 0.0)
        out[f"block {b}"] += t / K * 1e3
        tot += t / K * 1e3
    out["all blocks"] = tot
    if n_ups:
        out["neck"] = sum(ms[L + 2 + u] for u in range(n_ups)) / K * 1e3
    return out


def cpu_model() -> str:
    """The host CPU's model name (as lscpu prints it), from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.lower().startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, ws, strides, first, budget_s, neck=()):
    """The oracle as it stands (dense float64 recompute of every layer, and of
    the neck when there is one, plus the change lists) on consecutive strides
    of the timed range, until the time budget is spent."""
    import oracle
    from oracle import sparse as SP
    layers = layers_of(wl)
    sub = [l.sub for l in wl.layers]
    sparse = any(sub)
    ups = [(u.src, u.cout, u.stride, u.relu) for u in neck]
    uw = S.neck_weights(wl.name) if neck else []
    prev = oracle.canvas_bits(S.canvas(strides[first - 1], wl.H, wl.W, wl.C0), wl.dtype)
    prev_occ = SP.occupancy(strides[first - 1].idx, wl.H, wl.W)
    t_total, u_total, n = 0.0, 0, 0
    for st in strides[first:]:
        canvas = S.canvas(st, wl.H, wl.W, wl.C0)
        t0 = time.perf_counter()
        bits = oracle.canvas_bits(canvas, wl.dtype)
        x = oracle.exact_canvas(canvas, wl.dtype)
        if sparse:
            occ = SP.occupancy(st.idx, wl.H, wl.W)
            ys = SP.forward(x, occ, ws, layers, sub, bf16_storage=(wl.dtype == "bf16"))
            lists = SP.changed_lists(prev, bits, prev_occ, occ, layers, sub)
            prev_occ = occ
        else:
            ys = oracle.forward(x, ws, layers, bf16_storage=(wl.dtype == "bf16"))
            lists = oracle.changed_lists(prev, bits, [l[2] for l in layers])
        if ups:
            oracle.forward_neck(ys, uw, ups, bf16_storage=(wl.dtype == "bf16"))
        t_total += time.perf_counter() - t0
        u_total += sum(len(a) for a in lists[:-1]) + sum(len(lists[u[0]]) for u in ups)
        prev = bits
        n += 1
        if t_total >= budget_s:
            break
    return {"value": u_total / t_total, "unit": "updates/s", "cores": oracle.threads(), "kind": "oracle",
            "cpu_model": cpu_model(), "ms_per_stride": t_total / n * 1e3,
            "sample": f"{n} consecutive delta strides of the timed range, each a dense float64 recompute of "
                      f"all {len(layers)} layers{' and the neck' if ups else ''} plus the per-layer change lists "
                      f"({t_total:.1f} s, "
                      f"{t_total / n * 1e3:.1f} ms per stride)"}


def cpu_baseline_points(wl, ws, spec, pw, batches, first, budget_s):
    """Points mode: the oracle's pillar feature net over each window, the dense
    float64 recompute of every layer and the event-based change lists, on
    consecutive strides of the timed range until the time budget is spent."""
    import oracle
    from oracle import pfn as P
    layers = layers_of(wl)
    t_total, u_total, n = 0.0, 0, 0
    for k in range(first, len(batches)):
        t0 = time.perf_counter()
        x = P.canvas(batches[k - spec.window + 1:k + 1], wl.H, wl.W, spec.x_min, spec.y_min, spec.res, pw)
        oracle.forward(x, ws, layers)
        a0 = P.changed_cells(batches[k], batches[k - spec.window], wl.H, wl.W, spec.x_min, spec.y_min, spec.res)
        m = np.zeros(wl.H * wl.W, dtype=bool)
        m[a0] = True
        m = m.reshape(wl.H, wl.W)
        act = [len(a0)]
        for l in wl.layers[:-1]:
            m = oracle.propagate_gather(m, l.stride)
            act.append(int(m.sum()))
        t_total += time.perf_counter() - t0
        u_total += sum(act)
        n += 1
        if t_total >= budget_s:
            break
    return {"value": u_total / t_total, "unit": "updates/s", "cores": oracle.threads(), "kind": "oracle",
            "cpu_model": cpu_model(), "ms_per_stride": t_total / n * 1e3,
            "sample": f"{n} consecutive delta strides of the timed range, each the pillar feature net over the "
                      f"window's points plus a dense float64 recompute of all {len(layers)} layers and the change "
                      f"lists ({t_total:.1f} s, {t_total / n * 1e3:.1f} ms per stride)"}


# --------------------------------------------------------------------------
# rocprofv3 digests: per-kernel durations from a --kernel-trace csv, and the
# HBM traffic of the dominant kernel from --pmc FETCH_SIZE / WRITE_SIZE runs
# scaled by what the same counters read for a plain copy of known size.
# --------------------------------------------------------------------------
KERNEL_SOURCES = ("detect.hip", "layer.hip", "contract.hip", "misc.hip", "upsample.hip", "pfn.hip",
                  "device_common.h", "sscater_internal.h")


# the device-code sources each kernel family is built from
KERNEL_FILES = {
    "layer_kernel": ("layer.hip", "device_common.h", "sscater_internal.h"),
    "contract_kernel": ("contract.hip", "device_common.h", "sscater_internal.h"),
    "tap_sum_kernel": ("contract.hip", "device_common.h", "sscater_internal.h"),
    "detect_kernel": ("detect.hip", "device_common.h", "sscater_internal.h"),
    "detect_sorted_kernel": ("detect.hip", "device_common.h", "sscater_internal.h"),
    "upsample_kernel": ("upsample.hip", "device_common.h", "sscater_internal.h"),
    "pfn_kernel": ("pfn.hip", "device_common.h", "sscater_internal.h"),
    "pillar_update_kernel": ("pfn.hip", "device_common.h", "sscater_internal.h"),
}


def kernel_source_digest(kernel: str = "") -> str:
    """sha256 over the device-code sources `kernel` is built from (all of
    them when the kernel is not named): a measured traffic figure is only
    reported while the kernel is the one it was measured on."""
    base = kernel.split("<")[0]
    files = next((f for fam, f in KERNEL_FILES.items() if base == fam or base.startswith(fam + "_")), KERNEL_SOURCES)
    h = hashlib.sha256()
    for name in files:
        h.update(name.encode())
        with open(os.path.join(ROOT, "paper_2512_08557_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _traffic_records():
    """The records of the traffic file: blocks of "key value" lines, each
    opened by a "#" comment line."""
    recs, cur = [], None
    try:
        with open(TRAFFIC_FILE) as fh:
            for line in fh:
                line = line.rstrip("\n")
                if line.startswith("#"):
                    cur = {"#": line}
                    recs.append(cur)
                elif line.strip() and cur is not None:
                    k, _, v = line.strip().partition(" ")
                    cur[k] = v.strip()
    except OSError:
        pass
    return recs


def read_traffic(kernel: str, workload: str):
    """Measured HBM bytes per launch of `kernel` on `workload`, or None when
    absent or stale (measured on other kernel sources)."""
    for kv in _traffic_records():
        if (kv.get("source_sha256") == kernel_source_digest(kernel) and kv.get("kernel") == kernel
                and kv.get("workload") == workload):
            try:
                return float(kv["traffic_bytes_per_launch"])
            except (KeyError, ValueError):
                return None
    return None


def write_traffic(rec: str, kernel: str, workload: str) -> None:
    """Replace the record of (kernel, workload) in the traffic file by rec."""
    keep = [r for r in _traffic_records() if not (r.get("kernel") == kernel and r.get("workload") == workload)]
    out = []
    for r in keep:
        out.append(r["#"])
        out += [f"{k} {v}" for k, v in r.items() if k != "#"]
        out.append("")
    with open(TRAFFIC_FILE, "w") as fh:
        fh.write("\n".join(out) + rec)


def short_kernel(name: str) -> str:
    """'void ssc::layer_kernel<64, 64, 1, false>(ssc::LayerArgs)' -> 'layer_kernel<64,64,1,f32>'."""
    base = name.split("(")[0].replace("void ", "").replace("ssc::", "")
    if "<" not in base:
        return base
    fn, _, targs = base.partition("<")
    t = [x.strip() for x in targs.rstrip(">").split(",")]
    dt = lambda v: "bf16" if v == "true" else "f32"
    if fn == "detect_sorted_kernel" and len(t) in (3, 4):
        # the fourth argument: rows per lane group and wavefront (several for long lists)
        passes = f",{t[3]} passes" if len(t) == 4 and t[3] != "1" else ""
        return f"detect_sorted_kernel<{t[0]},{dt(t[1])}{passes}>"
    if fn == "detect_kernel" and len(t) in (3, 4):
        return f"detect_kernel<{t[0]},{dt(t[1])},{'vanished' if t[2] == 'true' else 'present'}>"
    if fn in ("layer_kernel", "layer_kernel_wide") and len(t) in (4, 5, 6):
        return f"{fn}<{t[0]},{t[1]},{t[2]},{dt(t[3])}>"
    if fn == "contract_kernel" and len(t) == 3:
        return f"contract_kernel<{t[0]},{t[1]},{dt(t[2])}>"
    if fn == "tap_sum_kernel" and len(t) == 3:
        return f"tap_sum_kernel<{t[0]},{dt(t[1])}>"
    if fn == "pfn_kernel" and len(t) == 1:
        return f"pfn_kernel<{dt(t[0])}>"
    return fn + "<" + ",".join(t) + ">"


def launches_per_stride(kernel: str, wl) -> int:
    if kernel.startswith(("detect_kernel", "detect_sorted_kernel", "pillar_update_kernel", "pfn_kernel")):
        return 1
    L = len(wl.layers)
    names = [kernel_name(1 + l, wl) for l in range(1, L + 1)]
    names += [kernel_name(L + 1 + l, wl) for l in range(1, L + 1) if layer_split(l, wl)]
    return sum(1 for n in names if n == kernel)


def _csv_rows(path):
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


def digest_trace(path: str, steps: int, warmup: int, wl) -> str:
    """Markdown tables of a --kernel-trace csv of the default bench command:
    three passes of (full window, warmup, the timed strides) -- timed, with an
    event after every stride, with events stamped by every launch -- then the
    full recomputes."""
    rows = sorted(_csv_rows(path), key=lambda r: int(r["Start_Timestamp"]))
    by = {}
    for r in rows:
        by.setdefault(short_kernel(r["Kernel_Name"]), []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    total = sum(sum(v) for v in by.values())
    out = ["| Kernel | Calls | Avg (us) | Median (us) | Min (us) | Max (us) | Share |",
           "|---|---|---|---|---|---|---|"]
    for k, v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| {k} | {len(v)} | {statistics.fmean(v):.2f} | {statistics.median(v):.2f} | {min(v):.2f} | "
                   f"{max(v):.2f} | {100 * sum(v) / total:.2f} % |")
    out += ["", "| Kernel | Timed strides: avg (us) | Event-timed pass: avg (us) |", "|---|---|---|"]
    for k, v in sorted(by.items()):
        n = launches_per_stride(k, wl)
        if n == 0:
            continue
        if wl.name in S.PFNS:
            first = S.PFNS[wl.name].window             # batches of the first window
        else:
            first = 0 if k.endswith("vanished>") else 1   # no vanish pass on a full window
        span = (first + warmup + steps) * n            # launches of one pass
        a0, a1 = (first + warmup) * n, (first + warmup + steps) * n
        b0, b1 = 2 * span + a0, 2 * span + a1          # third pass: events stamped by every launch
        if len(v) >= b1:
            out.append(f"| {k} | {statistics.fmean(v[a0:a1]):.2f} | {statistics.fmean(v[b0:b1]):.2f} |")
    return "\n".join(out)


def digest_sweep_trace(path: str, steps: int, warmup: int) -> str:
    """Per sweep shape, the layer kernel's rocprofv3 duration over the timed
    strides and over the event-timed pass of a --kernel-trace csv of
    `bench.py --sweep` (per shape: the timed pass, the event-timed pass, then
    10 full recomputes)."""
    rows = sorted(_csv_rows(path), key=lambda r: int(r["Start_Timestamp"]))
    by = {}
    for r in rows:
        by.setdefault(short_kernel(r["Kernel_Name"]), []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    span = 1 + warmup + steps
    out = ["| Cin | Cout | layer kernel | timed strides: avg (us) | event-timed pass: avg (us) | full recompute: avg (us) |",
           "|---|---|---|---|---|---|"]
    for ci in S.SWEEP_CIN:
        for co in S.SWEEP_COUT:
            k = layer_kernel_name(ci, co, 1, "f32")
            v = by.get(k, [])
            if len(v) < 2 * span:
                continue
            out.append(f"| {ci} | {co} | {k} | {statistics.fmean(v[1 + warmup:span]):.2f} | "
                       f"{statistics.fmean(v[span + 1 + warmup:2 * span]):.2f} | "
                       f"{statistics.fmean(v[2 * span:]):.2f} |")
    for k in sorted(by):
        if k.startswith(("detect_kernel", "detect_sorted_kernel")):
            v = by[k]
            out.append(f"| all | all | {k} | {statistics.fmean(v):.2f} (every launch) | | |")
    return "\n".join(out)


def digest_pmc(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, copy_bytes, kernel, per_stride,
               steps, workload) -> str:
    """HBM bytes per launch of `kernel` over the timed strides (the last
    steps*per_stride dispatches), FETCH_SIZE and WRITE_SIZE each scaled by the
    ratio of the copy's true size to what the counter reads for it."""
    def per_kernel(path, name_pred):
        vals = [float(r["Counter_Value"]) for r in sorted(_csv_rows(path), key=lambda r: int(r["Dispatch_Id"]))
                if name_pred(r["Kernel_Name"])]
        return vals
    fk = per_kernel(fetch_csv, lambda n: short_kernel(n) == kernel)[-steps * per_stride:]
    wk = per_kernel(write_csv, lambda n: short_kernel(n) == kernel)[-steps * per_stride:]
    cf = per_kernel(copy_fetch_csv, lambda n: "copyBuffer" in n)
    cw = per_kernel(copy_write_csv, lambda n: "copyBuffer" in n)
    cf_kib, cw_kib = max(cf), max(cw)
    f_scale, w_scale = copy_bytes / (cf_kib * 1024.0), copy_bytes / (cw_kib * 1024.0)
    fetch, write = statistics.fmean(fk), statistics.fmean(wk)
    traffic = fetch * 1024.0 * f_scale + write * 1024.0 * w_scale
    lines = [
        "# HBM traffic per launch of the dominant kernel (rocprofv3 --pmc FETCH_SIZE, WRITE_SIZE)",
        f"source_sha256 {kernel_source_digest(kernel)}",
        f"kernel {kernel}",
        f"workload {workload}",
        f"dispatches {len(fk)}",
        f"fetch_kib_per_launch {fetch:.3f}",
        f"write_kib_per_launch {write:.3f}",
        f"copy_bytes {copy_bytes}",
        f"copy_fetch_kib {cf_kib:.3f}",
        f"copy_write_kib {cw_kib:.3f}",
        f"fetch_scale {f_scale:.5f}",
        f"write_scale {w_scale:.5f}",
        f"traffic_bytes_per_launch {traffic:.1f}",
    ]
    return "\n".join(lines) + "\n"


def digest_counters(path: str, kernel: str, per_stride: int, steps: int) -> str:
    """Markdown table of every counter of a rocprofv3 --pmc csv, averaged over
    the timed launches of `kernel` (its last steps*per_stride dispatches)."""
    by = {}
    for r in sorted(_csv_rows(path), key=lambda r: int(r["Dispatch_Id"])):
        if short_kernel(r["Kernel_Name"]) == kernel:
            by.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    out = [f"| Counter ({kernel}) | Dispatches | Mean per launch |", "|---|---|---|"]
    for name in sorted(by):
        v = by[name][-steps * per_stride:]
        out.append(f"| {name} | {len(v)} | {statistics.fmean(v):.6g} |")
    return "\n".join(out)


def dense_torch_ms(wl, ws, canvases, reps: int = 20) -> float:
    """Context: the same layer stack recomputed densely from the canvas by
    the vendor convolution (torch conv2d, fp32 or bf16 storage as the
    workload, NCHW, one image per canvas), ms per pass, median of reps."""
    import torch
    import torch.nn.functional as F
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x = torch.stack([torch.from_numpy(np.ascontiguousarray(
        S.bf16_bits_to_f32(c.view(np.uint16)).reshape(c.shape) if wl.dtype == "bf16" else c)).permute(2, 0, 1)
        for c in canvases]).contiguous().to("cuda", dt)
    wt = [torch.from_numpy(np.ascontiguousarray(w)).to("cuda", dt) for w in ws]

    def run():
        y = x
        for l, w in zip(wl.layers, wt):
            y = F.conv2d(y, w, stride=l.stride, padding=1)
            if l.relu:
                y = torch.relu(y)
        return y

    for _ in range(3):
        run()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        run()
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    return statistics.median(times)


def copy_bandwidth(nbytes: int = 1 << 30, reps: int = 3) -> float:
    """Measured HBM bandwidth of a plain device copy of nbytes (larger than
    every cache): bytes read + written per second, best of reps, in GB/s."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    best = float("inf")
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b) / 1e3)
    del src, dst
    return 2.0 * nbytes / best / 1e9


def stride_roofline(wl, act, pairs, K: int, mean_pillars: float, t_us: float, copy_gbs: float) -> dict:
    """Roofline time of one stride from its algorithmic work, per layer the
    larger of its flops at the MFMA peak and its bytes at the bandwidth, plus
    the detection's bytes: t_roof = B_a1/BW + sum_l max(F_l/P, B_l/BW), against
    the MI355X HBM peak and against the measured copy bandwidth; frac =
    t_roof / the measured stride time.  act and pairs are per-layer totals
    over the K timed strides."""
    L = len(wl.layers)
    bf16 = wl.dtype == "bf16"
    e_in, e_d, e_w = (2.0 if bf16 else 4.0), 4.0, (2.0 if bf16 else 4.0)
    peak = PEAK_TFLOPS[wl.dtype] * 1e12
    A = [a / K for a in act]
    P = mean_pillars
    b_a1 = P * (4 + wl.C0 * e_in) + P * wl.C0 * e_in + A[0] * wl.C0 * (e_in + e_d) + 8.0 * P
    fl, by = [], []
    for l in range(1, L + 1):
        sp = wl.layers[l - 1]
        fl.append(2.0 * sp.cin * sp.cout * pairs[l] / K)
        by.append(A[l - 1] * sp.cin * e_d + A[l] * sp.cout * 8.0 + (A[l] * sp.cout * e_d if l < L else 0.0) +
                  9.0 * sp.cin * sp.cout * e_w + 8.0 * (A[l - 1] + A[l]))
    out = {"t_measured_us": t_us, "alg_flops": sum(fl), "alg_bytes": b_a1 + sum(by), "copy_gbs": copy_gbs}
    for tag, bw in (("spec", PEAK_HBM_GBS * 1e9), ("copy", copy_gbs * 1e9)):
        t = b_a1 / bw + sum(max(f / peak, b / bw) for f, b in zip(fl, by))
        out[f"t_roof_us_{tag}"] = t * 1e6
        out[f"frac_{tag}"] = t * 1e6 / t_us
    return out


def copy_calibration(nbytes: int) -> int:
    """A plain device-to-device copy of nbytes (the counters' calibration)."""
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] copied {nbytes} bytes 3 times")
    return 0


def stack_strides(per_stream, H: int, W: int):
    """One stride of a batched handle from one stride of every stream: image
    b's pillar p becomes cell b*H*W + p."""
    idx = np.concatenate([st.idx.astype(np.int64) + b * H * W for b, st in enumerate(per_stream)]).astype(np.int32)
    feats = np.ascontiguousarray(np.concatenate([st.feats for st in per_stream]))
    return S.Stride(per_stream[0].index, idx, feats)


def run_streams(wl, ws, K: int, W: int, n: int, cpu_seconds, no_cpu: bool, batched: bool = False,
                dense: bool = False) -> dict:
    """n independent sensor streams (scene seeds 2512 + k) advanced together,
    as the 1024x1024 four-stream workload runs: either one handle each on its
    own HIP stream, or (batched) one handle over all n images, so that every
    stride of all streams is one launch chain.  Whole-GPU throughput over K
    strides of every stream, per-kernel timing from dispatch-stamped events
    on every handle."""
    import torch
    from paper_2512_08557_amd import Engine

    data = [S.make_stream(wl.name, seed=S.SCENE_SEED + k, n_strides=W + K) for k in range(n)]
    if batched:
        devs = [upload([stack_strides([d[k] for d in data], wl.H, wl.W) for k in range(len(data[0]))], wl.dtype)]
        engs = [Engine(wl.H, wl.W, wl.C0, layers_of(wl), ws, dtype=wl.dtype, max_pillars=n * wl.max_pillars,
                       batch=n)]
        hs = [torch.cuda.Stream()]
    else:
        devs = [upload(st, wl.dtype) for st in data]
        engs = [Engine(wl.H, wl.W, wl.C0, layers_of(wl), ws, dtype=wl.dtype, max_pillars=wl.max_pillars)
                for _ in range(n)]
        hs = [torch.cuda.Stream() for _ in range(n)]
    L = len(wl.layers)

    def run_range(lo, hi):
        for k in range(lo, hi):
            for i in range(len(engs)):
                engs[i].step(*devs[i][k], stream=hs[i], sorted=SORTED)

    run_range(0, 1 + W)
    torch.cuda.synchronize()
    before = [e.stats(stream=h) for e, h in zip(engs, hs)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_range(1 + W, 1 + W + K)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    after = [e.stats(stream=h) for e, h in zip(engs, hs)]
    act = [[a["active_total"][l] - b["active_total"][l] for l in range(L + 1)] for a, b in zip(after, before)]
    prs = [[a["pairs_total"][l] - b["pairs_total"][l] for l in range(L + 1)] for a, b in zip(after, before)]
    updates = sum(sum(x[:L]) for x in act)
    value = updates / (wall_ms / 1e3)
    log(f"[bench] {n} streams ({'one batched handle' if batched else 'one handle each'}) x {K} strides in "
        f"{wall_ms:.2f} ms -> {wall_ms / K * 1e3:.1f} us per stride of all streams, {value:.3e} updates/s")

    # per-kernel pass: the same strides again, every handle timed
    for e, h in zip(engs, hs):
        e.reset(stream=h)
    run_range(0, 1 + W)
    torch.cuda.synchronize()
    b2 = [e.stats(stream=h) for e, h in zip(engs, hs)]
    for e, h in zip(engs, hs):
        e.profile_read(stream=h)
        e.profile(True)
    run_range(1 + W, 1 + W + K)
    kernels = {}
    for i, (e, h) in enumerate(zip(engs, hs)):
        ms, cnt = e.profile_read(stream=h)
        e.profile(False)
        a2 = e.stats(stream=h)
        pairs2 = [a2["pairs_total"][l] - b2[i]["pairs_total"][l] for l in range(L + 1)]
        for slot in range(L + 2):
            if cnt[slot] == 0:
                continue
            k = kernels.setdefault(kernel_name(slot, wl), {"ms": 0.0, "launches": 0, "flops": 0.0})
            k["ms"] += ms[slot]
            k["launches"] += cnt[slot]
            if slot >= 2:
                sp = wl.layers[slot - 2]
                k["flops"] += 2.0 * sp.cin * sp.cout * pairs2[slot - 1]
    for name, k in kernels.items():
        log(f"[bench] {name:34s} {k['launches']:5d} launches  avg {k['ms'] / k['launches'] * 1e3:8.2f} us")
    dom_name, dom = max(kernels.items(), key=lambda kv: kv[1]["ms"])
    launch_us = dom["ms"] / dom["launches"] * 1e3
    achieved = dom["flops"] / (dom["ms"] / 1e3) / 1e12
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[wl.dtype], "unit": "TFLOP/s",
                "frac": achieved / PEAK_TFLOPS[wl.dtype], "traffic": read_traffic(dom_name, wl.name),
                "kernel": dom_name, "launches": dom["launches"], "avg_launch_us": launch_us,
                "alg_flops_per_launch": dom["flops"] / dom["launches"],
                "note": ("one launch per kernel and stride covers every stream" if batched else
                         "kernels of the different streams overlap; each duration is the kernel's own")}
    for e in engs:
        e.close()
    dense_ms = None
    if dense:      # context: the vendor library's dense recompute of every stream (a batch of n images)
        try:
            dense_ms = dense_torch_ms(wl, ws, [S.canvas(d[W + K], wl.H, wl.W, wl.C0) for d in data])
            log(f"[bench] dense recompute with torch conv2d: {dense_ms * 1e3:.1f} us per pass of all streams "
                f"({dense_ms / (wall_ms / K):.1f}x the delta stride)")
        except Exception as exc:  # context only
            log(f"[bench] dense torch recompute skipped: {exc}")
    # all streams' work of one stride against the stride roofline
    cgbs = copy_bandwidth()
    sroof = stride_roofline(wl, [sum(x[l] for x in act) for l in range(L + 1)],
                            [sum(x[l] for x in prs) for l in range(L + 1)], K,
                            float(sum(np.mean([len(s.idx) for s in d[1 + W:]]) for d in data)), wall_ms / K * 1e3, cgbs)
    log(f"[bench] stride roofline: {sroof['t_roof_us_spec']:.1f} us at 8 TB/s ({100 * sroof['frac_spec']:.1f} %), "
        f"{sroof['t_roof_us_copy']:.1f} us at the measured copy bandwidth {cgbs:.0f} GB/s "
        f"({100 * sroof['frac_copy']:.1f} %)")
    cpu = None
    if not no_cpu:
        try:
            log(f"[bench] CPU oracle baseline (budget {cpu_seconds:.0f} s, stream 0)")
            cpu = cpu_baseline(wl, ws, data[0], 1 + W, cpu_seconds)
        except Exception as exc:  # the oracle is optional for the GPU number
            log(f"[bench] CPU baseline skipped: {exc}")
    return {"metric": METRIC, "value": value, "unit": "updates/s", "n_gpus": 1, "steps": K, "warmup": W,
            "ms_per_step": wall_ms / K, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": wl.dtype, "data": "synthetic",
            "config": {"workload": f"{wl.name}: {wl.description}", "grid": f"{wl.W}x{wl.H}", "C0": wl.C0,
                       "detection": "one launch (sorted pillar lists)" if SORTED else "two passes",
                       "streams": n, "batched": batched, "layers": [f"{l.cin}->{l.cout} s{l.stride}" for l in wl.layers],
                       "strides": "a stride is one step of every stream; full window + warmup untimed",
                       "mean_active_per_stream": [sum(x[l] for x in act) / (K * n) for l in range(L + 1)]},
            "kernels": {k: {"launches": v["launches"], "avg_us": v["ms"] / v["launches"] * 1e3}
                        for k, v in kernels.items()},
            "dense_torch_ms": dense_ms, "roofline": roofline, "stride_roofline": sroof, "cpu_baseline": cpu}


def run_sweep(K: int, W: int, n_full: int) -> dict:
    """Single-layer channel sweep (the shapes of the paper's single-layer
    timing tables, Sec. IV-B, Tables I and II) on the 504 x 504 drone stream:
    per shape the delta stride (wall clock over K strides), the layer kernel
    alone (dispatch-stamped events), and the full recompute of the same
    windows through the same kernels (reset + one pass over every active
    pillar, the scatter conv without recycling)."""
    import torch
    from paper_2512_08557_amd import Engine

    rows = []
    stream = torch.cuda.current_stream()
    for ci in S.SWEEP_CIN:
        for co in S.SWEEP_COUT:
            wl = S.workload(f"l{ci}x{co}")
            strides = S.make_stream(wl.name, n_strides=W + K)
            dev = upload(strides, wl.dtype)
            eng = Engine(wl.H, wl.W, wl.C0, layers_of(wl), S.weights(wl.name), dtype=wl.dtype,
                         max_pillars=wl.max_pillars)
            for k in range(1 + W):
                eng.step(*dev[k], sorted=SORTED)
            torch.cuda.synchronize()
            before = eng.stats()
            t0 = time.perf_counter()
            for k in range(1 + W, 1 + W + K):
                eng.step(*dev[k], sorted=SORTED)
            torch.cuda.synchronize()
            wall_ms = (time.perf_counter() - t0) * 1e3
            after = eng.stats()
            a_in = after["active_total"][0] - before["active_total"][0]
            a_out = after["active_total"][1] - before["active_total"][1]
            pairs = after["pairs_total"][1] - before["pairs_total"][1]
            # per-kernel pass over the same strides
            eng.reset()
            for k in range(1 + W):
                eng.step(*dev[k], sorted=SORTED)
            eng.profile_read()
            eng.profile(True)
            for k in range(1 + W, 1 + W + K):
                eng.step(*dev[k], sorted=SORTED)
            ms, cnt = eng.profile_read()
            eng.profile(False)
            # full recompute of n_full windows spread over the timed range
            full = []
            for k in range(1 + W, 1 + W + K, max(1, K // n_full)):
                eng.reset()
                torch.cuda.synchronize()
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                eng.step(*dev[k], sorted=SORTED)
                b.record(stream)
                torch.cuda.synchronize()
                full.append(a.elapsed_time(b))
            eng.close()
            ms_stride = wall_ms / K
            full_ms = statistics.fmean(full)
            layer_us = ms[2] / cnt[2] * 1e3
            rows.append({"cin": ci, "cout": co, "ms_per_stride": ms_stride, "layer_kernel_us": layer_us,
                         "detect_us": (ms[0] + ms[1]) / K * 1e3, "full_recompute_ms": full_ms,
                         "speedup_vs_full_recompute": full_ms / ms_stride,
                         "updates_per_s": a_in / (wall_ms / 1e3),
                         "layer_tflops": 2.0 * ci * co * pairs / (ms[2] / 1e3) / 1e12,
                         "mean_changed_in": a_in / K, "mean_changed_out": a_out / K,
                         "mean_pillars": float(np.mean([len(x.idx) for x in strides[1 + W:]]))})
            r = rows[-1]
            log(f"[sweep] {ci:4d} -> {co:4d}: {ms_stride * 1e3:7.1f} us/stride (layer {layer_us:6.1f} us, "
                f"{r['layer_tflops']:5.2f} TFLOP/s), full recompute {full_ms * 1e3:7.1f} us, "
                f"x{r['speedup_vs_full_recompute']:.2f}; |A_0| {r['mean_changed_in']:.0f}, "
                f"|A_1| {r['mean_changed_out']:.0f}")
    return {"metric": "single-layer sweep: ms per stride, layer kernel us, full recompute ms", "n_gpus": 1,
            "steps": K, "warmup": W, "dtype": "f32", "data": "synthetic",
            "config": {"workload": "single 3x3 s1 conv (ReLU), Cin 16..128 x Cout 8..128, 504x504 drone scan"},
            "rows": rows}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c3", choices=sorted(S.WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-kernel event pass")
    ap.add_argument("--no-full", action="store_true", help="skip the GPU full-recompute timing")
    ap.add_argument("--no-dense", action="store_true",
                    help="skip the context timing of the same layers recomputed densely by torch conv2d")
    ap.add_argument("--two-pass", action="store_true",
                    help="detect changes with the two passes of sscater_step instead of the one launch of "
                         "sscater_step_sorted (the synthetic pillar lists are sorted by cell)")
    ap.add_argument("--neck", action="store_true", help="include the upsampling neck (c3, c4)")
    ap.add_argument("--streams", type=int, default=0,
                    help="independent streams advanced together (default: 4 for c5, else 1)")
    ap.add_argument("--separate", action="store_true",
                    help="several streams: one handle per stream on its own HIP stream instead of one batched handle")
    ap.add_argument("--sweep", action="store_true",
                    help="single-layer channel sweep over all 20 (Cin, Cout) shapes on the 504x504 drone stream")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (counter calibration)")
    ap.add_argument("--digest-trace", metavar="CSV", help="summarise a rocprofv3 kernel-trace csv and exit")
    ap.add_argument("--digest-pmc", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="turn rocprofv3 --pmc csvs into the traffic record of the dominant kernel and exit")
    ap.add_argument("--digest-counters", metavar="CSV",
                    help="average every counter of a rocprofv3 --pmc csv over the timed launches of --kernel and exit")
    ap.add_argument("--kernel", default="layer_kernel<64,64,1,f32>", help="kernel of --digest-pmc / --digest-counters")
    args = ap.parse_args()
    global SORTED
    SORTED = not args.two_pass

    if args.digest_trace:
        if args.sweep:
            print(digest_sweep_trace(args.digest_trace, args.steps, args.warmup))
        else:
            print(digest_trace(args.digest_trace, args.steps, args.warmup, S.workload(args.workload)))
        return 0
    if args.digest_counters:
        per = launches_per_stride(args.kernel, S.workload(args.workload))
        print(digest_counters(args.digest_counters, args.kernel, max(per, 1), args.steps))
        return 0
    if args.digest_pmc:
        per = launches_per_stride(args.kernel, S.workload(args.workload))
        rec = digest_pmc(*args.digest_pmc, args.copy_bytes, args.kernel, max(per, 1), args.steps, args.workload)
        write_traffic(rec, args.kernel, args.workload)
        print(rec)
        return 0
    if args.copy_bytes:
        return copy_calibration(args.copy_bytes)

    if args.gpus != 1:
        log("bench.py: the benchmark runs on one GPU only; multi-GPU runs are not supported "
            "(independent sensor streams would shard one per GPU with no communication).")
        return 2
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        log("bench.py: launched with WORLD_SIZE > 1; the benchmark runs on one GPU only.")
        return 2

    import torch
    from paper_2512_08557_amd import Engine

    torch.cuda.set_device(0)
    if args.sweep:
        print(json.dumps(run_sweep(args.steps, args.warmup, 10)), flush=True)
        return 0
    wl = S.workload(args.workload)
    ws = S.weights(args.workload)
    K, W = args.steps, args.warmup
    n_streams = args.streams or (4 if wl.name == "c5" else 1)
    if n_streams > 1:
        print(json.dumps(run_streams(wl, ws, K, W, n_streams, args.cpu_seconds, args.no_cpu,
                                     batched=not args.separate, dense=not args.no_dense)), flush=True)
        return 0
    log(f"[bench] workload {wl.name}: {wl.description}; generating {W + K} delta strides")
    neck = S.neck(wl.name) if args.neck else ()
    if args.neck and not neck:
        log(f"bench.py: workload {wl.name} has no neck")
        return 2
    spec = S.PFNS.get(wl.name)
    if spec is not None:
        # points mode: batches -(window-1)..0 build the first window
        strides = S.make_point_stream(wl.name, n_strides=W + K)
        first = spec.window
        dev = [torch.from_numpy(b).cuda() for b in strides]
        torch.cuda.synchronize()
        pw = S.pfn_weights(wl.name)
        # sized so that one step may take a whole window's points (the full recompute)
        eng = Engine(wl.H, wl.W, wl.C0, layers_of(wl), ws, dtype=wl.dtype, max_pillars=0,
                     pfn=(spec.x_min, spec.y_min, spec.res, spec.max_points, spec.window,
                          spec.window * spec.max_new_points), pfn_weights=pw)
        step = lambda k: eng.step_points(dev[k])
    else:
        strides = S.make_stream(wl.name, n_strides=W + K)
        first = 1
        dev = upload(strides, wl.dtype)
        sub = [l.sub for l in wl.layers]
        eng = Engine(wl.H, wl.W, wl.C0, layers_of(wl), ws, dtype=wl.dtype, max_pillars=wl.max_pillars,
                     ups=[(u.src, u.cout, u.stride, u.relu) for u in neck],
                     up_weights=S.neck_weights(wl.name) if neck else (),
                     submanifold=sub if any(sub) else None)
        step = lambda k: eng.step(*dev[k], sorted=SORTED)
    L = len(wl.layers)

    def run_range(lo, hi):
        for k in range(lo, hi):
            step(k)

    # full window + warmup (untimed)
    run_range(0, first + W)
    torch.cuda.synchronize()
    before = eng.stats()

    # ---- timed region: exactly K delta strides, nothing else on the stream ----
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_range(first + W, first + W + K)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    after = eng.stats()
    wall_ms = (t1 - t0) * 1e3

    # ---- latency pass: the same strides again, a HIP event after each ----
    eng.reset()
    run_range(0, first + W)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k in range(K):
        step(first + W + k)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    per_stride = [evs[k].elapsed_time(evs[k + 1]) for k in range(K)]
    act_in = [after["active_total"][l] - before["active_total"][l] for l in range(L + 1)]
    pairs = [after["pairs_total"][l] - before["pairs_total"][l] for l in range(L + 1)]
    updates = sum(act_in[:L])          # sum_l |A_{l-1}| over the timed strides
    updates += sum(act_in[u.src] for u in neck)   # each upsampler takes its source layer's changed cells
    ms_per_step = wall_ms / K
    value = updates / (wall_ms / 1e3)
    log(f"[bench] {K} strides in {wall_ms:.2f} ms -> {ms_per_step * 1e3:.1f} us/stride, "
        f"{value:.3e} updates/s; mean |A_l| = {[round(a / K) for a in act_in]}")

    # ---- per-kernel pass: same strides, HIP events stamped by every launch ----
    roofline = None
    kernels = {}
    blocks = None
    if not args.no_profile:
        eng.reset()
        run_range(0, first + W)
        eng.profile_read()               # drop anything recorded so far
        b2 = eng.stats()
        eng.profile(True)
        run_range(first + W, first + W + K)
        ms, cnt = eng.profile_read()
        eng.profile(False)
        a2 = eng.stats()
        pairs2 = [a2["pairs_total"][l] - b2["pairs_total"][l] for l in range(L + 1)]
        act2 = [a2["active_total"][l] - b2["active_total"][l] for l in range(L + 1)]
        nu = len(neck)
        for slot in range(2 * L + 2 + nu):
            if cnt[slot] == 0:
                continue
            name = kernel_name(slot, wl, neck, points=spec is not None)
            k = kernels.setdefault(name, {"ms": 0.0, "launches": 0, "flops": 0.0, "bytes": 0.0})
            k["ms"] += ms[slot]
            k["launches"] += cnt[slot]
            if 2 <= slot < L + 2 or slot >= L + 2 + nu:
                contraction = slot >= L + 2 + nu
                l = slot - (L + 1 + nu) if contraction else slot - 1
                f, b_c, b_s = layer_work(wl, l, act2, pairs2, cnt[slot])
                if not layer_split(l, wl):
                    k["flops"] += f
                    k["bytes"] += b_c + b_s
                elif contraction:     # the product carries the flops, its operands the bytes
                    k["flops"] += f
                    k["bytes"] += b_c
                else:                 # the tap sum: Z, emitted deltas, lists
                    k["bytes"] += b_s
        for name, k in kernels.items():
            log(f"[bench] {name:34s} {k['launches']:5d} launches  avg {k['ms'] / k['launches'] * 1e3:8.2f} us  "
                f"total {k['ms']:.3f} ms")
        blocks = block_times(wl, ms, K, len(neck))
        log("[bench] per stride (sum of kernel durations): " +
            ", ".join(f"{k} {v:.1f} us" for k, v in blocks.items()))
        dom_name, dom = max(kernels.items(), key=lambda kv: kv[1]["ms"])
        if dom["flops"] > 0 or dom["bytes"] > 0:
            # start and end stamped by the kernel's own dispatch packet
            launch_us = dom["ms"] / dom["launches"] * 1e3
            secs = launch_us * 1e-6 * dom["launches"]
            intensity = dom["flops"] / max(dom["bytes"], 1.0)
            peak_t = PEAK_TFLOPS[wl.dtype]
            traffic = read_traffic(dom_name, wl.name)
            if intensity >= peak_t * 1e12 / (PEAK_HBM_GBS * 1e9):
                achieved = dom["flops"] / secs / 1e12
                roofline = {"bound": "mfma", "achieved": achieved, "peak": peak_t, "unit": "TFLOP/s",
                            "frac": achieved / peak_t, "traffic": traffic}
            else:
                achieved = dom["bytes"] / secs / 1e9
                roofline = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": achieved / PEAK_HBM_GBS, "traffic": traffic}
            roofline.update({"kernel": dom_name, "launches": dom["launches"],
                             "avg_launch_us": launch_us,
                             # measured HBM bytes per launch over the launch time
                             "traffic_gbs": traffic / (launch_us * 1e-6) / 1e9 if traffic else None,
                             "alg_flops_per_launch": dom["flops"] / dom["launches"],
                             "alg_bytes_per_launch": dom["bytes"] / dom["launches"],
                             "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, "
                                             "scaled by a plain copy)"})

    # ---- floor: strides whose input equals the previous one bit for bit ----
    # every launch of a stride runs and finds an empty list.  The per-launch
    # event times are the GPU's fixed cost per launch; the wall clock of such
    # strides is bound by the host's enqueue of the chain (the GPU finishes
    # right after the last call), unlike the work-carrying strides above
    floor = None
    if not args.no_profile:
        last_k = first + W + K - 1
        nz = 20

        def zero_change():
            if spec is not None:
                eng.step_points(None)      # no new points (the window keeps draining)
            else:
                step(last_k)

        for _ in range(3):                 # settle
            zero_change()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(nz):
            zero_change()
        torch.cuda.synchronize()
        wall_floor = (time.perf_counter() - t0) / nz * 1e6
        eng.profile_read()
        eng.profile(True)
        for _ in range(nz):
            zero_change()
        fms, fcnt = eng.profile_read()
        eng.profile(False)
        floor = {"stride_us": wall_floor,
                 "kernels_us": {kernel_name(sl, wl, neck, points=spec is not None): fms[sl] / fcnt[sl] * 1e3
                                for sl in range(len(fcnt)) if fcnt[sl]}}
        log(f"[bench] zero-change stride: {floor['stride_us']:.1f} us; per launch "
            + ", ".join(f"{k} {v:.2f} us" for k, v in floor["kernels_us"].items()))

    # ---- GPU full recompute: reset + full window through the same kernels ----
    full = []
    if spec is not None:       # every point of the last window in one step
        last_pts = torch.cat(dev[first + W + K - spec.window:first + W + K]).contiguous()
        full_step = lambda: eng.step_points(last_pts)
    else:
        full_step = lambda: eng.step(*dev[W + K], sorted=SORTED)
    for _ in range(0 if args.no_full else 5):
        eng.reset()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        full_step()
        b.record(stream)
        torch.cuda.synchronize()
        full.append(a.elapsed_time(b))
    full_ms = statistics.median(full) if full else None
    eng.close()

    # context: the vendor library's dense recompute of the same layers
    dense_ms = None
    if not args.no_dense and spec is None and not neck and not any(l.sub for l in wl.layers):
        try:
            dense_ms = dense_torch_ms(wl, ws, [S.canvas(strides[W + K], wl.H, wl.W, wl.C0)])
            log(f"[bench] dense recompute with torch conv2d: {dense_ms * 1e3:.1f} us per pass "
                f"({dense_ms / ms_per_step:.1f}x the delta stride)")
        except Exception as exc:  # context only: never fail the bench line for it
            log(f"[bench] dense torch recompute skipped: {exc}")

    # the whole stride against its own roofline (detection + every layer), for
    # the pillar workloads; points mode adds the feature net, which this model
    # does not price
    sroof = None
    if spec is None and not neck:
        cgbs = copy_bandwidth()
        sroof = stride_roofline(wl, act_in, pairs, K, float(np.mean([len(s.idx) for s in strides[1 + W:]])),
                                ms_per_step * 1e3, cgbs)
        log(f"[bench] stride roofline: {sroof['t_roof_us_spec']:.1f} us at 8 TB/s ({100 * sroof['frac_spec']:.1f} %), "
            f"{sroof['t_roof_us_copy']:.1f} us at the measured copy bandwidth {cgbs:.0f} GB/s "
            f"({100 * sroof['frac_copy']:.1f} %)")

    cpu = None
    if not args.no_cpu:
        try:
            log(f"[bench] CPU oracle baseline (budget {args.cpu_seconds:.0f} s)")
            if spec is not None:
                cpu = cpu_baseline_points(wl, ws, spec, pw, strides, first + W, args.cpu_seconds)
            else:
                cpu = cpu_baseline(wl, ws, strides, 1 + W, args.cpu_seconds, neck)
        except Exception as exc:  # the oracle is optional for the GPU number
            log(f"[bench] CPU baseline skipped: {exc}")

    srt = sorted(per_stride)
    line = {
        "metric": METRIC, "value": value, "unit": "updates/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}", "grid": f"{wl.W}x{wl.H}", "C0": wl.C0,
                   "detection": "one launch (sorted pillar lists)" if SORTED else "two passes",
                   "layers": [f"{l.cin}->{l.cout} s{l.stride}{' relu' if l.relu else ''}"
                              f"{' submanifold' if l.sub else (' sparse' if any(x.sub for x in wl.layers) else '')}"
                              for l in wl.layers],
                   "neck": [f"up(layer {u.src}) {wl.layers[u.src - 1].cout}->{u.cout} x{u.stride}" for u in neck],
                   "strides": "full window + warmup untimed, then the timed delta strides",
                   **({"mean_points": float(np.mean([len(b) for b in strides[first + W:]])),
                       "pillar_feature_net": f"9 -> {wl.C0}, N = {spec.max_points}, window {spec.window} strides"}
                      if spec is not None else
                      {"mean_pillars": float(np.mean([len(s.idx) for s in strides[1 + W:]]))}),
                   "mean_active": [a / K for a in act_in]},
        # per-stride latency from a second pass with an event after every stride
        "latency_ms": {"mean": statistics.fmean(per_stride), "p50": srt[len(srt) // 2],
                       "p99": srt[min(len(srt) - 1, int(0.99 * len(srt)))], "max": srt[-1],
                       "over_10ms_frac": sum(1 for x in per_stride if x > 10.0) / K},
        "alg_tflops": sum(2.0 * l.cin * l.cout * pairs[i + 1] for i, l in enumerate(wl.layers)) /
                      (wall_ms / 1e3) / 1e12,
        "full_recompute_ms": full_ms,
        "dense_torch_ms": dense_ms,
        "speedup_vs_dense_torch": dense_ms / ms_per_step if dense_ms else None,
        # the same launch chain on strides that change nothing (points mode:
        # strides without new points, so only the expiring points change)
        "zero_change_floor": floor,
        "speedup_vs_full_recompute": full_ms / ms_per_step if full_ms else None,
        "kernels": {n: {"launches": k["launches"], "avg_us": k["ms"] / k["launches"] * 1e3}
                    for n, k in kernels.items()},
        # Table III's split: each backbone block's kernels per stride
        "blocks_us": blocks,
        "roofline": roofline,
        "stride_roofline": sroof,
        # context only: the paper's own figures, other hardware and real data
        "paper_context": PAPER_CONTEXT,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
