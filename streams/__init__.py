"""Seeded synthetic pillar streams for the delta-scatter backbone.

This module only *generates inputs*: the occupied bird's-eye-view cells of a
synthetic LiDAR scene, the per-stride pillar lists (cell index + feature
vector) of a sliding window that sweeps one azimuth sector per stride, and the
random convolution weights.  It holds none of the convolution method's
arithmetic and is imported by both the CPU oracle's tests and the GPU path's
tests and benchmark.

Paper context (SSCATeR, arXiv 2512.08557):
  * pillar grid of 0.16 m cells, pseudo-image of C=64 channels, up to P=12,000
    pillars (Sec. III-B);
  * 100 ms window advanced in 10 ms strides, each stride corresponding to a
    36 degree wedge of a rotating sensor (Sec. I; Sec. II-C);
  * backbone of three Block(S, L, F) with S=2, L=4/6/6, F=64/128/256
    (Sec. III-B, backbone paragraph).
The real drone datasets are not available; these seeded scenes stand in for
them (the recipe is documented in the repository's design notes).

Conventions:
  * grid of H rows (y) by W columns (x); a cell index is p = r*W + c;
  * features are NHWC float32 (or bfloat16 bit patterns held as uint16);
  * every stride's pillar list is the full occupied set, sorted by cell index;
    pillars that were not refreshed carry bit-identical features;
  * stride 0 is the initial full window; strides 1..n are the delta strides and
    stride s sweeps sector (s-1) mod n_sectors.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Iterator, List, Optional, Tuple

import numpy as np

SCENE_SEED = 2512
WEIGHT_SEED = 8557

__all__ = [
    "LayerSpec", "Workload", "workload", "WORKLOADS", "weights", "make_stream", "UpSpec", "neck", "neck_weights",
    "Stream", "Stride", "round_to_bf16_bits", "bf16_bits_to_f32", "out_shape",
    "cell_azimuth_sector", "SWEEP_CIN", "SWEEP_COUT", "PfnSpec", "pfn_spec", "pfn_weights",
    "make_point_stream",
]


# --------------------------------------------------------------------------
# workload descriptions
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class LayerSpec:
    cin: int
    cout: int
    stride: int
    relu: bool
    sub: bool = False       # submanifold convolution (sparse workloads)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    H: int
    W: int
    C0: int
    dtype: str              # "f32" or "bf16"
    layers: Tuple[LayerSpec, ...]
    n_strides: int          # delta strides after the initial full window
    max_pillars: int
    description: str


def _block(cin: int, f: int, n: int) -> List[LayerSpec]:
    """Block(S=2, L=n, F=f): one stride-2 conv then n-1 stride-1 convs, ReLU."""
    out = [LayerSpec(cin, f, 2, True)]
    out += [LayerSpec(f, f, 1, True) for _ in range(n - 1)]
    return out


_BACKBONE = tuple(_block(64, 64, 4) + _block(64, 128, 6) + _block(128, 256, 6))


def _sparse_block(cin: int, f: int, n: int) -> List[LayerSpec]:
    """Sparse PointPillars block: a regular sparse stride-2 conv, then n-1
    submanifold convs (Sec. III-E)."""
    return [LayerSpec(cin, f, 2, True)] + [LayerSpec(f, f, 1, True, True) for _ in range(n - 1)]


_SPARSE_BACKBONE = tuple(_sparse_block(64, 64, 4) + _sparse_block(64, 128, 6) + _sparse_block(128, 256, 6))

# Single-layer channel sweep at the paper's drone-LiDAR sparsity: one 3x3
# stride-1 conv, Cin in {16, 32, 64, 128} x Cout in {8, 16, 32, 64, 128}, on a
# 504 x 504 grid of 0.16 m pillars (the shapes of the single-layer timing
# tables, Sec. IV-B, Tables I and II).
SWEEP_CIN = (16, 32, 64, 128)
SWEEP_COUT = (8, 16, 32, 64, 128)


def _sweep_workloads() -> dict:
    out = {}
    for ci in SWEEP_CIN:
        for co in SWEEP_COUT:
            name = f"l{ci}x{co}"
            out[name] = Workload(name, 504, 504, ci, "f32", (LayerSpec(ci, co, 1, True),), 100, 4096,
                                 f"single 3x3 s1 conv {ci}->{co} (ReLU), 504x504 forward-looking drone scan")
    return out


WORKLOADS = {
    "c1": Workload("c1", 64, 64, 16, "f32", (LayerSpec(16, 16, 1, False),), 10, 4096,
                   "single 3x3 s1 conv 16->16, 64x64 grid, no ReLU"),
    "c2": Workload("c2", 496, 432, 64, "f32", tuple(_block(64, 64, 4)), 100, 16000,
                   "PointPillars block 1 (s2 + 3 x s1, 64 ch, ReLU) on 432x496"),
    "c3": Workload("c3", 496, 432, 64, "f32", _BACKBONE, 100, 16000,
                   "3-block PointPillars backbone (64/128/256 ch), fp32, 432x496"),
    "c4": Workload("c4", 496, 432, 64, "bf16", _BACKBONE, 200, 16000,
                   "3-block backbone in bf16 (fp32 accumulate), 18 deg strides + 1% toggles"),
    "c5": Workload("c5", 1024, 1024, 64, "f32", tuple(_block(64, 64, 4)), 100, 48000,
                   "1024x1024 drone grid, block 1, 4 concurrent streams"),
    **_sweep_workloads(),
    # sparse backbones on the toggling 432x496 stream (18 degree sectors, 60
    # pillars appear and 60 vanish per stride): the active sets move
    "s2": Workload("s2", 496, 432, 64, "f32", tuple(_sparse_block(64, 64, 4)), 100, 16000,
                   "sparse block 1 (regular s2 + 3 submanifold, 64 ch) on 432x496 with toggles"),
    "s3": Workload("s3", 496, 432, 64, "f32", _SPARSE_BACKBONE, 100, 16000,
                   "sparse 3-block backbone (regular + submanifold), fp32, 432x496 with toggles"),
    "s4": Workload("s4", 496, 432, 64, "bf16", _SPARSE_BACKBONE, 200, 16000,
                   "sparse 3-block backbone in bf16, 18 deg strides + 1% toggles"),
    "p2": Workload("p2", 504, 504, 64, "f32", tuple(_block(64, 64, 4)), 100, 254016,
                   "points of the 504x504 drone scan -> incremental pillar feature net (9 -> 64) -> "
                   "PointPillars block 1"),
}


@dataclasses.dataclass(frozen=True)
class PfnSpec:
    """Pillar feature net front end (Sec. III-B): the grid corner in metres,
    the pillar edge, N points per pillar at most, the window in strides, and a
    bound on the points of one stride."""
    x_min: float
    y_min: float
    res: float
    max_points: int
    window: int
    max_new_points: int


# 504 x 504 pillars of 0.16 m centred on the sensor; N = 100 (Sec. III-B);
# 100 ms windows of 10 ms strides; every beam of a stride may return.
PFNS = {"p2": PfnSpec(-40.32, -40.32, 0.16, 100, 10, 2400)}


def pfn_spec(name: str) -> PfnSpec:
    return PFNS[name]


def pfn_weights(name: str) -> np.ndarray:
    """[C0, 9] float32 weights of the pillar feature net's linear layer,
    He-normal N(0, 2/9); batch norm folded to the identity, no bias."""
    wl = workload(name)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence((WEIGHT_SEED, 7, 1000))))
    return (rng.standard_normal((wl.C0, 9)) * math.sqrt(2.0 / 9.0)).astype(np.float32)


def _family(name: str) -> int:
    """Seed family of a workload: c1..c5 -> 1..5, the single-layer sweep -> 6,
    the point-level workloads (pillar feature net in front) -> 7."""
    if name.startswith("l"):
        return 6
    if name.startswith("p"):
        return 7
    if name.startswith("s"):
        return 4            # the toggling stream of c4
    return int(name[1])


def workload(name: str) -> Workload:
    return WORKLOADS[name]


@dataclasses.dataclass(frozen=True)
class UpSpec:
    """One upsampler of the neck: transposed conv with kernel = stride on the
    output of backbone layer `src` (1-based), then ReLU."""
    src: int
    cout: int
    stride: int
    relu: bool


# PointPillars neck on the 3-block backbone: every block output upsampled to
# the first block's 248x216 grid with 128 channels, concatenated (384).
_NECK = (UpSpec(4, 128, 1, True), UpSpec(10, 128, 2, True), UpSpec(16, 128, 4, True))
NECKS = {"c3": _NECK, "c4": _NECK}


def neck(name: str) -> Tuple[UpSpec, ...]:
    return NECKS.get(name, ())


def neck_weights(name: str) -> List[np.ndarray]:
    """Per-upsampler [cin, cout, s, s] float32 weights, He-normal N(0, 2/cin)
    (each output cell sums cin products); bf16-representable for bf16
    workloads."""
    wl = workload(name)
    out = []
    for u, up in enumerate(neck(name)):
        cin = wl.layers[up.src - 1].cout
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence((WEIGHT_SEED, 2, 100 + u))))
        w = (rng.standard_normal((cin, up.cout, up.stride, up.stride)) * math.sqrt(2.0 / cin)).astype(np.float32)
        if wl.dtype == "bf16":
            w = bf16_bits_to_f32(round_to_bf16_bits(w)).reshape(w.shape)
        out.append(np.ascontiguousarray(w))
    return out


def out_shape(H: int, W: int, stride: int) -> Tuple[int, int]:
    """Output grid of a 3x3 conv with zero padding 1: floor((H + 2 - 3)/s) + 1."""
    return (H - 1) // stride + 1, (W - 1) // stride + 1


# --------------------------------------------------------------------------
# bfloat16 bit handling (input preparation only)
# --------------------------------------------------------------------------
def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------
def weights(name: str) -> List[np.ndarray]:
    """Per-layer OIHW float32 weights.

    c1: N(0, 1/144).  c2..c5 and the sweep: He-normal N(0, 2/(9*cin)).  c2/c3/c4 share the
    432x496 backbone family, so c2's four layers equal c3's first four; c4 is
    c3 rounded to bfloat16 (returned as float32 values that are exactly
    representable in bfloat16).
    """
    wl = workload(name)
    family = {"c1": 1, "c2": 2, "c3": 2, "c4": 2, "c5": 5, "s2": 2, "s3": 2, "s4": 2}.get(name, 6)
    out = []
    for li, ls in enumerate(wl.layers):
        key = (WEIGHT_SEED, family, li) if family != 6 else (WEIGHT_SEED, family, ls.cin, ls.cout)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))
        std = (1.0 / 12.0) if name == "c1" else math.sqrt(2.0 / (9.0 * ls.cin))
        w = (rng.standard_normal((ls.cout, ls.cin, 3, 3)) * std).astype(np.float32)
        if wl.dtype == "bf16":
            w = bf16_bits_to_f32(round_to_bf16_bits(w)).reshape(w.shape)
        out.append(np.ascontiguousarray(w))
    return out


# --------------------------------------------------------------------------
# scene geometry helpers
# --------------------------------------------------------------------------
def cell_azimuth_sector(H: int, W: int, n_sectors: int) -> np.ndarray:
    """Sector id of every cell: azimuth of the cell centre about the grid
    centre, in [0, 360) degrees, split into n_sectors half-open wedges."""
    r = np.arange(H, dtype=np.float64)[:, None] + 0.5 - H / 2.0
    c = np.arange(W, dtype=np.float64)[None, :] + 0.5 - W / 2.0
    az = np.mod(np.arctan2(r, c), 2.0 * np.pi)
    sec = np.floor(az / (2.0 * np.pi / n_sectors)).astype(np.int64)
    return np.minimum(sec, n_sectors - 1).reshape(-1)


def _metres_to_cells(x: np.ndarray, y: np.ndarray, H: int, W: int, res: float) -> np.ndarray:
    """Sensor-centred metric coordinates -> unique in-grid cell indices."""
    c = np.floor(x / res + W / 2.0).astype(np.int64)
    r = np.floor(y / res + H / 2.0).astype(np.int64)
    ok = (r >= 0) & (r < H) & (c >= 0) & (c < W)
    return np.unique(r[ok] * W + c[ok])


def _rings(H: int, W: int, res: float, n_rings: int, r0: float, r1: float) -> np.ndarray:
    radii = r0 * (r1 / r0) ** (np.arange(n_rings) / max(n_rings - 1, 1))
    cells = []
    for rad in radii:
        n = int(math.ceil(2.0 * math.pi * rad / res))  # azimuth step <= res / r
        th = np.arange(n) * (2.0 * math.pi / n)
        cells.append(_metres_to_cells(rad * np.cos(th), rad * np.sin(th), H, W, res))
    return np.unique(np.concatenate(cells))


def _box_perimeter(cx, cy, a, b, yaw, H, W, res) -> np.ndarray:
    """Cells under the perimeter of an a x b rectangle centred at (cx, cy)."""
    step = res / 4.0
    pts = []
    ca, sa = math.cos(yaw), math.sin(yaw)
    corners = [(-a / 2, -b / 2), (a / 2, -b / 2), (a / 2, b / 2), (-a / 2, b / 2)]
    for k in range(4):
        (x0, y0), (x1, y1) = corners[k], corners[(k + 1) % 4]
        n = max(2, int(math.ceil(math.hypot(x1 - x0, y1 - y0) / step)) + 1)
        t = np.linspace(0.0, 1.0, n)
        lx, ly = x0 + (x1 - x0) * t, y0 + (y1 - y0) * t
        pts.append((cx + ca * lx - sa * ly, cy + sa * lx + ca * ly))
    xs = np.concatenate([p[0] for p in pts])
    ys = np.concatenate([p[1] for p in pts])
    return _metres_to_cells(xs, ys, H, W, res)


# Forward-looking drone LiDAR with a non-repeating rosette scan (the stand-in
# for the paper's drone datasets, Sec. III-A): 24,000 emitted beams per
# 100 ms, of which a minority return; active and changed cells per 10 ms stride
# come out near the means the paper reports for its 504 x 504 grid (1,781
# active, 483 changed, 27 %; Sec. IV-A).
_SCAN_BEAMS = 2400              # emitted beams per 10 ms stride
_SCAN_PRISM_HZ = (457.3, -319.9)  # two counter-rotating prisms ...
_SCAN_PRISM_DEG = 15.0          # ... each deflecting by 15 degrees: a 60 degree cone
_SCAN_ALT_M = 10.0              # sensor height above flat ground
_SCAN_PITCH_DEG = 45.0          # boresight below the horizon
_SCAN_SPEED = 3.0               # forward speed, m/s
_SCAN_X0 = -20.0                # sensor position relative to the grid centre at t = 0, m
_SCAN_RETURN = 0.12             # mean return probability of a beam that reaches the ground
_SCAN_RETURN_SWING = 0.4        # +-40 % over a 40-stride period (surfaces come and go)


def _rosette_returns(rng: np.random.Generator, s: int):
    """Ground hits (x, y) in metres, sensor-grid frame, of the beams of 10 ms
    stride s that return (s may be negative)."""
    T = 0.01
    t = s * T + np.arange(_SCAN_BEAMS) * (T / _SCAN_BEAMS)
    d = math.radians(_SCAN_PRISM_DEG)
    w1, w2 = 2.0 * math.pi * _SCAN_PRISM_HZ[0], 2.0 * math.pi * _SCAN_PRISM_HZ[1]
    az = d * (np.cos(w1 * t) + np.cos(w2 * t))           # beam offset from the boresight
    el = -math.radians(_SCAN_PITCH_DEG) + d * (np.sin(w1 * t) + np.sin(w2 * t))
    p = _SCAN_RETURN * (1.0 + _SCAN_RETURN_SWING * math.sin(2.0 * math.pi * s / 40.0))
    keep = (el < -1e-3) & (rng.random(_SCAN_BEAMS) < p)   # below the horizon, and returned
    rng_m = _SCAN_ALT_M / np.tan(-el[keep])               # ground range
    x = rng_m * np.cos(az[keep]) + _SCAN_X0 + _SCAN_SPEED * t[keep]
    y = rng_m * np.sin(az[keep])
    return x, y


def _rosette_hits(rng: np.random.Generator, s: int, H: int, W: int, res: float) -> np.ndarray:
    """Unique cells hit by the returns of 10 ms stride s (s may be negative)."""
    x, y = _rosette_returns(rng, s)
    return _metres_to_cells(x, y, H, W, res)


def make_point_stream(name: str, seed: int = SCENE_SEED, n_strides: Optional[int] = None) -> List[np.ndarray]:
    """Point batches of the drone scan for strides -(window-1)..n: float32
    [n_points, 4] = (x, y, z, intensity), metres in the grid frame.  The first
    window-1 batches and batch 0 build the first full window (the
    initialisation of Alg. 1); batches 1..n are the delta strides.  The ground
    hits are those of the sweep stream's scan; z is ground roughness N(0, 5 cm)
    and the intensity U(0, 1)."""
    wl = workload(name)
    spec = pfn_spec(name)
    n = wl.n_strides if n_strides is None else n_strides
    scan = np.random.Generator(np.random.PCG64(np.random.SeedSequence((seed, 6, 0))))
    attr = np.random.Generator(np.random.PCG64(np.random.SeedSequence((seed, 7, 0))))
    out = []
    for s in range(-(spec.window - 1), n + 1):
        x, y = _rosette_returns(scan, s)
        z = 0.05 * attr.standard_normal(x.size)
        r = attr.random(x.size)
        out.append(np.ascontiguousarray(np.stack([x, y, z, r], axis=1).astype(np.float32)))
    return out


def _thin(cells: np.ndarray, target: int, rng: np.random.Generator) -> np.ndarray:
    if cells.size <= target:
        return cells
    keep = rng.random(cells.size) < (target / cells.size)
    return cells[keep]


# --------------------------------------------------------------------------
# streams
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Stride:
    index: int               # 0 = initial full window
    idx: np.ndarray          # int32 [P], sorted, unique
    feats: np.ndarray        # float32 [P, C0] or uint16 (bf16 bits) [P, C0]


class Stream:
    """Iterator over the strides of one synthetic sweep stream."""

    def __init__(self, name: str, seed: int = SCENE_SEED, n_strides: Optional[int] = None):
        self.wl = workload(name)
        self.name = name
        self.seed = seed
        self.n_strides = self.wl.n_strides if n_strides is None else n_strides
        wl = self.wl
        self.HW = wl.H * wl.W
        self._bf16 = wl.dtype == "bf16"
        scene_rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence((seed, 0, 0))))
        self.moving: List[dict] = []
        if name == "c1":
            occ = np.sort(scene_rng.choice(self.HW, size=400, replace=False))
            self.n_sectors = 10
        elif name in ("c2", "c3", "c4", "s2", "s3", "s4"):
            occ = self._scene_432x496(scene_rng)
            self.n_sectors = 10 if name in ("c2", "c3") else 20
        elif name == "c5":
            occ = self._scene_1024(scene_rng)
            self.n_sectors = 20
        elif _family(name) == 6:
            occ = self._scene_drone_scan(seed)
            self.n_sectors = 1
        else:
            raise ValueError(name)
        self.sector = cell_azimuth_sector(wl.H, wl.W, self.n_sectors)
        self.occ = np.zeros(self.HW, dtype=bool)
        self.occ[occ] = True
        self.static_occ = self.occ.copy()
        if name == "c5":
            self.static_occ[:] = False
            self.static_occ[self._c5_static] = True
        # dense feature store (float32); bf16 streams round on the way in
        self.feat = np.zeros((self.HW, wl.C0), dtype=np.float32)
        init_rng = self._stride_rng(0)
        self._fill(np.flatnonzero(self.occ), init_rng)
        self.occupied_count0 = int(self.occ.sum())

    # -- scenes ------------------------------------------------------------
    def _scene_432x496(self, rng) -> np.ndarray:
        H, W, res = 496, 432, 0.16
        # sensor at the grid centre; ground rings at geometric ranges 2..35 m
        ground = _rings(H, W, res, 24, 2.0, 35.0)
        boxes = []
        for _ in range(20):
            a, b = rng.uniform(0.6, 4.5, size=2)
            cx = rng.uniform(-W * res / 2 + 3, W * res / 2 - 3)
            cy = rng.uniform(-H * res / 2 + 3, H * res / 2 - 3)
            boxes.append(_box_perimeter(cx, cy, a, b, rng.uniform(0, math.pi), H, W, res))
        cells = np.unique(np.concatenate([ground] + boxes))
        return np.sort(_thin(cells, 12000, rng))

    def _scene_drone_scan(self, seed: int) -> np.ndarray:
        """Cells hit in every stride -9..n (the window of stride s is the ten
        strides s-9..s); the initial window's occupied cells."""
        H, W, res = self.wl.H, self.wl.W, 0.16
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence((seed, 6, 0))))
        self._hits = [_rosette_hits(rng, s, H, W, res) for s in range(-9, self.n_strides + 1)]
        self._wcount = np.zeros(H * W, dtype=np.int16)     # strides of the window that hit each cell
        for h in self._hits[:10]:
            self._wcount[h] += 1
        return np.flatnonzero(self._wcount)

    def _scene_1024(self, rng) -> np.ndarray:
        H, W, res = 1024, 1024, 0.1
        ground = _rings(H, W, res, 40, 2.0, 70.0)
        parts = [ground]
        for _ in range(10):
            a, b = rng.uniform(5.0, 20.0, size=2)
            cx, cy = rng.uniform(-45, 45, size=2)
            parts.append(_box_perimeter(cx, cy, a, b, rng.uniform(0, math.pi), H, W, res))
        static = np.unique(np.concatenate(parts))
        static = _thin(static, 34000, rng)
        self._c5_static = static
        for _ in range(50):
            a, b = rng.uniform(0.5, 5.0, size=2)
            self.moving.append(dict(
                x=float(rng.uniform(-45, 45)), y=float(rng.uniform(-45, 45)), a=float(a), b=float(b),
                yaw=float(rng.uniform(0, math.pi)), v=float(rng.uniform(0, 15)),
                hd=float(rng.uniform(0, 2 * math.pi)), cells=np.zeros(0, dtype=np.int64)))
        self._c5_res = res
        dyn = []
        for bx in self.moving:
            bx["cells"] = _box_perimeter(bx["x"], bx["y"], bx["a"], bx["b"], bx["yaw"], H, W, res)
            dyn.append(bx["cells"])
        return np.unique(np.concatenate([static] + dyn))

    # -- per-stride randomness ----------------------------------------------
    def _stride_rng(self, s: int) -> np.random.Generator:
        cfg = _family(self.name)
        return np.random.Generator(np.random.PCG64(np.random.SeedSequence((self.seed, cfg, s + 1))))

    def _fill(self, cells: np.ndarray, rng) -> None:
        if cells.size == 0:
            return
        v = rng.standard_normal((cells.size, self.wl.C0), dtype=np.float32)
        if self._bf16:
            v = bf16_bits_to_f32(round_to_bf16_bits(v)).reshape(v.shape)
        self.feat[cells] = v

    # -- stride evolution ----------------------------------------------------
    def _advance(self, s: int) -> None:
        rng = self._stride_rng(s)
        sec = (s - 1) % self.n_sectors
        in_sec = self.sector == sec
        if self.name == "c1":
            occ_sec = np.flatnonzero(self.occ & in_sec)
            nref = min(40, occ_sec.size)
            if nref:
                self._fill(np.sort(rng.choice(occ_sec, size=nref, replace=False)), rng)
            sec_cells = np.flatnonzero(in_sec)
            tog = np.sort(rng.choice(sec_cells, size=min(10, sec_cells.size), replace=False))
            on = tog[~self.occ[tog]]
            off = tog[self.occ[tog]]
            self.occ[off] = False
            self.feat[off] = 0.0
            self.occ[on] = True
            self._fill(on, rng)
        elif self.name in ("c2", "c3"):
            self._fill(np.flatnonzero(self.occ & in_sec), rng)
        elif _family(self.name) == 6:
            # a cell changes when the new stride hits it or the expiring one
            # (stride s-10) did; it stays occupied while any stride of the
            # window hits it, with a fresh feature vector
            new, old = self._hits[s + 9], self._hits[s - 1]
            self._wcount[new] += 1
            self._wcount[old] -= 1
            changed = np.union1d(new, old)
            live = self._wcount[changed] > 0
            off, on = changed[~live], changed[live]
            self.occ[off] = False
            self.feat[off] = 0.0
            self.occ[on] = True
            self._fill(on, rng)
        elif self.name in ("c4", "s2", "s3", "s4"):
            self._fill(np.flatnonzero(self.occ & in_sec), rng)
            occ_sec = np.flatnonzero(self.occ & in_sec)
            emp_sec = np.flatnonzero(~self.occ & in_sec)
            n_off = min(60, occ_sec.size)
            n_on = min(60, emp_sec.size)
            off = np.sort(rng.choice(occ_sec, size=n_off, replace=False)) if n_off else occ_sec[:0]
            on = np.sort(rng.choice(emp_sec, size=n_on, replace=False)) if n_on else emp_sec[:0]
            self.occ[off] = False
            self.feat[off] = 0.0
            self.occ[on] = True
            self._fill(on, rng)
        elif self.name == "c5":
            H, W, res = self.wl.H, self.wl.W, self._c5_res
            dt = 0.005  # 1/20 of a 10 Hz revolution
            moved_on, moved_off = [], []
            for bx in self.moving:
                bx["x"] += bx["v"] * dt * math.cos(bx["hd"])
                bx["y"] += bx["v"] * dt * math.sin(bx["hd"])
                c = int(math.floor(bx["x"] / res + W / 2.0))
                r = int(math.floor(bx["y"] / res + H / 2.0))
                if 0 <= r < H and 0 <= c < W and self.sector[r * W + c] == sec:
                    new = _box_perimeter(bx["x"], bx["y"], bx["a"], bx["b"], bx["yaw"], H, W, res)
                    moved_off.append(np.setdiff1d(bx["cells"], new))
                    moved_on.append(np.setdiff1d(new, bx["cells"]))
                    bx["cells"] = new
            # refresh everything occupied in the sector first
            self._fill(np.flatnonzero(self.occ & in_sec), rng)
            if moved_off:
                off = np.unique(np.concatenate(moved_off))
                still = np.zeros(self.HW, dtype=bool)
                still[self.static_occ] = True
                for bx in self.moving:
                    still[bx["cells"]] = True
                off = off[~still[off]]
                self.occ[off] = False
                self.feat[off] = 0.0
            if moved_on:
                on = np.unique(np.concatenate(moved_on))
                on = on[~self.occ[on]]
                self.occ[on] = True
                self._fill(on, rng)

    def _emit(self, s: int) -> Stride:
        idx = np.flatnonzero(self.occ).astype(np.int32)
        f = self.feat[idx]
        if self._bf16:
            f = round_to_bf16_bits(f).reshape(f.shape)
        return Stride(s, idx, np.ascontiguousarray(f))

    def __iter__(self) -> Iterator[Stride]:
        yield self._emit(0)
        for s in range(1, self.n_strides + 1):
            self._advance(s)
            yield self._emit(s)


def make_stream(name: str, seed: int = SCENE_SEED, n_strides: Optional[int] = None) -> List[Stride]:
    """All strides of a stream (stride 0 = full window), materialised."""
    return list(Stream(name, seed, n_strides))


def canvas(stride: Stride, H: int, W: int, C0: int) -> np.ndarray:
    """Dense NHWC canvas of one stride (float32, or uint16 bf16 bits)."""
    out = np.zeros((H * W, C0), dtype=stride.feats.dtype)
    out[stride.idx] = stride.feats
    return out.reshape(H, W, C0)
