"""CPU oracle of the incremental pillar feature net -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this module; the GPU library shares no code with it.

What the pillar feature net computes (SSCATeR, arXiv 2512.08557, Sec. III-B
and Alg. 1, PFN part), written here from its definition, for one window:

* every point of the window (the last ``window`` strides' batches) falls into
  the pillar (grid cell) under it; points outside the grid belong to none;
* each point is decorated to D = 9 values: x, y, z, intensity, the offsets
  x_p, y_p of the point from its pillar's centre, and the offsets x_c, y_c,
  z_c of the point from the arithmetic mean of its pillar's points;
* a pointwise linear layer (batch norm folded to the identity, no bias) maps
  the 9 values to C0 channels, then ReLU, then the maximum over the pillar's
  points gives the pillar's feature vector.  Zero padding up to N points adds
  all-zero rows after the ReLU, which the maximum of non-negative values
  ignores, so it is left out here;
* a cell without points has no pillar (an all-zero feature row).

The change map of a stride is event based (Alg. 1): a pillar is changed when
a point is inserted into it (the new stride's batch) or removed from it (the
batch that leaves the window).

Binning decides an integer from floating point, so it is done in float32
exactly as the device does it: column = floor((x - x_min) * inv_res) with
inv_res = float32(1 / res), every operation rounded to float32; a point is in
the grid when 0 <= (x - x_min) * inv_res < W (and the same for y and H).
Everything else is float64.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np


def inv_res_f32(res: float) -> np.float32:
    """1 / res rounded to float32 (the device takes the same value)."""
    return np.float32(1.0) / np.float32(res)


def bin_points(points: np.ndarray, H: int, W: int, x_min: float, y_min: float, res: float) -> np.ndarray:
    """Cell index r*W + c of every point, or -1 outside the grid (float32 decision)."""
    p = np.asarray(points, dtype=np.float32).reshape(-1, 4)
    inv = inv_res_f32(res)
    with np.errstate(invalid="ignore"):
        fx = (p[:, 0] - np.float32(x_min)) * inv
        fy = (p[:, 1] - np.float32(y_min)) * inv
        ok = (fx >= 0) & (fx < np.float32(W)) & (fy >= 0) & (fy < np.float32(H))
    col = np.floor(np.where(ok, fx, 0)).astype(np.int64)
    row = np.floor(np.where(ok, fy, 0)).astype(np.int64)
    return np.where(ok, row * W + col, -1)


def decorate(pts: np.ndarray, cell: int, W: int, x_min: float, y_min: float, res: float) -> np.ndarray:
    """The D = 9 decorated values of a pillar's points [n, 4] -> [n, 9] (float64)."""
    p = np.asarray(pts, dtype=np.float64)
    r, c = divmod(int(cell), W)
    xc = x_min + (c + 0.5) * res          # pillar centre
    yc = y_min + (r + 0.5) * res
    mean = p[:, :3].mean(axis=0)          # arithmetic mean of the pillar's points
    return np.stack([p[:, 0], p[:, 1], p[:, 2], p[:, 3],
                     p[:, 0] - xc, p[:, 1] - yc,
                     p[:, 0] - mean[0], p[:, 1] - mean[1], p[:, 2] - mean[2]], axis=1)


def pillar_feature(pts: np.ndarray, cell: int, W: int, x_min: float, y_min: float, res: float,
                   w: np.ndarray) -> np.ndarray:
    """max over the pillar's points of ReLU(w @ decoration), float64 [C0]."""
    d = decorate(pts, cell, W, x_min, y_min, res)
    y = d @ np.asarray(w, dtype=np.float64).T           # [n, C0]
    return np.maximum(y, 0.0).max(axis=0)


def canvas(window_points: Sequence[np.ndarray], H: int, W: int, x_min: float, y_min: float, res: float,
           w: np.ndarray) -> np.ndarray:
    """Dense [H, W, C0] float64 pseudo-image of one window's points."""
    C0 = np.asarray(w).shape[0]
    out = np.zeros((H * W, C0), dtype=np.float64)
    pts = np.concatenate([np.asarray(b, dtype=np.float32).reshape(-1, 4) for b in window_points]) \
        if len(window_points) else np.zeros((0, 4), np.float32)
    cells = bin_points(pts, H, W, x_min, y_min, res)
    keep = cells >= 0
    pts, cells = pts[keep], cells[keep]
    order = np.argsort(cells, kind="stable")
    pts, cells = pts[order], cells[order]
    uniq, start = np.unique(cells, return_index=True)
    stop = np.append(start[1:], cells.size)
    for q, a, b in zip(uniq, start, stop):
        out[q] = pillar_feature(pts[a:b], int(q), W, x_min, y_min, res, w)
    return out.reshape(H, W, C0)


def changed_cells(new_batch: np.ndarray, old_batch, H: int, W: int, x_min: float, y_min: float,
                  res: float) -> np.ndarray:
    """Event-based A_0: sorted in-grid cells that gain a point (new batch) or
    lose one (the batch leaving the window, or None)."""
    parts = [bin_points(new_batch, H, W, x_min, y_min, res)]
    if old_batch is not None:
        parts.append(bin_points(old_batch, H, W, x_min, y_min, res))
    c = np.concatenate(parts)
    return np.unique(c[c >= 0]).astype(np.int64)


def occupancy(window_points: Sequence[np.ndarray], H: int, W: int, x_min: float, y_min: float,
              res: float) -> Tuple[np.ndarray, np.ndarray]:
    """Cells with at least one point in the window, and their point counts."""
    pts = np.concatenate([np.asarray(b, dtype=np.float32).reshape(-1, 4) for b in window_points])
    cells = bin_points(pts, H, W, x_min, y_min, res)
    cells = cells[cells >= 0]
    return np.unique(cells, return_counts=True)
