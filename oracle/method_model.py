"""Float64 CPU model of the delta-scatter method -- TEST INFRASTRUCTURE ONLY.

This follows the paper's method step by step, in its order and notation, so
that the claim "recycled maps equal recomputation" can be checked on the CPU
independently of any GPU code (SSCATeR, arXiv 2512.08557):

1. Input change map: a cell is changed when its pillar features differ from
   the previous window (Sec. III-B; Alg. 1, PFN part).
2. For each layer, every changed input site (i, j) scatters its feature delta
   (I_curr - I_prev) through every kernel tap (m, n) into the persistent
   output at (i - m + floor(k/2), j - n + floor(k/2)) (Eq. 2, Sec. III-D).
   For stride s the target is ((i - m + 1)/s, (j - n + 1)/s) when both are
   integers, i.e. the transpose of a strided gather.
3. Every output site touched by that scatter is marked changed (Alg. 1,
   backbone part: sites changed by the convolution; for stride > 1 the
   downsampled site under a changed site).  A site whose ReLU output becomes
   zero stays marked (Sec. III-D, ReLU paragraph): marking is structural.
4. The next layer's input delta at a marked site is phi(Z_new) - phi(Z_old)
   (the post-activation value delta); with bf16 storage both terms are the
   stored bf16 maps.

Sizes are small (pure Python loops over the changed sites).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from . import out_extent, round_bf16


class DeltaScatterModel:
    def __init__(self, H: int, W: int, C0: int, layers: Sequence[Tuple[int, int, int, bool]],
                 weights: Sequence[np.ndarray], bf16_storage: bool = False):
        self.layers = [tuple(l) for l in layers]
        self.w = [np.asarray(w, dtype=np.float64) for w in weights]
        self.bf16 = bf16_storage
        self.shapes = [(H, W, C0)]
        h, wd = H, W
        for (cin, cout, s, _r) in self.layers:
            h, wd = out_extent(h, s), out_extent(wd, s)
            self.shapes.append((h, wd, cout))
        self.reset()

    def reset(self) -> None:
        H, W, C0 = self.shapes[0]
        self.x = np.zeros((H, W, C0), dtype=np.float64)
        self.x_bits = None
        self.z = [np.zeros(s, dtype=np.float64) for s in self.shapes[1:]]

    def _phi(self, l: int, z: np.ndarray) -> np.ndarray:
        y = np.maximum(z, 0.0) if self.layers[l][3] else z.copy()
        return round_bf16(y) if self.bf16 else y

    def maps(self) -> List[np.ndarray]:
        """Y_l = phi(Z_l) for every layer (the layer outputs are not stored)."""
        return [self._phi(l, z) for l, z in enumerate(self.z)]

    def step(self, x_new: np.ndarray, x_new_bits: np.ndarray) -> List[np.ndarray]:
        """Advance one window; return the sorted changed lists A_0..A_L."""
        H, W, C0 = self.shapes[0]
        if self.x_bits is None:
            self.x_bits = np.zeros_like(x_new_bits)
        changed = np.any(self.x_bits != x_new_bits, axis=-1).reshape(-1)
        a_prev = np.flatnonzero(changed)
        d_prev = (x_new.reshape(H * W, C0)[a_prev] - self.x.reshape(H * W, C0)[a_prev])
        self.x = np.array(x_new, dtype=np.float64, copy=True)
        self.x_bits = np.array(x_new_bits, copy=True)
        lists = [a_prev]
        for l, (cin, cout, s, _relu) in enumerate(self.layers):
            hin, win, _ = self.shapes[l]
            ho, wo, _ = self.shapes[l + 1]
            wt = self.w[l]
            z = self.z[l]
            touched = set()
            z_old = {}
            for k, p in enumerate(a_prev):
                i, j = divmod(int(p), win)
                for m in range(3):
                    for n in range(3):
                        rn, cn = i - m + 1, j - n + 1
                        if rn % s or cn % s:
                            continue
                        r, c = rn // s, cn // s
                        if not (0 <= r < ho and 0 <= c < wo):
                            continue
                        q = r * wo + c
                        if q not in z_old:
                            z_old[q] = z[r, c].copy()
                        # Eq. 2: O[.] += (I_curr - I_prev) * W[m, n], summed over input channels
                        z[r, c] += wt[:, :, m, n] @ d_prev[k]
                        touched.add(q)
            a_next = np.array(sorted(touched), dtype=np.int64)
            if a_next.size:
                rr, cc = np.divmod(a_next, wo)
                zn = z[rr, cc]
                zo = np.stack([z_old[int(q)] for q in a_next])
                d_next = self._phi(l, zn) - self._phi(l, zo)
            else:
                d_next = np.zeros((0, cout), dtype=np.float64)
            lists.append(a_next)
            a_prev, d_prev = a_next, d_next
        return lists


class DeltaFormModel:
    """Vectorised model of the method for the bf16 storage case, used to
    measure how the form of the delta affects drift against recomputation
    (the delta-form question of the bf16 case).

    Per stride: the input delta is the exact difference of the two canvases;
    for each layer the persistent pre-activation map takes Z += conv(delta)
    (Eq. 2 summed over the taps: the scatter of every changed site, as one
    dense convolution of a map that is zero off the changed sites), kept in
    float32 (`z32`, one rounding per stride) or float64; the stored output is
    bf16(phi(Z)) and the next layer's delta is
      delta="pair":    bf16(phi(Z_new)) - bf16(phi(Z_old)) exactly (the
                       difference of two bf16 values, carried as the pair);
      delta="rounded": that difference rounded to bf16 before the scatter.
    """

    def __init__(self, layers: Sequence[Tuple[int, int, int, bool]], weights: Sequence[np.ndarray],
                 delta: str = "pair", z32: bool = True):
        from . import conv3x3
        assert delta in ("pair", "rounded")
        self._conv = conv3x3
        self.layers = [tuple(l) for l in layers]
        self.w = [np.asarray(w, dtype=np.float64) for w in weights]
        self.delta = delta
        self.z32 = z32
        self.x = None
        self.z = None

    def _phi(self, l: int, z: np.ndarray) -> np.ndarray:
        y = np.maximum(z, 0.0) if self.layers[l][3] else z
        return round_bf16(y)

    def step(self, x_new: np.ndarray) -> List[np.ndarray]:
        """Advance one window (x_new: the canvas's exact values); return the
        stored outputs Y_1..Y_L."""
        x_new = np.asarray(x_new, dtype=np.float64)
        if self.x is None:
            self.x = np.zeros_like(x_new)
        d = x_new - self.x
        self.x = x_new.copy()
        ys = []
        zs = []
        for l, (_ci, _co, s, _r) in enumerate(self.layers):
            if self.delta == "rounded":
                d = round_bf16(d)
            contrib = self._conv(d, self.w[l], s)
            z_old = self.z[l] if self.z is not None else np.zeros_like(contrib)
            z_new = z_old + contrib
            if self.z32:
                z_new = z_new.astype(np.float32).astype(np.float64)
            y_new, y_old = self._phi(l, z_new), self._phi(l, z_old)
            d = y_new - y_old
            zs.append(z_new)
            ys.append(y_new)
        self.z = zs
        return ys
