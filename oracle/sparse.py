"""CPU oracle of the sparse backbone (regular sparse and submanifold
convolutions) -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this module; the GPU library shares no code with it.

The paper's sparse backbone follows Sparse PointPillars: each block starts
with a regular sparse 3x3 convolution and continues with submanifold
convolutions, and SSCATeR is applied to both (Sec. III-E; Sec. II-B for the
submanifold operator).  Written from those definitions, for one window:

* a sparse tensor is a set S of active sites with a feature row each; the
  input's active set S_0 is the set of pillars (cells with a pillar, whatever
  its values);
* a regular sparse convolution (stride s) has the active output sites
  D_s(S) = every output site whose 3x3 receptive field holds an active input
  site; its values there are the dense convolution of the zero-filled input;
* a submanifold convolution (stride 1) keeps the active set: its output is
  computed only at the active input sites (the dense convolution there),
  every other site stays empty;
* ReLU follows each convolution; an empty site holds zeros.

So every layer's output is 1[S_l] * phi(conv3x3(Y_{l-1})) with S_l = D_s(S_{l-1})
for a regular layer and S_l = S_{l-1} for a submanifold one.

Changed sites (Alg. 1: a site is changed when the convolution or the ReLU
changes it; empty sites hold zeros in both windows): A_0 is the set of cells
whose stored feature vector differs bit for bit or whose pillar appeared or
vanished; A_l holds the sites of the receptive-field rule over A_{l-1} that
are active in the current or in the previous window.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from . import conv3x3, propagate_gather, round_bf16


def active_sets(occ: np.ndarray, layers: Sequence[Tuple[int, int, int, bool]], sub: Sequence[bool]) -> List[np.ndarray]:
    """[H_l, W_l] bool active sets S_1..S_L from the pillar set occ [H0, W0]."""
    out, s_prev = [], np.asarray(occ, dtype=bool)
    for (_ci, _co, stride, _r), is_sub in zip(layers, sub):
        if is_sub:
            assert stride == 1
            s_prev = s_prev.copy()
        else:
            s_prev = propagate_gather(s_prev, stride)
        out.append(s_prev)
    return out


def forward(x0: np.ndarray, occ: np.ndarray, weights: Sequence[np.ndarray],
            layers: Sequence[Tuple[int, int, int, bool]], sub: Sequence[bool],
            bf16_storage: bool = False) -> List[np.ndarray]:
    """Outputs Y_1..Y_L (float64) of the sparse backbone, recomputed from the
    window's canvas x0 [H0, W0, C0] (zero off the pillars) and pillar set occ."""
    y = np.asarray(x0, dtype=np.float64)
    ys = []
    for (ci, co, stride, relu), w, s_l in zip(layers, weights, active_sets(occ, layers, sub)):
        z = conv3x3(y, w, stride)
        y = np.maximum(z, 0.0) if relu else z
        if bf16_storage:
            y = round_bf16(y)
        y = y * s_l[..., None]
        ys.append(y)
    return ys


def changed_lists(prev_bits: np.ndarray, new_bits: np.ndarray, prev_occ: np.ndarray, new_occ: np.ndarray,
                  layers: Sequence[Tuple[int, int, int, bool]], sub: Sequence[bool]) -> List[np.ndarray]:
    """Sorted row-major change lists A_0..A_L (int64)."""
    m = np.any(prev_bits != new_bits, axis=-1) | (np.asarray(prev_occ, bool) ^ np.asarray(new_occ, bool))
    out = [np.flatnonzero(m)]
    s_old, s_new = active_sets(prev_occ, layers, sub), active_sets(new_occ, layers, sub)
    for (_ci, _co, stride, _r), so, sn in zip(layers, s_old, s_new):
        m = propagate_gather(m, stride) & (so | sn)
        out.append(np.flatnonzero(m))
    return out


def occupancy(idx: np.ndarray, H: int, W: int) -> np.ndarray:
    """[H, W] bool pillar set of a stride's cell list."""
    m = np.zeros(H * W, dtype=bool)
    m[np.asarray(idx, dtype=np.int64)] = True
    return m.reshape(H, W)
