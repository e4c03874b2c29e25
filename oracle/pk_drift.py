"""Drift of the bf16 delta forms against recomputation on the 432x496
backbone stream with bf16 storage (18 degree strides, 1% pillar toggles) --
TEST INFRASTRUCTURE ONLY: a CPU measurement with the oracle, no GPU code.

For every stride: the float64 recompute of all 16 layers with bf16 storage
(`oracle.forward`), and the same stream through `DeltaFormModel` with float32
pre-activation maps, once with the exact [new | old] pair delta and once with
the delta rounded to bf16.  Prints, at chosen strides, the largest error over
layers relative to that layer's max |ref|.

    python3 -m oracle.pk_drift [--strides 200] [--every 10]
"""
from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import streams as S  # noqa: E402
from oracle.method_model import DeltaFormModel  # noqa: E402


def rel_err(ys, refs):
    return max(float(np.abs(y - r).max()) / max(float(np.abs(r).max()), 1e-30) for y, r in zip(ys, refs))


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--strides", type=int, default=200)
    ap.add_argument("--every", type=int, default=10)
    args = ap.parse_args()
    wl = S.workload(args.workload)
    ws = S.weights(args.workload)
    layers = [(l.cin, l.cout, l.stride, bool(l.relu)) for l in wl.layers]
    models = {f: DeltaFormModel(layers, ws, delta=f) for f in ("pair", "rounded")}
    worst = {f: 0.0 for f in models}
    print(f"# {args.workload}: {wl.description}; {args.strides} delta strides after the full window; "
          f"oracle threads {oracle.threads()}")
    print("| stride | pair form: max rel err | rounded delta: max rel err |")
    print("|---|---|---|")
    t0 = time.time()
    for k, st in enumerate(S.make_stream(args.workload, n_strides=args.strides)):
        x = oracle.exact_canvas(S.canvas(st, wl.H, wl.W, wl.C0), wl.dtype)
        refs = oracle.forward(x, ws, layers, bf16_storage=True)
        errs = {f: rel_err(m.step(x), refs) for f, m in models.items()}
        for f in errs:
            worst[f] = max(worst[f], errs[f])
        if k == 0 or k % args.every == 0 or k == args.strides:
            print(f"| {k} | {errs['pair']:.3e} | {errs['rounded']:.3e} |", flush=True)
    print(f"| worst | {worst['pair']:.3e} | {worst['rounded']:.3e} |")
    print(f"# {time.time() - t0:.0f} s")
    return 0


if __name__ == "__main__":
    sys.exit(main())
