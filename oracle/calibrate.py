"""Calibrate the per-layer weight scale k of the synthetic workloads.

Writes ``paper_2607_14672_amd/calibration.json``. For each workload whose
weights follow W = (k / fan_in) (1 + 0.3 sqrt(fan_in) z), layer by layer, on
the first 8 samples, propagating the oracle's own (float32-rounded) spike
times to the next layer:
  - the last layer of a workload: k is bisected (log space) so that ~70 % of
    its neurons fire;
  - a hidden layer: k maximises the fraction of its spikes that land inside
    the next layer's event support [T_0' - dt', T_M' + dt'), so that activity
    propagates through the synfire windows (at random initialisation leaky
    neurons mostly fire inside their own input window).
Only the fp64 oracle is used. The paper leaves the initial weight
distribution open (Table "tab:search_space" searches scales); this fixes one
reproducible choice that keeps every layer active.

Run: python -m oracle.calibrate [workload ...]
"""
from __future__ import annotations

import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_14672_amd import workloads as wlmod  # noqa: E402

TARGET = 0.70
N_CAL = 8


def layer_forward(lay, t_in, W):
    p = lay.params()
    if lay.kind == "dense":
        return oracle.dstd_forward(p, t_in.reshape(t_in.shape[0], -1), W)
    B = t_in.shape[0]
    r = oracle.conv_forward(p, lay.conv_shape(), t_in.reshape(B, lay.C_in, lay.H, lay.W), W)
    return {k: v.reshape(B, -1) for k, v in r.items()}


def in_grid_fraction(lay, t):
    lo = lay.t0 - lay.dt
    hi = lay.t0 + (lay.M + 1) * lay.dt
    return float(np.mean((t >= lo) & (t < hi)))


def calibrate(name):
    wl = wlmod.get(name)
    dr = wlmod.Draws(wl, batch=N_CAL)
    t = dr.t_in.astype(np.float32)
    ks, fires, ingrid = [], [], []
    for l, lay in enumerate(wl.layers):
        ingrid.append(in_grid_fraction(lay, t))

        def frac(k):
            W = dr.weights(l, k)
            r = layer_forward(lay, t, W)
            return float(np.mean(r["q"] >= 0)), r

        if l + 1 < len(wl.layers):
            nxt = wl.layers[l + 1]

            def score(k):
                f, r = frac(k)
                return in_grid_fraction(nxt, r["t_out"]), f

            grid = np.exp(np.linspace(math.log(0.1), math.log(3000.0), 36))
            vals = [score(k)[0] for k in grid]
            best = int(np.argmax(vals))
            lo_k = grid[max(best - 1, 0)]
            hi_k = grid[min(best + 1, len(grid) - 1)]
            fine = np.exp(np.linspace(math.log(lo_k), math.log(hi_k), 13))
            fv = [score(k)[0] for k in fine]
            k = float(fine[int(np.argmax(fv))])
        else:
            lo, hi = math.log(0.05), math.log(3000.0)
            f_hi, _ = frac(math.exp(hi))
            if f_hi < TARGET:
                k = math.exp(hi)
            else:
                for _ in range(18):
                    mid = 0.5 * (lo + hi)
                    f, _ = frac(math.exp(mid))
                    if f >= TARGET:
                        hi = mid
                    else:
                        lo = mid
                k = math.exp(hi)
        f, r = frac(k)
        ks.append(k)
        fires.append(f)
        t = r["t_out"].astype(np.float32).reshape(N_CAL, -1)
        print(f"  {name} layer {l + 1}: k={k:.5g} fire={f:.3f} in-grid inputs={ingrid[-1]:.3f}",
              flush=True)
    return dict(k=ks, fire_frac=fires, in_grid_frac=ingrid, samples=N_CAL,
                rule="hidden: max next-grid fraction; last: 70% fire")


def main(names):
    path = os.path.join(ROOT, "paper_2607_14672_amd", "calibration.json")
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    for n in names:
        t0 = time.time()
        data[n] = calibrate(n)
        print(f"{n}: {time.time() - t0:.1f}s", flush=True)
        with open(path, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    default = ["dense1-cal", "mlp3", "wide-M8", "wide-M32", "wide-M64", "wide-M128", "conv9", "conv20"]
    main(sys.argv[1:] or default)
