"""Host-side logic of bench.py (CPU only): the algorithmic work count that
the roofline figures are based on."""
import numpy as np
import pytest

import bench
from paper_2607_14672_amd import workloads as wl


def _brute_updates(lay, ing):
    """Count (input with events, output neuron) connections by walking every
    output neuron's receptive field."""
    B = ing.shape[0]
    if lay.kind == "dense":
        return int(ing.reshape(B, -1).sum()) * lay.n_out
    x = ing.reshape(B, lay.C_in, lay.H, lay.W)
    if lay.pool_in == 2:
        Hp, Wp = lay.H // 2, lay.W // 2
    elif lay.pool_in == 0:
        Hp, Wp = 1, 1
    else:
        Hp, Wp = lay.H, lay.W
    Ho = (Hp + 2 * lay.pad - lay.KH) // lay.stride + 1
    Wo = (Wp + 2 * lay.pad - lay.KW) // lay.stride + 1
    tot = 0
    for b in range(B):
        for oy in range(Ho):
            for ox in range(Wo):
                for ky in range(lay.KH):
                    for kx in range(lay.KW):
                        py, px = oy * lay.stride + ky - lay.pad, ox * lay.stride + kx - lay.pad
                        if not (0 <= py < Hp and 0 <= px < Wp):
                            continue
                        if lay.pool_in == 2:
                            tot += int(x[b, :, 2 * py:2 * py + 2, 2 * px:2 * px + 2].sum())
                        elif lay.pool_in == 0:
                            tot += int(x[b].sum())
                        else:
                            tot += int(x[b, :, py, px].sum())
    return tot * lay.C_out


@pytest.mark.parametrize("kw", [
    dict(C_in=3, H=7, W=6, C_out=5, KH=3, KW=3, stride=1, pad=1, pool_in=1),
    dict(C_in=2, H=9, W=7, C_out=4, KH=3, KW=3, stride=2, pad=1, pool_in=1),
    dict(C_in=3, H=8, W=6, C_out=2, KH=3, KW=3, stride=1, pad=1, pool_in=2),
    dict(C_in=4, H=3, W=3, C_out=5, KH=1, KW=1, stride=1, pad=0, pool_in=0),
    dict(C_in=2, H=6, W=7, C_out=3, KH=3, KW=1, stride=1, pad=0, pool_in=1),
])
def test_event_updates_matches_receptive_field_walk(kw):
    rng = np.random.default_rng(0)
    lay = wl.LayerSpec("conv", kw["C_in"] * kw["H"] * kw["W"], 0, 8, 0.0, 0.125, 1.0, 0.3, **kw)
    ing = rng.random((3, kw["C_in"], kw["H"], kw["W"])) < 0.6
    assert bench.event_updates(lay, ing) == _brute_updates(lay, ing)


def test_event_updates_dense():
    lay = wl.LayerSpec("dense", 10, 7, 8, 0.0, 0.125, 1.0, 0.3)
    ing = np.random.default_rng(1).random((4, 10)) < 0.5
    assert bench.event_updates(lay, ing) == int(ing.sum()) * 7


def test_gpus_other_than_one_exit_with_message():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True,
                       text=True)
    assert r.returncode == 2 and "one GPU" in r.stderr
