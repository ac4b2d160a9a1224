"""GPU parity of the closed-form kernel rows (Table "tab:kernel" rows
(tau, tau), (inf, tau), (inf, inf), and the general row at tau_v = 2 tau_I,
whose crossing has the quadratic closed form of Table "tab:timing_DSTD")
against the fp64 oracle, dense and conv, through the C ABI."""
import math

import numpy as np
import pytest

from tests.test_gpu_dense import dev, _fwd_bwd_parity, _layer_case, _special_inputs  # noqa: F401
from tests import test_gpu_conv as tc

pytestmark = pytest.mark.gpu

INF = math.inf
# (tau_m, tau_s, weight scale k, t_max): k brings 50-90 % of the neurons to
# fire; (inf, inf) potentials with positive input grow without bound, so that
# row closes the last interval to keep silent neurons in the cases
ROWS = [(INF, 0.5, 3.0, INF), (INF, INF, 1.2, 1.6), (0.5, 0.5, 8.0, INF), (1.0, 1.0, 4.5, INF),
        (0.3, INF, 5.0, INF), (1.0, 0.5, 8.0, INF), (0.4, 0.8, 8.0, 1.5)]
IDS = ["inf-tau", "inf-inf", "tau-tau-0.5", "tau-tau-1", "tau-inf", "2tau-tau", "tau-2tau-tmax"]


@pytest.mark.parametrize("M", [8, 16, 33])
@pytest.mark.parametrize("tm,ts,k,tmax", ROWS, ids=IDS)
def test_dense_row(dev, tm, ts, k, tmax, M):  # noqa: F811
    p, t, W = _layer_case(100 + M, 5, 37, 70, M, tm, ts, k=k, t_max=tmax)
    t = _special_inputs(t, p, np.random.default_rng(M))
    gpu, orc = _fwd_bwd_parity(dev, p, t, W, f"row ({tm},{ts}) M={M}", seed=M)
    assert 0 < (orc["q"] >= 0).sum() < orc["q"].size


@pytest.mark.parametrize("tm,ts,k,tmax", ROWS[:4], ids=IDS[:4])
def test_dense_row_multi_tile_bf16_finite_t_max(dev, tm, ts, k, tmax):  # noqa: F811
    p, t, W = _layer_case(7, 9, 300, 260, 32, tm, ts, k=k, t_max=1.4)
    _fwd_bwd_parity(dev, p, t, W, f"row ({tm},{ts}) bf16 t_max", bf16=True, seed=3)


@pytest.mark.parametrize("tm,ts,k,tmax", ROWS[:4], ids=IDS[:4])
def test_dense_row_large_M(dev, tm, ts, k, tmax):  # noqa: F811
    p, t, W = _layer_case(8, 3, 120, 90, 100, tm, ts, k=k, t_max=tmax)
    _fwd_bwd_parity(dev, p, t, W, f"row ({tm},{ts}) M=100", seed=4)


@pytest.mark.parametrize("tm,ts,k,tmax", ROWS[:4], ids=IDS[:4])
@pytest.mark.parametrize("geom", [dict(C_in=3, H=9, W=11, C_out=20, K=3),
                                  dict(C_in=8, H=8, W=8, C_out=70, K=3, stride=2),
                                  dict(C_in=6, H=10, W=10, C_out=16, K=3, pool_in=2)],
                         ids=["s1", "s2", "pool2"])
def test_conv_row(dev, tm, ts, k, tmax, geom):  # noqa: F811
    cs = tc._cs(**geom)
    p, t, W = tc._conv_case(5, 3, cs, 16, tm, ts, k=k, t_max=tmax)
    t = tc._special_inputs(t, p, np.random.default_rng(9))
    tc._conv_parity(dev, p, cs, t, W, f"conv row ({tm},{ts}) {geom}", seed=2)


# Kernels much faster than the grid (taus well below dt = 1/8): crossings
# lie on bumps inside one interval, with v below threshold at both of its
# ends (so for every fired neuron of the dense cases, checked on the oracle's
# grid potentials for these seeds), where the scan's interval filter can only
# pass them through its curvature term.
FAST = [(0.05, 0.02), (0.03, 0.03), (0.02, 0.06)]
FAST_IDS = ["general", "tau-tau", "tau-2tau"]


@pytest.mark.parametrize("tm,ts", FAST, ids=FAST_IDS)
def test_dense_fast_kernel_interior_crossings(dev, tm, ts):  # noqa: F811
    p, t, W = _layer_case(11, 5, 120, 70, 8, tm, ts, k=60.0, spread=0.3)
    gpu, orc = _fwd_bwd_parity(dev, p, t, W, f"fast kernel ({tm},{ts})", seed=5)
    assert (orc["q"] >= 0).sum() > 50


@pytest.mark.parametrize("tm,ts", FAST[:2], ids=FAST_IDS[:2])
@pytest.mark.parametrize("geom", [dict(C_in=8, H=8, W=8, C_out=40), dict(C_in=4, H=9, W=9, C_out=24),
                                  dict(C_in=2, H=10, W=10, C_out=70)],
                         ids=["walk", "list", "direct"])
def test_conv_fast_kernel_interior_crossings(dev, tm, ts, geom):  # noqa: F811
    cs = tc._cs(**geom)
    p, t, W = tc._conv_case(7, 3, cs, 8, tm, ts, k=60.0, spread=0.3)
    tc._conv_parity(dev, p, cs, t, W, f"conv fast kernel ({tm},{ts}) {geom}", seed=6)
