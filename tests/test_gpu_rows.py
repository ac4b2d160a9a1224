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
