"""GPU parity of the dense forward's MFMA contraction (the event matrix split
into three bf16 planes times bf16 W on the matrix cores, then the interval
scan) against the fp64 oracle, through the C ABI: ragged tile edges, inputs
not a multiple of the 32-input K tile or of 8, several row and column
tiles, every kernel row, special inputs, finite t_max and M = 1. The
backward (event-sparse) runs on the MFMA forward's outputs."""
import math

import numpy as np
import pytest

from tests.test_gpu_dense import dev, _fwd_bwd_parity, _layer_case, _special_inputs  # noqa: F401

pytestmark = pytest.mark.gpu

MFMA = 0x4


def _mfma(p):
    return dict(p, flags=MFMA)


@pytest.mark.parametrize("B,N_in,N_out,M,tm,ts,k", [
    (5, 37, 70, 8, 1.0, 0.3, 8.0),        # one partial tile each way, N_in % 8 != 0
    (9, 530, 200, 24, 1.0, 0.5, 7.0),     # (2 tau, tau) row, ragged K tail
    (40, 1024, 384, 8, 2.0, 0.4, 6.0),    # 3 x 3 tiles, 32 K tiles
    (3, 96, 130, 1, 1.0, 0.3, 6.0),       # M = 1: two grid points
    (16, 256, 256, 16, 1.5, 0.5, 7.0),    # exact tile multiples
])
def test_mfma_dense_layer(dev, B, N_in, N_out, M, tm, ts, k):  # noqa: F811
    p, t, W = _layer_case(400 + M + B, B, N_in, N_out, M, tm, ts, k=k)
    t = _special_inputs(t, p, np.random.default_rng(M + B))
    _fwd_bwd_parity(dev, _mfma(p), t, W, f"mfma B={B} {N_in}->{N_out} M={M}", bf16=True, seed=M)


INF = math.inf


@pytest.mark.parametrize("tm,ts,k,tmax", [(INF, 0.5, 3.0, INF), (INF, INF, 1.2, 1.6),
                                          (0.5, 0.5, 8.0, INF), (0.3, INF, 5.0, INF),
                                          (1.0, 0.3, 7.0, 1.3)],
                         ids=["inf-tau", "inf-inf", "tau-tau", "tau-inf", "t_max"])
def test_mfma_kernel_rows(dev, tm, ts, k, tmax):  # noqa: F811
    p, t, W = _layer_case(77, 6, 300, 150, 16, tm, ts, k=k, t_max=tmax)
    t = _special_inputs(t, p, np.random.default_rng(5))
    _fwd_bwd_parity(dev, _mfma(p), t, W, f"mfma row ({tm},{ts}) t_max={tmax}", bf16=True, seed=7)


def test_mfma_matches_sparse_decisions(dev):  # noqa: F811
    """Both contractions on the same layer: identical fire / no-fire and
    interval decisions outside the oracle's ambiguity set, times within the
    tolerance of each other (each is also checked against the oracle)."""
    p, t, W = _layer_case(91, 12, 512, 256, 8, 1.0, 0.3, k=7.0)
    g1, o1 = _fwd_bwd_parity(dev, dict(p, flags=0x2), t, W, "sparse twin", bf16=True)
    g2, _ = _fwd_bwd_parity(dev, _mfma(p), t, W, "mfma twin", bf16=True)
    keep = o1["margin"] >= 1e-5
    assert np.array_equal(g1["q"][keep], g2["q"][keep])
    both = keep & (g1["q"] >= 0)
    assert np.all(np.abs(g1["t_out"][both] - g2["t_out"][both]) <= 2e-5)
