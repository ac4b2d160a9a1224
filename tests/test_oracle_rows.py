"""Pins of the oracle's closed-form kernel rows (Table "tab:kernel" rows
(tau, tau), (inf, tau), (inf, inf); Tables "tab:DSTD_kernels",
"tab:timing_DSTD"), each against a route the oracle does not use: numerical
integration of the LIF ODE with infinite or equal time constants, limits of
the general row, exact values of the Lambert W function, finite
differences."""
import math

import numpy as np
import pytest

import oracle
from tests.bruteforce import simulate

INF = math.inf
ROWS = [(INF, 0.5), (INF, INF), (0.5, 0.5), (1.0, 1.0)]
IDS = ["inf-tau", "inf-inf", "tau-tau-0.5", "tau-tau-1"]


def _p(tm, ts, M=16, t0=0.0, dt=None, theta=1.0, t_max=INF):
    return dict(tau_m=tm, tau_s=ts, threshold=theta, M=M, t0=t0, dt=(1.0 / M if dt is None else dt),
                t_max=t_max)


def _wscale(tm, ts):
    """Total input weight that brings one unit-window layer near threshold:
    the PSP grows like u (inf, inf), saturates at tau (inf, tau), peaks at
    tau/e (tau, tau)."""
    if math.isinf(tm) and math.isinf(ts):
        return 3.0
    if math.isinf(tm) or math.isinf(ts):
        return 3.0 / min(tm, ts)
    return 3.0 * math.e / tm


# ----------------------------------------------------------- Lambert W_0 --
def test_lambert_w0_exact_values():
    assert oracle.lambert_w0(0.0) == 0.0
    assert oracle.lambert_w0(-1.0 / math.e) == pytest.approx(-1.0, abs=1e-7)
    # w e^w = x at w = -ln 2, ln 2 and the omega constant
    assert oracle.lambert_w0(-math.log(2) / 2) == pytest.approx(-math.log(2), rel=1e-14)
    assert oracle.lambert_w0(2 * math.log(2)) == pytest.approx(math.log(2), rel=1e-14)
    assert oracle.lambert_w0(1.0) == pytest.approx(0.567143290409783873, rel=1e-15)
    assert oracle.lambert_w0(math.e) == pytest.approx(1.0, rel=1e-14)
    assert math.isnan(oracle.lambert_w0(-0.5))


def test_lambert_w0_defining_identity_and_branch():
    for x in np.concatenate([-np.geomspace(1e-12, 1 / math.e - 1e-9, 40), np.geomspace(1e-12, 1e6, 40)]):
        w = oracle.lambert_w0(float(x))
        assert w >= -1.0
        assert w * math.exp(w) == pytest.approx(x, rel=1e-12, abs=1e-300)


# ---------------------------------------------------------------- kernels --
@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_kernel_row_is_lif_impulse_response(tm, ts):
    """K(t) of each row equals v(t) of the LIF ODE after a unit input at 0."""
    qs = [0.0, 0.01, 0.1, 0.37, 1.0, 2.5]
    _, vals = simulate(tm, ts, [0.0], [1.0], 3.0, query=qs)
    for t in qs:
        assert oracle.kernel(tm, ts, t) == pytest.approx(vals[t], abs=1e-11)
        assert oracle.kernel(ts, tm, t) == oracle.kernel(tm, ts, t)  # symmetric
    assert oracle.kernel(tm, ts, -0.1) == 0.0


@pytest.mark.parametrize("t", [-0.09, -0.03, 0.0, 0.02, 0.07, 0.099])
def test_closed_rows_are_limits_of_the_general_row(t):
    """The (inf, tau), (tau, tau) and (inf, inf) rows of the kernel and DSTD
    kernel tables are the limits of the general row."""
    D = 0.1
    pairs = [((1e8, 0.5), (INF, 0.5), 1e-6), ((0.5 * (1 + 1e-7), 0.5), (0.5, 0.5), 1e-6),
             ((2e7, 1e7), (INF, INF), 1e-6)]
    for (gv, gi), (cv, ci), tol in pairs:
        if t >= 0:
            assert oracle.kernel(gv, gi, t) == pytest.approx(oracle.kernel(cv, ci, t), rel=tol, abs=1e-12)
        assert oracle.kdstd(gv, gi, D, t) == pytest.approx(oracle.kdstd(cv, ci, D, t), rel=tol, abs=1e-9)


@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_dstd_matches_exact_potential_at_grid_points(tm, ts):
    """Defining property of DSTD (App. B.2) for each row: v^(T_m) = v(T_m),
    and v^ = v after the right grid point of the last input. Both potentials
    come from the ODE; only the event weights are the oracle's."""
    rng = np.random.default_rng(17)
    M = 10
    p = _p(tm, ts, M=M, t0=0.2, dt=0.1)
    t_in = (0.2 + rng.random((1, 12)) * 0.999).astype(np.float64)
    w = rng.normal(0.3, 0.5, 12)
    s, _ = oracle.dstd_events(p, t_in)
    wh = (s[0] * w[None, :]).sum(axis=1)
    grid = 0.2 + 0.1 * np.arange(M + 1)
    late = [1.25, 1.6, 2.3]
    _, v = simulate(tm, ts, t_in[0], w, 3.0, query=list(grid) + late)
    _, vh = simulate(tm, ts, grid, wh, 3.0, query=list(grid) + late)
    for tq in list(grid) + late:
        assert vh[tq] == pytest.approx(v[tq], abs=1e-9)


@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_event_support_and_unit_weight_on_grid(tm, ts):
    p = _p(tm, ts, M=8, t0=0.0, dt=0.125)
    t = np.array([[0.0, 0.3, 0.5, 0.999, -0.1, -0.13, 1.1249, 1.13, np.inf]])
    s, ds = oracle.dstd_events(p, t)
    nz = (s[0] != 0).sum(axis=0)
    assert list(nz) == [1, 2, 1, 2, 1, 0, 1, 0, 0]
    assert s[0, 0, 0] == pytest.approx(1.0, abs=1e-14)
    assert s[0, 4, 2] == pytest.approx(1.0, abs=1e-14)
    # derivative of each weight by central differences
    for j, tj in [(1, 0.3), (3, 0.999)]:
        h = 1e-7
        sp, _ = oracle.dstd_events(p, np.array([[tj + h]]))
        sm, _ = oracle.dstd_events(p, np.array([[tj - h]]))
        np.testing.assert_allclose(ds[0, :, j], (sp[0, :, 0] - sm[0, :, 0]) / (2 * h), rtol=1e-6, atol=1e-6)


# ------------------------------------------------------------ spike times --
@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_dstd_spike_time_is_first_crossing_of_impulse_ode(tm, ts):
    """The closed-form candidates of Table "tab:timing_DSTD" (W_0 branch for
    (tau, tau)) give the first threshold crossing of the ODE driven by the
    weighted events."""
    rng = np.random.default_rng(31)
    M = 12
    p = _p(tm, ts, M=M)
    B, N_in, N_out = 3, 40, 6
    t_in = rng.random((B, N_in))
    W = rng.normal(1.0, 2.0, (N_out, N_in)) * (_wscale(tm, ts) / N_in)
    f = oracle.dstd_forward(p, t_in, W, want_what=True)
    grid = np.arange(M + 1) / M
    fired = 0
    for b in range(B):
        for i in range(N_out):
            fire, _ = simulate(tm, ts, grid, f["what"][b, :, i], 30.0, theta=1.0)
            if np.isfinite(fire):
                fired += 1
                assert f["t_out"][b, i] == pytest.approx(fire, abs=1e-8)
            else:
                assert f["q"][b, i] == -1
    assert fired >= 3


@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_exact_spike_time_is_first_crossing_of_input_ode(tm, ts):
    rng = np.random.default_rng(32)
    p = _p(tm, ts)
    B, N_in, N_out = 2, 30, 5
    t_in = rng.random((B, N_in))
    t_in[0, 3] = np.inf
    W = rng.normal(1.0, 2.0, (N_out, N_in)) * (_wscale(tm, ts) / N_in)
    e = oracle.exact_forward(p, t_in, W)
    fired = 0
    for b in range(B):
        for i in range(N_out):
            fire, _ = simulate(tm, ts, t_in[b], W[i], 30.0, theta=1.0)
            if np.isfinite(fire):
                fired += 1
                assert e["t_out"][b, i] == pytest.approx(fire, abs=1e-8)
            else:
                assert not np.isfinite(e["t_out"][b, i])
    assert fired >= 3


def test_non_leaky_spike_is_eq_spike_no_leak():
    """Row (inf, inf): the spike time is (V_th + sum_S w t_j) / sum_S w over
    the inputs S before it (Eq. (spike_no_leak)), checked with the set S
    found from the result itself."""
    rng = np.random.default_rng(33)
    p = _p(INF, INF)
    t_in = rng.random((1, 20))
    W = rng.random((5, 20)) * 0.4
    e = oracle.exact_forward(p, t_in, W)
    for i in range(5):
        t = e["t_out"][0, i]
        S = t_in[0] <= t
        assert t == pytest.approx((1.0 + np.sum(W[i, S] * t_in[0, S])) / np.sum(W[i, S]), rel=1e-12)


@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_dstd_equals_exact_when_inputs_on_grid_points(tm, ts):
    rng = np.random.default_rng(34)
    M = 16
    p = _p(tm, ts, M=M)
    t = rng.integers(0, M + 1, (3, 50)) / M
    W = (_wscale(tm, ts) / 50) * (1 + 0.3 * math.sqrt(50) * rng.standard_normal((10, 50)))
    a = oracle.dstd_forward(p, t, W)
    e = oracle.exact_forward(p, t, W)
    np.testing.assert_array_equal(np.isfinite(a["t_out"]), np.isfinite(e["t_out"]))
    f = np.isfinite(a["t_out"])
    assert f.sum() >= 5
    np.testing.assert_allclose(a["t_out"][f], e["t_out"][f], atol=1e-10)


@pytest.mark.parametrize("tm,ts", [(INF, 0.5), (INF, INF), (0.5, 0.5)], ids=IDS[:3])
def test_dstd_converges_to_exact_as_M_grows(tm, ts):
    rng = np.random.default_rng(35)
    t = rng.random((4, 200))
    W = (_wscale(tm, ts) / 200) * (1 + 0.3 * math.sqrt(200) * rng.standard_normal((30, 200)))
    e = oracle.exact_forward(_p(tm, ts), t, W)
    errs = []
    for M in [5, 10, 20, 40, 80, 160, 320]:
        a = oracle.dstd_forward(_p(tm, ts, M=M), t, W)
        both = np.isfinite(a["t_out"]) & np.isfinite(e["t_out"])
        assert both.sum() > 40
        errs.append(np.sqrt(np.mean((a["t_out"][both] - e["t_out"][both]) ** 2)))
    assert errs[0] > 3 * errs[2]
    assert errs[-1] < errs[3] < errs[1]
    assert errs[-1] < 2e-4


# --------------------------------------------------------------- backward --
@pytest.mark.parametrize("tm,ts", ROWS, ids=IDS)
def test_backward_matches_finite_differences(tm, ts):
    rng = np.random.default_rng(36)
    B, N_in, N_out, M = 2, 16, 5, 12
    p = _p(tm, ts, M=M)
    t = rng.random((B, N_in))
    W = (_wscale(tm, ts) * 1.5 / N_in) * (1 + 0.3 * math.sqrt(N_in) * rng.standard_normal((N_out, N_in)))
    g = rng.standard_normal((B, N_out))

    def loss(tt, WW):
        f = oracle.dstd_forward(p, tt, WW)
        return float(np.sum(g * np.where(f["q"] >= 0, f["t_out"], 0.0))), f

    L0, f0 = loss(t, W)
    assert (f0["q"] >= 0).sum() >= 4
    dW, dt = oracle.dstd_backward(p, t, W, f0, np.where(f0["q"] >= 0, g, 0.0))
    h = 1e-6
    checked = 0
    for i in range(N_out):
        for j in range(0, N_in, 3):
            Wp, Wm = W.copy(), W.copy()
            Wp[i, j] += h
            Wm[i, j] -= h
            Lp, fp = loss(t, Wp)
            Lm, fm = loss(t, Wm)
            if not (np.array_equal(fp["q"], f0["q"]) and np.array_equal(fm["q"], f0["q"])):
                continue
            assert dW[i, j] == pytest.approx((Lp - Lm) / (2 * h), rel=1e-5, abs=1e-8)
            checked += 1
    for b in range(B):
        for j in range(N_in):
            x = t[b, j] * M
            if abs(x - round(x)) < 1e-3:
                continue
            tp, tmn = t.copy(), t.copy()
            tp[b, j] += h
            tmn[b, j] -= h
            Lp, fp = loss(tp, W)
            Lm, fm = loss(tmn, W)
            if not (np.array_equal(fp["q"], f0["q"]) and np.array_equal(fm["q"], f0["q"])):
                continue
            assert dt[b, j] == pytest.approx((Lp - Lm) / (2 * h), rel=1e-5, abs=1e-8)
            checked += 1
    assert checked > 30
