"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these tests re-types the oracle's own formulas: each checks it
against an independent route (numerical ODE integration, a closed form the
oracle does not use, a defining property, an invariant, finite differences).
"""
import math

import numpy as np
import pytest

import oracle
from tests.bruteforce import simulate

TAU = [(1.0, 0.3), (1.0, 0.5), (2.0, 0.4), (1.5, 0.5), (0.4, 0.2)]


def _p(tm, ts, M=16, t0=0.0, dt=None, theta=1.0, t_max=math.inf):
    return dict(tau_m=tm, tau_s=ts, threshold=theta, M=M, t0=t0, dt=(1.0 / M if dt is None else dt),
                t_max=t_max)


# ---------------------------------------------------------------- kernel K --
@pytest.mark.parametrize("tm,ts", TAU)
def test_kernel_is_lif_impulse_response(tm, ts):
    """K(t) (Table "tab:kernel") equals v(t) of the LIF ODE after a unit input at 0."""
    ts_q = [0.0, 0.01, 0.1, 0.37, 1.0, 2.5]
    _, vals = simulate(tm, ts, [0.0], [1.0], 3.0, query=ts_q)
    for t in ts_q:
        assert oracle.kernel(max(tm, ts), min(tm, ts), t) == pytest.approx(vals[t], abs=1e-11)
    assert oracle.kernel(max(tm, ts), min(tm, ts), -0.1) == 0.0


@pytest.mark.parametrize("tm,ts", TAU)
def test_single_input_fires_iff_weight_reaches_psp_peak(tm, ts):
    """One input of weight w fires iff w * K_max >= theta, with the PSP peak
    K_max = tau_I (tau_I/tau_v)^(tau_I/(tau_v - tau_I)) (maximum of K)."""
    tv, ti = max(tm, ts), min(tm, ts)
    kmax = ti * (ti / tv) ** (ti / (tv - ti))
    p = _p(tm, ts, M=8)
    t_in = np.array([[0.25]])  # exactly on a grid point
    for scale, fires in [(1 + 1e-7, True), (1 - 1e-7, False)]:
        W = np.array([[scale / kmax]])
        f = oracle.dstd_forward(p, t_in, W)
        e = oracle.exact_forward(p, t_in, W)
        assert (f["q"][0, 0] >= 0) == fires
        assert np.isfinite(e["t_out"][0, 0]) == fires
    # near-tangent crossing happens at the PSP peak time
    upk = math.log(tv / ti) / (1 / ti - 1 / tv)
    f = oracle.dstd_forward(p, t_in, np.array([[(1 + 1e-10) / kmax]]))
    assert f["t_out"][0, 0] == pytest.approx(0.25 + upk, abs=2e-4)


# --------------------------------------------------------------- events --
@pytest.mark.parametrize("tm,ts", TAU)
def test_dstd_matches_exact_potential_at_grid_points(tm, ts):
    """Defining property of DSTD (App. B.2): v^(T_m) = v(T_m) for every m, and
    v^ = v after the right grid point of the last input. Both potentials are
    integrated numerically from the ODE; only the event weights s_jm come from
    the oracle."""
    rng = np.random.default_rng(7)
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


@pytest.mark.parametrize("tm,ts", TAU)
def test_event_support_and_values(tm, ts):
    """Compact two-point support (App. B.3), weight 1 at a grid point, and
    continuity of the weights across grid points (a spike moving through a
    grid point does not jump)."""
    p = _p(tm, ts, M=8, t0=0.0, dt=0.125)
    t = np.array([[0.0, 0.125, 0.3, 0.49999999, 0.5, 0.999, 1.0, 1.1249, 1.13, -0.1, -0.13, np.inf]])
    s, _ = oracle.dstd_events(p, t)
    nz = (s[0] != 0).sum(axis=0)
    assert list(nz[:9]) == [1, 1, 2, 2, 1, 2, 1, 1, 0]
    assert list(nz[9:]) == [1, 0, 0]
    assert s[0, 0, 0] == pytest.approx(1.0, abs=1e-14)
    assert s[0, 1, 1] == pytest.approx(1.0, abs=1e-14)
    assert s[0, 4, 4] == pytest.approx(1.0, abs=1e-14)
    # just below the grid point 0.5 the weight sits at T_4 (right neighbour)
    assert s[0, 4, 3] == pytest.approx(1.0, abs=1e-6)
    assert s[0, 3, 3] == pytest.approx(0.0, abs=1e-6)
    # all weights lie in [0, 1]
    assert s.min() >= -1e-15 and s.max() <= 1 + 1e-15


def test_event_kernel_reduces_to_hat_for_large_time_constants():
    """For tau_v, tau_I -> inf the kernel table's (inf, inf) row is the hat
    function max(1 - |t|/dt, 0); the general row must approach it."""
    for t in [-0.09, -0.05, -0.001, 0.0, 0.02, 0.07, 0.099]:
        hat = max(1 - abs(t) / 0.1, 0.0)
        assert oracle.kdstd(2e5, 1e5, 0.1, t) == pytest.approx(hat, abs=1e-5)


# -------------------------------------------------------- interval solver --
@pytest.mark.parametrize("tm,ts", TAU)
def test_dstd_spike_time_is_first_crossing_of_impulse_ode(tm, ts):
    """The DSTD spike time (Eq. (timing_DSTD)) equals the first threshold
    crossing of the LIF ODE driven by impulses w^_m at T_m."""
    rng = np.random.default_rng(11)
    M = 12
    p = _p(tm, ts, M=M)
    B, N_in, N_out = 3, 40, 6
    t_in = rng.random((B, N_in))
    W = rng.normal(3.0 / N_in, 6.0 / N_in, (N_out, N_in)) * (3.0 / max(tm, ts))
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


@pytest.mark.parametrize("tm,ts", TAU)
def test_exact_spike_time_is_first_crossing_of_input_ode(tm, ts):
    """The exact method (Alg. 1, Eq. (timing_exact)) equals the first crossing
    of the LIF ODE driven by the actual input spikes."""
    rng = np.random.default_rng(12)
    p = _p(tm, ts)
    B, N_in, N_out = 2, 30, 5
    t_in = rng.random((B, N_in))
    t_in[0, 3] = np.inf
    W = rng.normal(3.0 / N_in, 6.0 / N_in, (N_out, N_in)) * (3.0 / max(tm, ts))
    e = oracle.exact_forward(p, t_in, W)
    for b in range(B):
        for i in range(N_out):
            fire, _ = simulate(tm, ts, t_in[b], W[i], 30.0, theta=1.0)
            if np.isfinite(fire):
                assert e["t_out"][b, i] == pytest.approx(fire, abs=1e-8)
            else:
                assert not np.isfinite(e["t_out"][b, i])


def _closed_form_2tau(a, b, th, tau):
    """(2tau, tau) rows of Tables "tab:spike_timing" / "tab:timing_DSTD"."""
    D = b * b - 2 * a * th / tau
    return 2 * tau * math.log((b - math.sqrt(D)) / (th / tau))


def test_dstd_matches_paper_closed_form_2tau_tau():
    """Config-2 time constants (1.0, 0.5) = (2 tau, tau): the candidate of
    Table "tab:timing_DSTD" evaluated at the selected interval reproduces the
    oracle's bisection root."""
    rng = np.random.default_rng(3)
    M, tau = 32, 0.5
    p = _p(2 * tau, tau, M=M, t0=1.0)
    t_in = 1.0 + rng.random((4, 200))
    W = (6.0 / 200) * (1 + 0.3 * math.sqrt(200) * rng.standard_normal((30, 200)))
    f = oracle.dstd_forward(p, t_in, W, want_what=True)
    T = 1.0 + np.arange(M + 1) / M
    n = 0
    for b in range(4):
        for i in range(30):
            q = f["q"][b, i]
            if q < 0:
                continue
            a = np.sum(f["what"][b, :q + 1, i] * np.exp(T[:q + 1] / tau))
            bb = np.sum(f["what"][b, :q + 1, i] * np.exp(T[:q + 1] / (2 * tau)))
            assert _closed_form_2tau(a, bb, 1.0, tau) == pytest.approx(f["t_out"][b, i], abs=1e-10)
            n += 1
    assert n > 20


def test_exact_matches_paper_closed_form_2tau_tau():
    rng = np.random.default_rng(4)
    tau = 0.5
    p = _p(2 * tau, tau)
    t_in = rng.random((3, 100))
    W = (6.0 / 100) * (1 + 0.3 * 10 * rng.standard_normal((20, 100)))
    e = oracle.exact_forward(p, t_in, W)
    n = 0
    for b in range(3):
        for i in range(20):
            t = e["t_out"][b, i]
            if not np.isfinite(t):
                continue
            sel = t_in[b] <= t
            a = np.sum(W[i, sel] * np.exp(t_in[b, sel] / tau))
            bb = np.sum(W[i, sel] * np.exp(t_in[b, sel] / (2 * tau)))
            assert _closed_form_2tau(a, bb, 1.0, tau) == pytest.approx(t, abs=1e-10)
            n += 1
    assert n > 20


def test_non_leaky_limit_matches_eq_spike_no_leak():
    """With both time constants large the potential is ~ sum_S w (t - t_j)
    (Table "tab:kernel" row (inf, inf)); the exact spike time approaches
    Eq. (spike_no_leak): t = (V_th + sum_S w t_j) / sum_S w."""
    rng = np.random.default_rng(5)
    p = _p(4e5, 2e5)
    t_in = rng.random((1, 20))
    W = rng.random((5, 20)) * 0.4
    e = oracle.exact_forward(p, t_in, W)
    for i in range(5):
        t = e["t_out"][0, i]
        S = t_in[0] <= t
        ref = (1.0 + np.sum(W[i, S] * t_in[0, S])) / np.sum(W[i, S])
        assert t == pytest.approx(ref, rel=1e-4)


# -------------------------------------------------------------- invariants --
def _layer(seed=0, B=4, N_in=60, N_out=12, k=6.0):
    rng = np.random.default_rng(seed)
    t = rng.random((B, N_in))
    W = (k / N_in) * (1 + 0.3 * math.sqrt(N_in) * rng.standard_normal((N_out, N_in)))
    return t, W


def test_no_input_no_spike():
    p = _p(1.0, 0.3)
    t = np.full((2, 10), np.inf)
    W = np.ones((3, 10))
    for fn in (oracle.dstd_forward, oracle.exact_forward):
        r = fn(p, t, W)
        assert np.all(np.isinf(r["t_out"]))


def test_monotone_in_uniform_weight_scale():
    """Scaling all weights by lambda > 1 never delays a spike and never
    silences a neuron (potential scales by lambda pointwise)."""
    p = _p(1.0, 0.3)
    t, W = _layer(1, k=4.0)
    base = oracle.dstd_forward(p, t, W)
    for lam in [1.01, 1.3, 2.0]:
        r = oracle.dstd_forward(p, t, W * lam)
        fired = base["q"] >= 0
        assert np.all(r["q"][fired] >= 0)
        assert np.all(r["t_out"][fired] <= base["t_out"][fired] + 1e-12)


def test_time_constant_swap_symmetry():
    t, W = _layer(2)
    a = oracle.dstd_forward(_p(1.0, 0.3), t, W)
    b = oracle.dstd_forward(_p(0.3, 1.0), t, W)
    assert np.array_equal(a["q"], b["q"])
    np.testing.assert_allclose(a["t_out"], b["t_out"], rtol=0, atol=1e-12)


def test_shift_of_inputs_and_grid_shifts_output():
    t, W = _layer(3)
    a = oracle.dstd_forward(_p(1.0, 0.3, t0=0.0), t, W)
    b = oracle.dstd_forward(_p(1.0, 0.3, t0=2.0), t + 2.0, W)
    assert np.array_equal(a["q"], b["q"])
    f = a["q"] >= 0
    np.testing.assert_allclose(b["t_out"][f], a["t_out"][f] + 2.0, atol=1e-11)


def test_input_permutation_and_batch_independence():
    t, W = _layer(4)
    perm = np.random.default_rng(0).permutation(t.shape[1])
    a = oracle.dstd_forward(_p(1.0, 0.3), t, W)
    b = oracle.dstd_forward(_p(1.0, 0.3), t[:, perm], W[:, perm])
    assert np.array_equal(a["q"], b["q"])
    np.testing.assert_allclose(a["t_out"], b["t_out"], atol=1e-12)
    c = oracle.dstd_forward(_p(1.0, 0.3), t[2:3], W)
    np.testing.assert_array_equal(c["t_out"][0], a["t_out"][2])


def test_dstd_equals_exact_when_inputs_on_grid_points():
    """Inputs exactly on grid points are represented without error
    (K_DSTD(0) = 1), so DSTD reproduces the exact spike time."""
    rng = np.random.default_rng(6)
    M = 16
    p = _p(1.0, 0.3, M=M)
    t = rng.integers(0, M + 1, (3, 50)) / M
    W = (8.0 / 50) * (1 + 0.3 * math.sqrt(50) * rng.standard_normal((10, 50)))
    a = oracle.dstd_forward(p, t, W)
    e = oracle.exact_forward(p, t, W)
    np.testing.assert_array_equal(np.isfinite(a["t_out"]), np.isfinite(e["t_out"]))
    f = np.isfinite(a["t_out"])
    np.testing.assert_allclose(a["t_out"][f], e["t_out"][f], atol=1e-10)


def test_dstd_equals_exact_after_last_input_grid_point():
    """v^ = v for t >= the right grid point of the last input, so a crossing
    there is exact (App. B.2)."""
    rng = np.random.default_rng(8)
    M = 20
    p = _p(1.0, 0.3, M=M)
    t = rng.random((4, 80)) * 0.5          # inputs in [0, 0.5), right grid point <= 0.5
    W = (6.0 / 80) * (1 + 0.3 * math.sqrt(80) * rng.standard_normal((40, 80)))
    a = oracle.dstd_forward(p, t, W)
    e = oracle.exact_forward(p, t, W)
    late = np.isfinite(e["t_out"]) & (e["t_out"] > 0.5 + 1e-9)
    assert late.sum() > 10
    np.testing.assert_allclose(a["t_out"][late], e["t_out"][late], atol=1e-10)


@pytest.mark.parametrize("tm,ts,mult", [(1.0, 0.3, 1.0), (0.4, 0.2, 3.0)])
def test_dstd_converges_to_exact_as_M_grows(tm, ts, mult):
    """|t^_M - t| -> 0 as M grows (App. D.1); the error at small M is visibly
    larger than at M = 20 (Sec. 3, Fig. 2a)."""
    rng = np.random.default_rng(9)
    t = rng.random((4, 200))
    W = mult * (6.0 / 200) * (1 + 0.3 * math.sqrt(200) * rng.standard_normal((30, 200)))
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


# ---------------------------------------------------------------- backward --
def _fd_setup(seed, tm, ts, M=12):
    rng = np.random.default_rng(seed)
    B, N_in, N_out = 2, 16, 5
    p = _p(tm, ts, M=M)
    t = rng.random((B, N_in))
    W = (10.0 / N_in) * (1 + 0.3 * math.sqrt(N_in) * rng.standard_normal((N_out, N_in)))
    g = rng.standard_normal((B, N_out))
    return p, t, W, g


def _loss(p, t, W, g):
    f = oracle.dstd_forward(p, t, W)
    tt = np.where(f["q"] >= 0, f["t_out"], 0.0)
    return float(np.sum(g * tt)), f


@pytest.mark.parametrize("tm,ts", [(1.0, 0.3), (1.0, 0.5), (2.0, 0.4)])
def test_backward_matches_finite_differences(tm, ts):
    """Implicit-function gradients (dL/dW, dL/dt_in) against central finite
    differences of the fp64 forward, away from kinks."""
    p, t, W, g = _fd_setup(21, tm, ts)
    L0, f0 = _loss(p, t, W, g)
    assert (f0["q"] >= 0).sum() >= 4
    dW, dt = oracle.dstd_backward(p, t, W, f0, np.where(f0["q"] >= 0, g, 0.0))
    h = 1e-6
    M = p["M"]
    checked = 0
    for i in range(W.shape[0]):
        for j in range(0, W.shape[1], 3):
            Wp, Wm = W.copy(), W.copy()
            Wp[i, j] += h
            Wm[i, j] -= h
            Lp, fp = _loss(p, t, Wp, g)
            Lm, fm = _loss(p, t, Wm, g)
            if not (np.array_equal(fp["q"], f0["q"]) and np.array_equal(fm["q"], f0["q"])):
                continue
            fd = (Lp - Lm) / (2 * h)
            assert dW[i, j] == pytest.approx(fd, rel=1e-5, abs=1e-8)
            checked += 1
    for b in range(t.shape[0]):
        for j in range(t.shape[1]):
            x = t[b, j] * M
            if abs(x - round(x)) < 1e-3:
                continue  # too close to a grid point (one-sided derivative)
            tp, tmn = t.copy(), t.copy()
            tp[b, j] += h
            tmn[b, j] -= h
            Lp, fp = _loss(p, tp, W, g)
            Lm, fm = _loss(p, tmn, W, g)
            if not (np.array_equal(fp["q"], f0["q"]) and np.array_equal(fm["q"], f0["q"])):
                continue
            fd = (Lp - Lm) / (2 * h)
            assert dt[b, j] == pytest.approx(fd, rel=1e-5, abs=1e-8)
            checked += 1
    assert checked > 30


def test_backward_row_selection_and_linearity():
    p, t, W, g = _fd_setup(22, 1.0, 0.3)
    f = oracle.dstd_forward(p, t, W)
    dW, dt = oracle.dstd_backward(p, t, W, f, g)
    dW2, dt2 = oracle.dstd_backward(p, t, W, f, 2.5 * g, isel=[3, 1], bsel=[1])
    np.testing.assert_allclose(dW2, 2.5 * dW[[3, 1]], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(dt2, 2.5 * dt[[1]], rtol=1e-13, atol=1e-15)


# -------------------------------------------------------------------- conv --
def _conv_dense_matrix(cs):
    """Dense connectivity of a conv layer with event pooling (numpy, explicit)."""
    C_in, H, Wd, C_out, KH, KW, st, pad, pool = (cs[k] for k in
                                                 ("C_in", "H", "W", "C_out", "KH", "KW", "stride", "pad", "pool_in"))
    Hp, Wp, P = (H // 2, Wd // 2, 4) if pool == 2 else ((1, 1, H * Wd) if pool == 0 else (H, Wd, 1))
    Ho, Wo = (Hp + 2 * pad - KH) // st + 1, (Wp + 2 * pad - KW) // st + 1
    idx = []  # (out index, in index, weight index, factor)
    for co in range(C_out):
        for oy in range(Ho):
            for ox in range(Wo):
                o = (co * Ho + oy) * Wo + ox
                for ci in range(C_in):
                    for ky in range(KH):
                        for kx in range(KW):
                            py, px = oy * st + ky - pad, ox * st + kx - pad
                            if not (0 <= py < Hp and 0 <= px < Wp):
                                continue
                            if pool == 2:
                                cells = [(2 * py + a, 2 * px + b) for a in range(2) for b in range(2)]
                            elif pool == 0:
                                cells = [(y, x) for y in range(H) for x in range(Wd)]
                            else:
                                cells = [(py, px)]
                            for (y, x) in cells:
                                idx.append((o, (ci * H + y) * Wd + x, ((co * C_in + ci) * KH + ky) * KW + kx, 1.0 / P))
    return idx, C_out * Ho * Wo, C_in * H * Wd, (Ho, Wo)


@pytest.mark.parametrize("cs", [
    dict(C_in=2, H=6, W=5, C_out=3, KH=3, KW=3, stride=1, pad=1, pool_in=1),
    dict(C_in=2, H=7, W=7, C_out=3, KH=3, KW=3, stride=2, pad=1, pool_in=1),
    dict(C_in=3, H=8, W=6, C_out=2, KH=3, KW=3, stride=1, pad=1, pool_in=2),
    dict(C_in=4, H=3, W=3, C_out=5, KH=1, KW=1, stride=1, pad=0, pool_in=0),
])
def test_conv_equals_dense_layer_with_conv_connectivity(cs):
    rng = np.random.default_rng(31)
    p = _p(1.0, 0.3, M=8)
    B = 2
    nin = cs["C_in"] * cs["H"] * cs["W"]
    t = rng.random((B, nin))
    fan = cs["C_in"] * cs["KH"] * cs["KW"]
    Wc = (6.0 / fan) * (1 + 0.3 * math.sqrt(fan) * rng.standard_normal((cs["C_out"], cs["C_in"], cs["KH"], cs["KW"])))
    if cs["pool_in"] == 0:
        Wc *= 3.0
    idx, nout, nin2, (Ho, Wo) = _conv_dense_matrix(cs)
    Wd = np.zeros((nout, nin))
    for o, j, wi, fac in idx:
        Wd[o, j] += Wc.reshape(-1)[wi] * fac
    fc = oracle.conv_forward(p, cs, t.reshape(B, cs["C_in"], cs["H"], cs["W"]), Wc)
    fd = oracle.dstd_forward(p, t, Wd)
    np.testing.assert_array_equal(fc["q"].reshape(B, -1), fd["q"])
    assert (fd["q"] >= 0).sum() > 0
    np.testing.assert_allclose(fc["t_out"].reshape(B, -1), fd["t_out"], atol=1e-12)
    # conditioning outputs (pinned for dense layers in test_oracle_conditioning)
    for k in ("margin", "vabs", "emass"):
        np.testing.assert_allclose(fc[k].reshape(B, -1), fd[k], rtol=1e-10, atol=1e-13)
    g = rng.standard_normal(fc["t_out"].shape)
    rho = rng.random(g.shape) * 1e-3
    delta = rng.random(g.shape) * 1e-4
    dWc, dtc, dWca, dtca, dWce, dtce = oracle.conv_backward(
        p, cs, t.reshape(B, cs["C_in"], cs["H"], cs["W"]), Wc, fc, g, want_abs=True, err=(rho, delta))
    dWd, dtd, dWda, dtda, dWde, dtde = oracle.dstd_backward(
        p, t, Wd, fd, g.reshape(B, -1), want_abs=True, err=(rho.reshape(B, -1), delta.reshape(B, -1)))
    np.testing.assert_allclose(dtc.reshape(B, -1), dtd, rtol=1e-10, atol=1e-12)
    # each (output, input) pair is reached by one tap, so the |term| and the
    # error-weighted sums agree too
    np.testing.assert_allclose(dtca.reshape(B, -1), dtda, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dtce.reshape(B, -1), dtde, rtol=1e-10, atol=1e-15)
    ref = np.zeros(Wc.size)
    ref_abs = np.zeros(Wc.size)
    ref_err = np.zeros(Wc.size)
    for o, j, wi, fac in idx:
        ref[wi] += dWd[o, j] * fac
        ref_abs[wi] += dWda[o, j] * fac
        ref_err[wi] += dWde[o, j] * fac
    np.testing.assert_allclose(dWc.reshape(-1), ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dWca.reshape(-1), ref_abs, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dWce.reshape(-1), ref_err, rtol=1e-10, atol=1e-15)
    assert (dWce > 0).any()
    assert (dWca.reshape(-1) >= np.abs(dWc.reshape(-1)) - 1e-15).all()
