"""Pins of the oracle's conditioning outputs, which decide what the GPU
parity tests check: the ambiguity margin, the term scales vabs and emass of
the forward, and the |term| and error-weighted sums of the backward.

Each is recomputed here by another route:
- margin and the crossing interval: direct superposition
  v^(t) = sum_m w^_m K(t - T_m) (or sum_j w_j K(t - t_j) for the exact
  path) sampled densely on every interval with the maxima refined by Brent's
  method, instead of the oracle's prefix sums and closed-form critical point;
- vabs, emass and the backward sums: NumPy sums over the dense event tensor
  s[b, m, j] and the spike kernel, instead of the oracle's per-neuron loops.
K is the oracle's (pinned against the LIF ODE in test_oracle_pins); K' is
its central difference. A planted mistake in any of these outputs fails one
of the tests below (tests/test_oracle_mutations.py plants them).
"""
import math

import numpy as np
import pytest
from scipy.optimize import minimize_scalar

import oracle

ROWS = [(1.0, 0.3), (1.0, 0.5), (2.0, 0.4), (0.5, 0.5), (math.inf, 0.4), (math.inf, math.inf)]


def _p(tm, ts, M=8, t0=0.0, dt=None, theta=1.0, t_max=math.inf):
    return dict(tau_m=tm, tau_s=ts, threshold=theta, M=M, t0=t0, dt=(1.0 / M if dt is None else dt),
                t_max=t_max)


def _canon(p):
    return max(p["tau_m"], p["tau_s"]), min(p["tau_m"], p["tau_s"])


def _K(tv, ti, u):
    u = np.asarray(u, dtype=np.float64)
    return np.vectorize(lambda x: oracle.kernel(tv, ti, float(x)), otypes=[float])(u)


def _Kd(tv, ti, u, h=1e-6):
    """K'(u) for u >= 0 (right derivative at 0) by central / one-sided differences."""
    u = np.asarray(u, dtype=np.float64)
    c = (_K(tv, ti, u + h) - _K(tv, ti, u - h)) / (2 * h)
    r = (-3 * _K(tv, ti, u) + 4 * _K(tv, ti, u + h) - _K(tv, ti, u + 2 * h)) / (2 * h)
    return np.where(u >= h, c, r)


def _layer(rng, tm, ts, B=3, N_in=24, N_out=10, M=8, k=None):
    p = _p(tm, ts, M=M)
    t = rng.random((B, N_in))
    t[rng.random((B, N_in)) < 0.1] = np.inf
    tv, ti = _canon(p)
    if k is None:
        peak = max(_K(tv, ti, np.linspace(0, 1, 200)))
        k = 1.6 / peak
    W = (k / N_in) * (1 + 0.6 * math.sqrt(N_in) * rng.standard_normal((N_out, N_in)))
    return p, t, W


# ------------------------------------------------------------- DSTD forward --
def _bruteforce_scan(p, what_row):
    """Crossing interval and margin of one neuron from direct superposition."""
    tv, ti = _canon(p)
    M, th = int(p["M"]), p["threshold"]
    T = p["t0"] + p["dt"] * np.arange(M + 1)
    far = T[M] + 30.0 * (tv if math.isfinite(tv) else 1.0)

    def v(t):
        t = np.atleast_1d(np.asarray(t, dtype=np.float64))
        out = np.zeros_like(t)
        for m in range(M + 1):
            out += what_row[m] * _K(tv, ti, t - T[m]) * (t >= T[m])
        return out

    pre = math.inf
    for q in range(M + 1):
        lo = T[q]
        hi = T[q + 1] if q < M else min(p["t_max"], far)
        xs = np.linspace(lo, hi, 257)
        vs = v(xs)
        k = int(np.argmax(vs))
        a, b = xs[max(k - 1, 0)], xs[min(k + 1, len(xs) - 1)]
        peak = float(vs[k])
        if b > a:
            r = minimize_scalar(lambda x: -v(x)[0], bounds=(a, b), method="bounded",
                                options=dict(xatol=1e-13))
            peak = max(peak, -float(r.fun))
        if q == M and not math.isfinite(p["t_max"]) and math.isinf(tv) and math.isinf(ti):
            # (inf, inf): v is linear on the open last interval, unbounded when rising
            slope_last = float(what_row[: M + 1].sum())
            if slope_last > 0:
                peak = math.inf
        if peak >= th:
            m = min(pre, abs(peak - th), abs(float(v(lo)[0]) - th))
            if q < M:
                m = min(m, abs(float(v(hi)[0]) - th))
            return q, m
        pre = min(pre, th - peak)
    return -1, pre


@pytest.mark.parametrize("tm,ts", ROWS)
def test_dstd_margin_and_interval_match_superposition(tm, ts):
    rng = np.random.default_rng(5)
    p, t, W = _layer(rng, tm, ts, B=2, N_in=16, N_out=12)
    f = oracle.dstd_forward(p, t, W, want_what=True)
    n_fired = 0
    for b in range(t.shape[0]):
        for i in range(W.shape[0]):
            q, m = _bruteforce_scan(p, f["what"][b, :, i])
            assert q == f["q"][b, i]
            assert f["margin"][b, i] == pytest.approx(m, abs=1e-9, rel=1e-7)
            n_fired += q >= 0
    assert n_fired > 0


def test_dstd_margin_earlier_interval_term_binds():
    """A neuron whose potential nearly reaches V_th in an earlier interval and
    crosses later: the margin is that earlier near-miss (theta - peak)."""
    p = _p(1.0, 0.3, M=8)
    tv, ti = _canon(p)
    kmax = ti * (ti / tv) ** (ti / (tv - ti))
    # input 0 on a grid point alone peaks just below theta (at t ~ 0.52); an
    # input after that peak makes the neuron cross later
    t = np.array([[0.0, 0.875]])
    W = np.array([[(1 - 3e-3) / kmax, 2.0 / kmax]])
    f = oracle.dstd_forward(p, t, W, want_what=True)
    q, m = _bruteforce_scan(p, f["what"][0, :, 0])
    assert q == f["q"][0, 0] and q >= 4
    assert m == pytest.approx(3e-3, rel=1e-3)
    assert f["margin"][0, 0] == pytest.approx(m, abs=1e-9)


def test_dstd_margin_right_end_term_binds():
    """A crossing interval whose potential peaks well above V_th and decays to
    just above it at the interval's right grid point: the margin is
    |v(T_q*+1) - theta|."""
    p = _p(0.4, 0.2, M=2, dt=0.5)
    tv, ti = _canon(p)
    k_end = oracle.kernel(tv, ti, 0.5)
    t = np.array([[0.0]])
    W = np.array([[(1 + 2e-3) / k_end]])
    f = oracle.dstd_forward(p, t, W, want_what=True)
    q, m = _bruteforce_scan(p, f["what"][0, :, 0])
    assert q == f["q"][0, 0] == 0
    assert m == pytest.approx(2e-3, rel=1e-6)
    assert f["margin"][0, 0] == pytest.approx(m, abs=1e-9)


@pytest.mark.parametrize("tm,ts", ROWS)
def test_dstd_vabs_and_emass_are_direct_sums(tm, ts):
    rng = np.random.default_rng(7)
    p, t, W = _layer(rng, tm, ts)
    tv, ti = _canon(p)
    f = oracle.dstd_forward(p, t, W)
    S, _ = oracle.dstd_events(p, t)  # [B, M+1, N_in]
    T = p["t0"] + p["dt"] * np.arange(p["M"] + 1)
    wabs = np.einsum("ij,bmj->bmi", np.abs(W), np.abs(S))  # [B, M+1, N_out]
    for b in range(t.shape[0]):
        for i in range(W.shape[0]):
            q = f["q"][b, i]
            last = q if q >= 0 else p["M"]
            em = wabs[b, : last + 1, i].sum()
            assert f["emass"][b, i] == pytest.approx(em, rel=1e-12, abs=1e-15)
            if q >= 0:
                va = (np.abs(_K(tv, ti, f["t_out"][b, i] - T[: q + 1])) * wabs[b, : q + 1, i]).sum()
                assert f["vabs"][b, i] == pytest.approx(va, rel=1e-12, abs=1e-15)
            else:
                assert f["vabs"][b, i] == 0.0
    assert (f["q"] >= 0).any()


# ------------------------------------------------------------ DSTD backward --
def _dense_G(p, f, g, rho, delta):
    tv, ti = _canon(p)
    B, N_out = f["q"].shape
    M = int(p["M"])
    T = p["t0"] + p["dt"] * np.arange(M + 1)
    G = np.zeros((B, M + 1, N_out))
    GE = np.zeros((B, M + 1, N_out))
    for b in range(B):
        for i in range(N_out):
            q = f["q"][b, i]
            if q < 0 or g[b, i] == 0:
                continue
            gam = -g[b, i] / f["slope"][b, i]
            u = f["t_out"][b, i] - T[: q + 1]
            G[b, : q + 1, i] = gam * _K(tv, ti, u)
            GE[b, : q + 1, i] = abs(gam) * (rho[b, i] * np.abs(_K(tv, ti, u)) +
                                            delta[b, i] * np.abs(_Kd(tv, ti, u)))
    return G, GE


@pytest.mark.parametrize("tm,ts", ROWS)
def test_dstd_backward_abs_and_error_sums_are_direct_sums(tm, ts):
    rng = np.random.default_rng(11)
    p, t, W = _layer(rng, tm, ts)
    f = oracle.dstd_forward(p, t, W)
    g = rng.standard_normal(f["q"].shape)
    rho = rng.random(f["q"].shape) * 1e-3
    delta = rng.random(f["q"].shape) * 1e-4
    dW, dt, dWa, dta, dWe, dte = oracle.dstd_backward(p, t, W, f, g, want_abs=True, err=(rho, delta))
    S, dS = oracle.dstd_events(p, t)
    G, GE = _dense_G(p, f, g, rho, delta)
    # dW[i, j] = sum_b sum_m G[b,m,i] s[b,m,j]; dt[b, j] = sum_m sum_i G[b,m,i] w_ij ds[b,m,j]
    np.testing.assert_allclose(dW, np.einsum("bmi,bmj->ij", G, S), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(dWa, np.einsum("bmi,bmj->ij", np.abs(G), np.abs(S)), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dWe, np.einsum("bmi,bmj->ij", GE, np.abs(S)), rtol=1e-6, atol=1e-15)
    np.testing.assert_allclose(dt, np.einsum("bmi,ij,bmj->bj", G, W, dS), rtol=1e-9, atol=1e-13)
    np.testing.assert_allclose(dta, np.einsum("bmi,ij,bmj->bj", np.abs(G), np.abs(W), np.abs(dS)),
                               rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dte, np.einsum("bmi,ij,bmj->bj", GE, np.abs(W), np.abs(dS)),
                               rtol=1e-6, atol=1e-15)
    assert (dWe > 0).any() and (dte > 0).any()


def test_dstd_error_sums_scale_linearly_in_rho_and_delta():
    rng = np.random.default_rng(12)
    p, t, W = _layer(rng, 1.0, 0.3)
    f = oracle.dstd_forward(p, t, W)
    g = rng.standard_normal(f["q"].shape)
    z = np.zeros(f["q"].shape)
    _, _, dWa, dta, dWe1, dte1 = oracle.dstd_backward(p, t, W, f, g, want_abs=True, err=(z + 1.0, z))
    # rho = 1, delta = 0: the error sum is the |term| sum itself
    np.testing.assert_allclose(dWe1, dWa, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dte1, dta, rtol=1e-12, atol=1e-15)
    _, _, dWe2, dte2 = oracle.dstd_backward(p, t, W, f, g, err=(z + 2.0, z))
    np.testing.assert_allclose(dWe2, 2 * dWe1, rtol=1e-12, atol=1e-15)


# -------------------------------------------------------------- exact path --
def _bruteforce_exact(p, t_row, w_row):
    tv, ti = _canon(p)
    th = p["threshold"]
    keep = np.isfinite(t_row)
    ts, ws = t_row[keep], w_row[keep]
    order = np.argsort(ts, kind="stable")
    ts, ws = ts[order], ws[order]
    far = (ts[-1] if len(ts) else 0.0) + 30.0 * (tv if math.isfinite(tv) else 1.0)

    def v(t):
        t = np.atleast_1d(np.asarray(t, dtype=np.float64))
        out = np.zeros_like(t)
        for tj, wj in zip(ts, ws):
            out += wj * _K(tv, ti, t - tj) * (t >= tj)
        return out

    pre = math.inf
    uniq = np.unique(ts)
    for k, lo in enumerate(uniq):
        hi = uniq[k + 1] if k + 1 < len(uniq) else min(p["t_max"], far)
        xs = np.linspace(lo, hi, 257)
        vs = v(xs)
        kk = int(np.argmax(vs))
        a, b = xs[max(kk - 1, 0)], xs[min(kk + 1, len(xs) - 1)]
        peak = float(vs[kk])
        if b > a:
            r = minimize_scalar(lambda x: -v(x)[0], bounds=(a, b), method="bounded",
                                options=dict(xatol=1e-13))
            peak = max(peak, -float(r.fun))
        if peak >= th:
            m = min(pre, abs(peak - th), abs(float(v(lo)[0]) - th))
            if k + 1 < len(uniq):
                m = min(m, abs(float(v(hi)[0]) - th))
            causal = ts <= lo
            return True, m, causal, ts, ws
        pre = min(pre, th - peak)
    return False, pre, np.ones(len(ts), dtype=bool), ts, ws


@pytest.mark.parametrize("tm,ts", [(1.0, 0.3), (0.5, 0.5), (math.inf, 0.4)])
def test_exact_margin_vabs_emass_match_direct_sums(tm, ts):
    rng = np.random.default_rng(9)
    p, t, W = _layer(rng, tm, ts, B=2, N_in=10, N_out=8)
    tv, ti = _canon(p)
    f = oracle.exact_forward(p, t, W)
    fired = 0
    for b in range(t.shape[0]):
        for i in range(W.shape[0]):
            hit, m, causal, tsrt, wsrt = _bruteforce_exact(p, t[b], W[i])
            assert hit == (f["q"][b, i] >= 0)
            assert f["margin"][b, i] == pytest.approx(m, abs=1e-9, rel=1e-7)
            em = np.abs(wsrt[causal]).sum() if hit else np.abs(wsrt).sum()
            assert f["emass"][b, i] == pytest.approx(em, rel=1e-12)
            if hit:
                fired += 1
                va = np.abs(wsrt[causal] * _K(tv, ti, f["t_out"][b, i] - tsrt[causal])).sum()
                assert f["vabs"][b, i] == pytest.approx(va, rel=1e-12)
    assert fired > 0


def test_exact_margin_earlier_interval_term_binds():
    """Exact path: a first input alone peaks just below V_th, a later input
    makes the neuron cross; the margin is the earlier near-miss."""
    p = _p(1.0, 0.3)
    tv, ti = _canon(p)
    kmax = ti * (ti / tv) ** (ti / (tv - ti))
    t = np.array([[0.0, 0.875]])
    W = np.array([[(1 - 3e-3) / kmax, 2.0 / kmax]])
    f = oracle.exact_forward(p, t, W)
    hit, m, _, _, _ = _bruteforce_exact(p, t[0], W[0])
    assert hit and f["q"][0, 0] == 1
    assert m == pytest.approx(3e-3, rel=1e-3)
    assert f["margin"][0, 0] == pytest.approx(m, abs=1e-9)


@pytest.mark.parametrize("tm,ts", [(1.0, 0.3), (math.inf, math.inf)])
def test_exact_backward_abs_and_error_sums_are_direct_sums(tm, ts):
    rng = np.random.default_rng(10)
    p, t, W = _layer(rng, tm, ts, B=2, N_in=10, N_out=8)
    tv, ti = _canon(p)
    k2 = (0.0 if math.isinf(tv) else 1.0 / tv) + (0.0 if math.isinf(ti) else 1.0 / ti)
    f = oracle.exact_forward(p, t, W)
    g = rng.standard_normal(f["q"].shape)
    rho = rng.random(g.shape) * 1e-3
    delta = rng.random(g.shape) * 1e-4
    r = oracle.exact_backward(p, t, W, f, g, err=(rho, delta))
    B, N_in = t.shape
    N_out = W.shape[0]
    dWa = np.zeros((N_out, N_in)); dWe = np.zeros((N_out, N_in))
    dta = np.zeros((B, N_in)); dte = np.zeros((B, N_in))
    for b in range(B):
        for i in range(N_out):
            if f["q"][b, i] < 0:
                continue
            hit, _, causal, tsrt, _ = _bruteforce_exact(p, t[b], W[i])
            tl = tsrt[causal].max()
            gam = -g[b, i] / f["slope"][b, i]
            for j in range(N_in):
                if not (np.isfinite(t[b, j]) and t[b, j] <= tl):
                    continue
                u = f["t_out"][b, i] - t[b, j]
                K, Kd = _K(tv, ti, u), _Kd(tv, ti, u)
                dWa[i, j] += abs(gam * K)
                dWe[i, j] += abs(gam) * (rho[b, i] * abs(K) + delta[b, i] * abs(Kd))
                dta[b, j] += abs(gam * W[i, j] * Kd)
                dte[b, j] += abs(gam * W[i, j]) * (rho[b, i] * abs(Kd) + delta[b, i] * k2)
    np.testing.assert_allclose(r["grad_W_abs"], dWa, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r["grad_W_err"], dWe, rtol=1e-6, atol=1e-15)
    np.testing.assert_allclose(r["grad_t_in_abs"], dta, rtol=1e-6, atol=1e-15)
    np.testing.assert_allclose(r["grad_t_in_err"], dte, rtol=1e-6, atol=1e-15)
    assert (dWe > 0).any()
