"""Pins of the oracle's exact spike-time path (App. A, Alg. 1, Eq. (timing_exact))
and of its gradients.

The gradients come from the implicit function theorem over the causal set of
the crossing interval. They are checked against routes that share nothing with
that formula: central finite differences of the exact forward pass, and the
hand-differentiated closed forms of the (inf, inf) and (inf, tau) rows.
"""
import math

import numpy as np
import pytest

import oracle

INF = math.inf
ROWS = [(1.0, 0.3), (1.0, 0.5), (0.4, 0.2), (2.0, 0.4), (0.5, 0.5), (INF, 0.3), (0.3, INF),
        (INF, INF)]


def _p(tm, ts, theta=1.0, t_max=INF):
    return dict(tau_m=tm, tau_s=ts, threshold=theta, t_max=t_max)


def _layer(tm, ts, seed, B=3, N_in=7, N_out=5):
    """Tiny layer whose neurons mostly fire: inputs in [0, 1], weights mostly
    positive and scaled to the kernel's peak."""
    rng = np.random.default_rng(seed)
    t = rng.uniform(0.0, 1.0, (B, N_in))
    t[0, 1] = INF  # one silent input
    tv, ti = max(tm, ts), min(tm, ts)
    if math.isinf(tv) and math.isinf(ti):
        kpk = 1.0
    elif math.isinf(tv):
        kpk = ti
    elif tv == ti:
        kpk = tv / math.e
    else:
        kpk = ti * (ti / tv) ** (ti / (tv - ti))
    W = rng.uniform(-0.3, 1.0, (N_out, N_in)) * (7.0 / (N_in * kpk))
    return t, W


def _loss(p, t, W, g):
    f = oracle.exact_forward(p, t, W)
    fired = f["q"] >= 0
    return float(np.sum(np.where(fired, g * np.where(fired, f["t_out"], 0.0), 0.0))), f["q"]


@pytest.mark.parametrize("tm,ts", ROWS)
def test_exact_gradients_match_finite_differences(tm, ts):
    p = _p(tm, ts)
    t, W = _layer(tm, ts, seed=11)
    rng = np.random.default_rng(5)
    g = rng.normal(size=(t.shape[0], W.shape[0]))
    f = oracle.exact_forward(p, t, W)
    assert (f["q"] >= 0).mean() >= 0.5
    gr = oracle.exact_backward(p, t, W, f, g)
    h = 1e-6
    checked = 0
    for which, base, grad in (("W", W, gr["grad_W"]), ("t", t, gr["grad_t_in"])):
        for idx in np.ndindex(base.shape):
            if not np.isfinite(base[idx]):
                assert grad[idx] == 0.0
                continue
            xp, xm = base.copy(), base.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = (xp, W) if which == "t" else (t, xp)
            args_m = (xm, W) if which == "t" else (t, xm)
            lp, qp = _loss(p, *args_p, g)
            lm, qm = _loss(p, *args_m, g)
            if not (np.array_equal(qp, f["q"]) and np.array_equal(qm, f["q"])):
                continue  # the causal set changes inside +-h: a kink
            fd = (lp - lm) / (2 * h)
            assert grad[idx] == pytest.approx(fd, rel=1e-6, abs=1e-7), (which, idx)
            checked += 1
    assert checked >= 0.9 * (W.size + np.isfinite(t).sum())


def test_exact_gradients_no_leak_closed_form():
    """(inf, inf): Eq. (spike_no_leak) t = (V_th + sum_S w_j t_j) / sum_S w_j, so
    dt/dw_j = (t_j - t) / sum_S w and dt/dt_j = w_j / sum_S w on the causal set."""
    p = _p(INF, INF, theta=0.7)
    t = np.array([[0.1, 0.5, 0.2, 0.9, 0.35]])
    W = np.array([[0.8, 1.1, 0.6, 2.0, -0.3]])
    f = oracle.exact_forward(p, t, W)
    k = int(f["q"][0, 0])
    order = np.argsort(t[0])
    S = order[: k + 1]
    sw = W[0, S].sum()
    t_hat = (0.7 + (W[0, S] * t[0, S]).sum()) / sw
    assert f["t_out"][0, 0] == pytest.approx(t_hat, rel=1e-14)
    gr = oracle.exact_backward(p, t, W, f, np.ones((1, 1)))
    dW = np.zeros(5)
    dt = np.zeros(5)
    dW[S] = (t[0, S] - t_hat) / sw
    dt[S] = W[0, S] / sw
    np.testing.assert_allclose(gr["grad_W"][0], dW, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(gr["grad_t_in"][0], dt, rtol=1e-12, atol=1e-15)


def test_exact_gradients_inf_tau_closed_form():
    """(inf, tau): Table "tab:spike_timing" gives t = tau ln(a / (b - V_th/tau)) with
    a = sum_S w_j e^{t_j/tau}, b = sum_S w_j; differentiating by hand,
    dt/dw_j = tau (e^{t_j/tau}/a - 1/(b - V_th/tau)), dt/dt_j = w_j e^{t_j/tau}/a."""
    tau, th = 0.4, 0.5
    p = _p(INF, tau, theta=th)
    t = np.array([[0.05, 0.3, 0.12, 0.6, 0.45, 0.2]])
    W = np.array([[1.2, 0.9, 1.0, 1.5, -0.2, 0.4]])
    f = oracle.exact_forward(p, t, W)
    k = int(f["q"][0, 0])
    assert k >= 1
    S = np.argsort(t[0])[: k + 1]
    a = (W[0, S] * np.exp(t[0, S] / tau)).sum()
    b = W[0, S].sum()
    t_hat = tau * math.log(a / (b - th / tau))
    assert f["t_out"][0, 0] == pytest.approx(t_hat, rel=1e-13)
    gr = oracle.exact_backward(p, t, W, f, np.ones((1, 1)))
    dW = np.zeros(6)
    dt = np.zeros(6)
    dW[S] = tau * (np.exp(t[0, S] / tau) / a - 1.0 / (b - th / tau))
    dt[S] = W[0, S] * np.exp(t[0, S] / tau) / a
    np.testing.assert_allclose(gr["grad_W"][0], dW, rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(gr["grad_t_in"][0], dt, rtol=1e-11, atol=1e-14)


@pytest.mark.parametrize("tm,ts", [(1.0, 0.3), (INF, INF)])
def test_exact_interval_index_is_causal_count(tm, ts):
    """q is the last position (ascending order) of the inputs at or before the
    spike; equal times share one interval, so q ends a group of ties."""
    p = _p(tm, ts)
    t, W = _layer(tm, ts, seed=3, B=4, N_in=9, N_out=6)
    t[1, 2] = t[1, 5]  # a tie
    t[2, :3] = 0.5  # a group of three
    f = oracle.exact_forward(p, t, W)
    for b in range(t.shape[0]):
        for i in range(W.shape[0]):
            q = f["q"][b, i]
            if q < 0:
                assert np.isinf(f["t_out"][b, i]) and f["slope"][b, i] == 0.0
                continue
            n_causal = int(np.sum(np.isfinite(t[b]) & (t[b] <= f["t_out"][b, i])))
            assert q == n_causal - 1
            assert f["slope"][b, i] > 0.0
            assert f["margin"][b, i] >= 0.0


def test_exact_backward_silent_and_zero_upstream():
    """Silent neurons and zero upstream gradients give zero gradients; the
    backward pass is linear in the upstream gradient."""
    p = _p(1.0, 0.3)
    t, W = _layer(1.0, 0.3, seed=8, B=3, N_in=8, N_out=4)
    W[2] = -np.abs(W[2])  # an inhibitory neuron never fires
    f = oracle.exact_forward(p, t, W)
    assert np.all(f["q"][:, 2] < 0)
    z = oracle.exact_backward(p, t, W, f, np.zeros((3, 4)))
    assert not z["grad_W"].any() and not z["grad_t_in"].any()
    rng = np.random.default_rng(1)
    g1, g2 = rng.normal(size=(3, 4)), rng.normal(size=(3, 4))
    a = oracle.exact_backward(p, t, W, f, g1)
    b = oracle.exact_backward(p, t, W, f, g2)
    c = oracle.exact_backward(p, t, W, f, 2.0 * g1 - g2)
    assert not a["grad_W"][2].any()
    np.testing.assert_allclose(c["grad_W"], 2 * a["grad_W"] - b["grad_W"], atol=1e-13)
    np.testing.assert_allclose(c["grad_t_in"], 2 * a["grad_t_in"] - b["grad_t_in"], atol=1e-13)
