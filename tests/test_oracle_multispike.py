"""Pins of the oracle's multi-spike DSTD (App. "multi-spikes", Eq.
(Vmem_multiSpikes) and its DSTD form): the first spike is the TTFS spike;
all spikes match a numerical integration of the LIF ODE driven by the
weighted events, with v reset to 0 at each spike and the current kept; the
gradients match central finite differences of the forward pass."""
import math

import numpy as np
import pytest

import oracle
from tests.bruteforce import simulate_reset

TAU = [(1.0, 0.3), (1.0, 0.5), (0.5, 0.5), (math.inf, 0.3), (math.inf, math.inf)]


def _p(tm, ts, M=12, t0=0.0, theta=1.0):
    return dict(tau_m=tm, tau_s=ts, threshold=theta, M=M, t0=t0, dt=1.0 / M, t_max=math.inf)


def _case(seed, B, N_in, F_in, N_out, scale):
    rng = np.random.default_rng(seed)
    t = np.sort(rng.random((B, N_in, F_in)), axis=2)
    t[0, 0, -1] = np.inf  # an input that fires fewer times
    W = rng.uniform(-0.2, 1.0, (N_out, N_in)) * scale
    return t, W


def _scale(tm, ts):
    return {(math.inf, math.inf): 0.25, (math.inf, 0.3): 0.8}.get((tm, ts), 2.0)


@pytest.mark.parametrize("tm,ts", TAU)
def test_first_spike_is_the_ttfs_spike(tm, ts):
    p = _p(tm, ts)
    t, W = _case(1, 3, 20, 2, 6, _scale(tm, ts))
    ms = oracle.ms_forward(p, t, W, 3)
    # every input spike is an input of its own with its neuron's weights
    tt = oracle.dstd_forward(p, t.reshape(3, -1), np.repeat(W, 2, axis=1))
    assert np.array_equal(ms["q"][:, :, 0], tt["q"])
    fired = tt["q"] >= 0
    assert fired.mean() > 0.5
    np.testing.assert_allclose(ms["t_out"][:, :, 0][fired], tt["t_out"][fired], rtol=0, atol=1e-13)
    np.testing.assert_allclose(ms["slope"][:, :, 0][fired], tt["slope"][fired], rtol=1e-12)


@pytest.mark.parametrize("tm,ts", TAU)
def test_spikes_match_ode_with_reset(tm, ts):
    """Impulses w^_m at T_m drive the ODE (Eq. (LIF_model_TTFS)); at each
    crossing v is set to 0 and I kept (the reset of App. "multi-spikes")."""
    p = _p(tm, ts)
    t, W = _case(2, 2, 15, 2, 4, _scale(tm, ts))
    F = 4
    ms = oracle.ms_forward(p, t, W, F)
    what = oracle.dstd_forward(p, t.reshape(2, -1), np.repeat(W, 2, axis=1), want_what=True)["what"]
    T = p["t0"] + p["dt"] * np.arange(p["M"] + 1)
    tv, ti = max(tm, ts), min(tm, ts)
    n_multi = 0
    for b in range(2):
        for i in range(4):
            ref = simulate_reset(tv, ti, T, what[b, :, i], T[-1] + 3.0, 1.0, F)
            got = [x for x in ms["t_out"][b, i] if np.isfinite(x) and x < T[-1] + 3.0]
            assert len(got) == len(ref), (b, i, got, ref)
            np.testing.assert_allclose(got, ref, rtol=0, atol=1e-8)
            n_multi += len(ref) >= 2
    assert n_multi >= 2


@pytest.mark.parametrize("tm,ts", [(1.0, 0.3), (0.5, 0.5), (math.inf, 0.3), (math.inf, math.inf)])
def test_gradients_match_finite_differences(tm, ts):
    """L = sum over spikes of g_k t_k; the reset chain (t_k depends on t_{k-1})
    is part of what the differences see."""
    p = _p(tm, ts)
    t, W = _case(3, 2, 8, 2, 3, _scale(tm, ts))
    F = 3
    f = oracle.ms_forward(p, t, W, F)
    assert (f["q"][:, :, 1] >= 0).sum() >= 2  # second spikes exist
    g = np.random.default_rng(4).standard_normal(f["t_out"].shape)
    gr = oracle.ms_backward(p, t, W, f, np.where(f["q"] >= 0, g, 0.0))
    h = 1e-6

    def loss(tt, WW):
        r = oracle.ms_forward(p, tt, WW, F)
        return float(np.sum(np.where(r["q"] >= 0, g * np.where(r["q"] >= 0, r["t_out"], 0), 0))), r["q"]

    checked = 0
    for which, base, grad in (("W", W, gr["grad_W"]), ("t", t, gr["grad_t_in"])):
        for idx in np.ndindex(base.shape):
            if not np.isfinite(base[idx]):
                assert grad[idx] == 0.0
                continue
            xp, xm = base.copy(), base.copy()
            xp[idx] += h
            xm[idx] -= h
            lp, qp = loss(xp, W) if which == "t" else loss(t, xp)
            lm, qm = loss(xm, W) if which == "t" else loss(t, xm)
            if not (np.array_equal(qp, f["q"]) and np.array_equal(qm, f["q"])):
                continue
            x = base[idx] if which == "t" else None
            if x is not None and abs(x * p["M"] - round(x * p["M"])) < 1e-4:
                continue  # the event derivative jumps at a grid point
            fd = (lp - lm) / (2 * h)
            assert grad[idx] == pytest.approx(fd, rel=1e-5, abs=1e-7), (which, idx)
            checked += 1
    assert checked >= 0.8 * (W.size + np.isfinite(t).sum())


def test_silent_and_single_spike_cases():
    p = _p(1.0, 0.3)
    t, W = _case(5, 2, 10, 2, 3, 2.0)
    W[1] = -np.abs(W[1])
    f = oracle.ms_forward(p, t, W, 3)
    assert np.all(f["q"][:, 1] == -1) and np.all(np.isinf(f["t_out"][:, 1]))
    z = oracle.ms_backward(p, t, W, f, np.zeros(f["t_out"].shape))
    assert not z["grad_W"].any() and not z["grad_t_in"].any()
    # spikes are increasing and later spikes exist only after earlier ones
    for b in range(2):
        for i in range(3):
            q = f["q"][b, i]
            k = int((q >= 0).sum())
            assert np.all(q[:k] >= 0) and np.all(q[k:] == -1)
            assert np.all(np.diff(f["t_out"][b, i, :k]) > 0)
