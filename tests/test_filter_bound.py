"""The scan's interval filter before T_M (CPU only).

Between grid points the potential is v(u) = V e^{-u/tau_v} + I K(u) (the
state form of the interval analysis of Eq. (timing_DSTD)). The GPU scan skips
an interval [0, dt] unless

    max(V, v(dt)) + dt^2/8 (|V| / tau_v^2 + |I| max|K''|) >= theta / 1.0001,

with max|K''| on [0, dt] taken per kernel row (general: c / tau_I^2;
(tau, tau): 2/tau + dt/tau^2; (inf, tau): 1/tau; (inf, inf): 0). A crossing
is never skipped only if that expression bounds v on the whole interval.
This checks it by dense sampling of v, with K from the oracle's kernel, over
random states, interval lengths and every kernel row, including kernels much
faster than the interval (bumps inside it). The bound is conservative (its
curvature term is 2-3x the largest excess of v over its ends in these
cases); what is checked here is that it is never below the maximum.
"""
import math

import numpy as np
import pytest

import oracle

INF = math.inf


def _kpp(tv, ti, dt):
    """The filter's max |K''| on [0, dt] (canonical order tv >= ti)."""
    if math.isinf(ti):
        return 0.0
    if math.isinf(tv):
        return 1.0 / ti
    if tv == ti:
        return 2.0 / ti + dt / (ti * ti)
    return tv / (ti * (tv - ti))  # c / ti^2 with c = tv ti / (tv - ti)


ROWS = [(1.0, 0.5), (0.4, 0.2), (0.05, 0.02), (0.3, 0.3), (0.03, 0.03), (INF, 0.5), (INF, 0.02),
        (INF, INF)]


@pytest.mark.parametrize("tv,ti", ROWS, ids=[f"{a}-{b}" for a, b in ROWS])
def test_interval_filter_bounds_the_potential(tv, ti):
    rng = np.random.default_rng(7)
    kv = np.vectorize(lambda u: oracle.kernel(tv, ti, u))
    worst = -np.inf
    for dt in (1.0 / 8, 1.0 / 32, 0.5):
        u = np.linspace(0.0, dt, 2001)
        K = kv(u)
        ev = np.exp(-u / tv) if not math.isinf(tv) else np.ones_like(u)
        curv_v = 0.0 if math.isinf(tv) else dt * dt / 8.0 / (tv * tv)
        curv_i = dt * dt / 8.0 * _kpp(tv, ti, dt)
        # cases with the maximum inside the interval first (V = I tv makes
        # v'(0) = 0 and v concave there), then random states
        cases = ([] if math.isinf(tv) else [(I * tv, I) for I in (1.0, 5.0)]) + [
            (rng.uniform(-2.0, 2.0), rng.uniform(-6.0, 6.0) * (20.0 if ti < 0.1 else 1.0))
            for _ in range(300)]
        for V, I in cases:
            v = V * ev + I * K
            bound = max(V, v[-1]) + curv_v * abs(V) + curv_i * abs(I)
            scale = abs(V) + abs(I) * float(np.abs(K).max()) + 1.0
            assert v.max() <= bound + 1e-12 * scale, (tv, ti, dt, V, I, v.max(), bound)
            worst = max(worst, v.max() - max(V, v[-1]))
    # the curvature term is needed: some interval's maximum lies above both of
    # its ends (not on the monotone (inf, tau) and linear (inf, inf) rows)
    if not math.isinf(tv):
        assert worst > 0.0
