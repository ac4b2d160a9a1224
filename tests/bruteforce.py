"""Brute-force integration of the LIF ODE (Eq. (LIF_model_TTFS)) with scipy.

Independent of the spike kernel K and of the oracle: the two linear ODEs
dv/dt = -v/tau_v + I, dI/dt = -I/tau_I are integrated numerically (DOP853,
tight tolerances) between input impulses, each impulse adding its weight to I.
Used to pin the oracle's kernel, DSTD events and interval solver.
"""
import numpy as np
from scipy.integrate import solve_ivp


def _rhs(tau_v, tau_i):
    def f(t, y):
        return [-y[0] / tau_v + y[1], -y[1] / tau_i]
    return f


def simulate(tau_v, tau_i, times, weights, t_end, theta=None, query=(), rtol=1e-12, atol=1e-14):
    """Integrate from the first impulse to t_end.

    Returns (first time v >= theta or inf, dict query_time -> v(query_time)).
    Impulses at equal times are merged. Query times are sampled just after the
    impulses scheduled at the same time (v is continuous, so this is v(t)).
    """
    times = np.asarray(times, dtype=float)
    weights = np.asarray(weights, dtype=float)
    order = np.argsort(times, kind="stable")
    times, weights = times[order], weights[order]
    keep = np.isfinite(times)
    times, weights = times[keep], weights[keep]
    f = _rhs(tau_v, tau_i)
    query = sorted(set(float(q) for q in query))
    vals = {}
    fire = np.inf
    y = np.array([0.0, 0.0])
    t = -np.inf
    if len(times):
        t = times[0]
    for q in query:
        if len(times) == 0 or q < times[0]:
            vals[q] = 0.0
    uniq = np.unique(times)
    for k, tk in enumerate(uniq):
        y = y.copy()
        y[1] += weights[times == tk].sum()
        t_next = uniq[k + 1] if k + 1 < len(uniq) else t_end
        if t_next <= tk:
            continue
        qs = [q for q in query if tk <= q < t_next or (k + 1 == len(uniq) and q == t_end)]
        ev = None
        if theta is not None and not np.isfinite(fire):
            def ev(tt, yy):
                return yy[0] - theta
            ev.direction = 1
            ev.terminal = False
        sol = solve_ivp(f, (tk, t_next), y, method="DOP853", rtol=rtol, atol=atol,
                        t_eval=qs if qs else None, events=ev, dense_output=False)
        for qq, vv in zip(qs, sol.y[0] if qs else []):
            vals[qq] = float(vv)
        if theta is not None and not np.isfinite(fire):
            if y[0] >= theta:
                fire = tk
            elif sol.t_events and len(sol.t_events[0]):
                fire = float(sol.t_events[0][0])
        y = sol.y[:, -1] if not qs else _final(f, tk, t_next, y, rtol, atol)
        t = t_next
    return fire, vals


def _final(f, a, b, y, rtol, atol):
    sol = solve_ivp(f, (a, b), y, method="DOP853", rtol=rtol, atol=atol)
    return sol.y[:, -1]


def simulate_reset(tau_v, tau_i, times, weights, t_end, theta, n_spikes, rtol=1e-12, atol=1e-14):
    """The same ODE with the multi-spike reset: when v reaches theta the time
    is recorded and v is set to 0 while I carries on. Returns the first
    n_spikes spike times (fewer if the neuron stops firing before t_end)."""
    times = np.asarray(times, dtype=float)
    weights = np.asarray(weights, dtype=float)
    keep = np.isfinite(times)
    times, weights = times[keep], weights[keep]
    f = _rhs(tau_v, tau_i)
    uniq = np.unique(times)
    spikes = []
    y = np.array([0.0, 0.0])

    def ev(tt, yy):
        return yy[0] - theta
    ev.direction = 1
    ev.terminal = True
    for k, tk in enumerate(uniq):
        y = y.copy()
        y[1] += weights[times == tk].sum()
        t_next = uniq[k + 1] if k + 1 < len(uniq) else t_end
        t = tk
        while t < t_next and len(spikes) < n_spikes:
            sol = solve_ivp(f, (t, t_next), y, method="DOP853", rtol=rtol, atol=atol, events=ev)
            if sol.status == 1 and len(sol.t_events[0]):
                ts = float(sol.t_events[0][0])
                spikes.append(ts)
                y = np.array([0.0, sol.y_events[0][0][1]])
                t = ts
            else:
                y = sol.y[:, -1]
                t = t_next
        if len(spikes) >= n_spikes:
            break
    return spikes
