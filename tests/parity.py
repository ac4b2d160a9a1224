"""Comparison rules between the HIP path (fp32) and the fp64 oracle.

- Fire / no-fire and the interval index q must agree exactly outside the
  ambiguity set: neurons whose decision-relevant potentials lie within 1e-5
  of the threshold (the oracle's `margin`).
- Spike times must agree within 1e-5 of the time window outside the
  ambiguity set, except where fp32 conditioning makes that unattainable: the
  potential at the spike is a sum whose terms have magnitude `vabs`
  (oracle), so its fp32 rounding is about est_v = 2^-24 vabs and moves the
  time by est = est_v / |slope|. Every spike must satisfy
  |dt| <= max(1e-5 * window, 16 * est); the spikes beyond 1e-5 (the
  ill-conditioned bucket) are counted, reported and must stay below 0.5 %.
  Their upstream gradient is zeroed for the gradient checks, as is that of
  spikes with 16 * est > 1e-5 * window.
- Gradients: the upstream gradient of excluded neurons is zeroed on both sides
  before the backward pass; dW and dt_in must then agree within 1e-3 relative.
  Each element is a sum of many signed terms, so the absolute floor is
  1e-6 or KAPPA times the element's sum of |terms| (its conditioning: fp32
  rounding of the terms, and of the slope of each contributing spike, scales
  with that sum, not with the possibly cancelled result), whichever is larger.
"""
import numpy as np

TOL_T = 1e-5        # of the window
MARGIN = 1e-5       # |v - theta| ambiguity
COND = 16.0
MAX_BEYOND = 0.005
MAX_AMBIGUOUS = 0.01
GRAD_RTOL = 1e-3
GRAD_ATOL = 1e-6
KAPPA = 1e-4


def conditioning(orc):
    """Per-neuron fp32 time-error estimate 2^-24 * vabs / |slope| (inf if flat)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        est = 2.0 ** -24 * orc["vabs"] / np.abs(orc["slope"])
    return np.where(orc["q"] >= 0, est, 0.0)


def excluded(orc, n_in, window):
    """(ambiguous, gradient-sensitive) masks from the oracle alone."""
    amb = orc["margin"] < MARGIN
    sens = (orc["q"] >= 0) & ~(COND * conditioning(orc) <= TOL_T * window)
    return amb, sens & ~amb


def check_forward(gpu, orc, n_in, window, label="", max_ambiguous=MAX_AMBIGUOUS):
    """gpu: dict of numpy arrays t_out, slope, q (fp32 path); orc: oracle dict.
    Returns the mask of neurons whose upstream gradient is zeroed."""
    amb, sens = excluded(orc, n_in, window)
    ok = ~amb
    qg, qo = gpu["q"].astype(np.int64), orc["q"].astype(np.int64)
    bad_q = ok & (qg != qo)
    both = ok & (qo >= 0) & (qg >= 0)
    with np.errstate(invalid="ignore"):
        dt = np.abs(gpu["t_out"].astype(np.float64) - orc["t_out"])
    est = conditioning(orc)
    lim = np.maximum(TOL_T * window, COND * est)
    bad_t = both & ~(dt <= lim)
    beyond = both & ~(dt <= TOL_T * window)
    silent_ok = np.all(np.isinf(gpu["t_out"][ok & (qo < 0)]))
    n = qo.size
    nf = max(int((qo >= 0).sum()), 1)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(both, dt / est, 0.0)
    stats = dict(label=label, n=n, fired=int((qo >= 0).sum()), ambiguous=int(amb.sum()),
                 q_mismatch=int(bad_q.sum()), t_bad=int(bad_t.sum()),
                 beyond_tol=int(beyond.sum()), grad_masked=int((amb | sens | beyond).sum()),
                 max_dt=float(dt[both].max()) if both.any() else 0.0,
                 max_dt_well_conditioned=float(dt[both & ~sens].max()) if (both & ~sens).any() else 0.0,
                 max_err_over_est=float(np.nanmax(ratio)) if both.any() else 0.0)
    print("forward parity", stats, flush=True)
    assert bad_q.sum() == 0, f"{label}: interval index mismatch outside ambiguity set: {stats}"
    assert bad_t.sum() == 0, f"{label}: spike time beyond tolerance: {stats}"
    assert silent_ok, f"{label}: GPU fired where the oracle is silent"
    assert beyond.sum() <= MAX_BEYOND * nf + 1, f"{label}: ill-conditioned bucket too large: {stats}"
    assert amb.sum() <= max_ambiguous * n + 1, f"{label}: ambiguity set too large: {stats}"
    return amb | sens | beyond, stats


def near_grid(t_in, p, rel=1e-5):
    """Inputs within rel*dt of a grid point: the event derivatives jump there
    (one-sided), so fp32 and fp64 binning may legitimately take different sides."""
    x = (np.asarray(t_in, dtype=np.float64) - p["t0"]) / p["dt"]
    with np.errstate(invalid="ignore"):
        return np.isfinite(x) & (np.abs(x - np.round(x)) < rel)


def check_grad(g_gpu, g_orc, label, g_abs=None, rtol=GRAD_RTOL, atol=GRAD_ATOL, kappa=KAPPA):
    g_gpu = np.asarray(g_gpu, dtype=np.float64)
    err = np.abs(g_gpu - g_orc)
    floor = atol if g_abs is None else np.maximum(atol, kappa * g_abs)
    lim = rtol * np.abs(g_orc) + floor
    bad = ~(err <= lim)
    scale = float(np.abs(g_orc).max()) if g_orc.size else 0.0
    cond = float((err / np.maximum(g_abs, 1e-30)).max()) if (g_abs is not None and err.size) else None
    stats = dict(label=label, n=int(g_orc.size), bad=int(bad.sum()), scale=scale,
                 max_abs_err=float(err.max()) if err.size else 0.0,
                 max_rel=float((err / (np.abs(g_orc) + 1e-30)).max()) if err.size else 0.0,
                 max_err_over_abs=cond)
    print("grad parity", stats, flush=True)
    assert bad.sum() == 0, f"{label}: gradient mismatch: {stats}"
    return stats
