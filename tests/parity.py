"""Comparison rules between the HIP path (fp32, fp64 scan state) and the fp64
oracle.

Forward:
- Fire / no-fire and the interval index q must agree exactly outside the
  ambiguity set: neurons whose decision-relevant potentials lie within 1e-5
  of the threshold (the oracle's `margin`).
- Spike times must agree within 1e-5 of the time window outside the
  ambiguity set. The fp32 path cannot reach that where the crossing is flat:
  the potential at the spike is a sum of terms of total magnitude `vabs`, so
  its fp32 rounding (unit u = 2^-24) moves the time by about
  u * vabs / |slope|, and the fp32 time itself carries u * |t|. The time
  error model is delta = C_T * u * (vabs / |slope| + |t|). Spikes beyond
  1e-5 of the window form the ill-conditioned bucket: they must still lie
  within delta, are reported separately as outside the 1e-5 tolerance, and
  must stay below 0.5 % of the fired neurons.

Gradients (1e-3 relative, per element):
- The slope carries a relative error rho = (C_T u E + k2 E delta) / |slope|,
  with E the event mass of the spike (the oracle's `emass`, which bounds the
  terms of v' since |K'| <= 1) and k2 = 1/tau_v + 1/tau_I (which bounds |K''|,
  so k2 E bounds |v''| and k2 E delta the slope moved by the time error).
- Each term's factor G = gamma K(t - T_m) then moves by at most
  |gamma| (rho K + delta |K'|) to first order; the oracle sums that bound over
  each element's terms (its error-weighted sum `err`, pinned in
  test_oracle_conditioning). The fp32 products and sums add
  u (C0 + sqrt(n)) times the element's sum of |terms| (`abs`), n its number
  of terms, C0 a few ulps for each term's own factors.
- An element passes when |gpu - oracle| <= 1e-3 |oracle| +
  max(1e-6, C_G (err + u (C0 + sqrt(n)) abs)).
- The upstream gradient is zeroed on both sides only for ambiguous neurons,
  for the ill-conditioned bucket, and where the first-order model breaks
  down (rho > RHO_MAX). The masked share is reported; outside the ambiguity
  set (capped on its own) it may not exceed 5 % of the fired neurons.
"""
import math

import numpy as np

U = 2.0 ** -24
TOL_T = 1e-5         # of the window
MARGIN = 1e-5        # |v - theta| ambiguity
C_T = 4.0            # time / slope error model constant (measured ratios stay below ~3)
C_G = 2.0            # safety factor on the first-order gradient error bound
C0 = 8.0             # ulps of each term's own factors (event weight, G, weight)
RHO_MAX = 5e-2       # relative slope error beyond which the first-order model is not used
MAX_BEYOND = 0.005
MAX_AMBIGUOUS = 0.01
MAX_MASKED = 0.05
GRAD_RTOL = 1e-3
GRAD_ATOL = 1e-6


def k2_of(taus):
    """1/tau_v + 1/tau_I (bound of |K''| on every kernel row; 1/inf = 0)."""
    return sum(0.0 if math.isinf(t) else 1.0 / t for t in taus)


def error_model(orc, taus=None):
    """Per-neuron (delta, rho): time error and relative slope error bounds.
    Silent neurons get 0. Without time constants (or without `emass`) rho
    is 0."""
    fired = orc["q"] >= 0
    with np.errstate(divide="ignore", invalid="ignore"):
        aslope = np.abs(orc["slope"])
        delta = C_T * U * (orc["vabs"] / aslope + np.abs(orc["t_out"]))
        delta = np.where(fired, delta, 0.0)
        if taus is not None and "emass" in orc:
            E = orc["emass"]
            rho = (C_T * U * E + k2_of(taus) * E * delta) / aslope + U
            rho = np.where(fired, rho, 0.0)
        else:
            rho = np.zeros_like(delta)
    return delta, rho


def check_forward(gpu, orc, n_in, window, label="", max_ambiguous=MAX_AMBIGUOUS, taus=None,
                  max_masked=MAX_MASKED):
    """gpu: dict of numpy arrays t_out, slope, q (fp32 path); orc: oracle dict.
    Returns (mask of neurons whose upstream gradient is zeroed, stats); the
    stats carry the per-neuron error model (delta, rho) for the gradient
    check."""
    del n_in
    amb = orc["margin"] < MARGIN
    ok = ~amb
    qg, qo = gpu["q"].astype(np.int64), orc["q"].astype(np.int64)
    bad_q = ok & (qg != qo)
    both = ok & (qo >= 0) & (qg >= 0)
    with np.errstate(invalid="ignore"):
        dt = np.abs(gpu["t_out"].astype(np.float64) - orc["t_out"])
    delta, rho = error_model(orc, taus)
    lim = np.maximum(TOL_T * window, delta)
    bad_t = both & ~(dt <= lim)
    beyond = both & ~(dt <= TOL_T * window)
    breakdown = both & ~(rho <= RHO_MAX)
    silent_ok = np.all(np.isinf(gpu["t_out"][ok & (qo < 0)]))
    mask = amb | beyond | breakdown
    n = qo.size
    nf = int((qo >= 0).sum())
    nfe = max(nf, 1)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(both, dt / delta, 0.0)
    masked_fired = int((mask & (qo >= 0)).sum())
    masked_unamb = int((mask & (qo >= 0) & ~amb).sum())
    stats = dict(label=label, n=n, fired=nf, ambiguous=int(amb.sum()),
                 q_mismatch=int(bad_q.sum()), t_bad=int(bad_t.sum()),
                 beyond_tol=int(beyond.sum()),
                 max_dt_beyond=float(dt[beyond].max()) if beyond.any() else 0.0,
                 rho_breakdown=int(breakdown.sum()),
                 grad_masked=masked_fired, grad_masked_frac=masked_fired / nfe,
                 grad_masked_unambiguous=masked_unamb,
                 max_dt=float(dt[both].max()) if both.any() else 0.0,
                 max_dt_within_tol=float(dt[both & ~beyond].max()) if (both & ~beyond).any() else 0.0,
                 max_err_over_delta=float(np.nanmax(ratio)) if both.any() else 0.0,
                 max_rho=float(rho[both].max()) if both.any() else 0.0)
    print("forward parity", stats, flush=True)
    stats["delta"], stats["rho"] = delta, rho
    assert bad_q.sum() == 0, f"{label}: interval index mismatch outside ambiguity set: {stats}"
    assert bad_t.sum() == 0, f"{label}: spike time beyond tolerance and error model: {stats}"
    assert silent_ok, f"{label}: GPU fired where the oracle is silent"
    assert beyond.sum() <= MAX_BEYOND * nfe + 1, f"{label}: ill-conditioned bucket too large: {stats}"
    assert amb.sum() <= max_ambiguous * n + 1, f"{label}: ambiguity set too large: {stats}"
    assert masked_unamb <= max_masked * nf + 2, f"{label}: too many neurons masked from the gradient check: {stats}"
    return mask, stats


def grad_err_inputs(stats, mask):
    """(rho, delta) for the oracle's error-weighted sums (masked neurons carry
    no gradient, their entries do not matter)."""
    return np.where(mask, 0.0, stats["rho"]), np.where(mask, 0.0, stats["delta"])


def near_grid(t_in, p, rel=1e-5):
    """Inputs within rel*dt of a grid point: the event derivatives jump there
    (one-sided), so fp32 and fp64 binning may legitimately take different sides."""
    x = (np.asarray(t_in, dtype=np.float64) - p["t0"]) / p["dt"]
    with np.errstate(invalid="ignore"):
        return np.isfinite(x) & (np.abs(x - np.round(x)) < rel)


def check_grad(g_gpu, g_orc, label, g_abs, g_err=None, n_terms=1, rtol=GRAD_RTOL, atol=GRAD_ATOL,
               kappa=None):
    """Per-element gradient check. g_abs: the oracle's sum of |terms|; g_err:
    its error-weighted sum (None: no spike-time / slope contribution);
    n_terms: the number of terms an element sums (upper bound). `kappa`, when
    given, replaces the derived floor by kappa * g_abs (the multi-spike path,
    whose error model through the reset chain is not derived)."""
    g_gpu = np.asarray(g_gpu, dtype=np.float64)
    err = np.abs(g_gpu - g_orc)
    if kappa is not None:
        model = kappa * g_abs
    else:
        model = C_G * ((0.0 if g_err is None else g_err) + U * (C0 + math.sqrt(n_terms)) * g_abs)
    lim = rtol * np.abs(g_orc) + np.maximum(atol, model)
    bad = ~(err <= lim)
    scale = float(np.abs(g_orc).max()) if g_orc.size else 0.0
    with np.errstate(divide="ignore", invalid="ignore"):
        over_model = float(np.nanmax(np.where(model > 0, err / model, 0.0))) if err.size else 0.0
        over_abs = float((err / np.maximum(g_abs, 1e-30)).max()) if err.size else 0.0
    stats = dict(label=label, n=int(g_orc.size), bad=int(bad.sum()), scale=scale,
                 max_abs_err=float(err.max()) if err.size else 0.0,
                 max_rel=float((err / (np.abs(g_orc) + 1e-30)).max()) if err.size else 0.0,
                 max_err_over_abs=over_abs, max_err_over_model=over_model,
                 kappa=kappa)
    print("grad parity", stats, flush=True)
    assert bad.sum() == 0, f"{label}: gradient mismatch: {stats}"
    return stats
