/*
 * dstd_oracle.c -- plain, slow, fp64 CPU oracle for the DSTD-LIF layer.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call
 * this file: only the test suite, the smoke check and the benchmark's CPU
 * baseline leg use it. It shares no code, header, table or constant with the
 * HIP library; it is written from the paper (Sakemi et al., "Scalable Training
 * of Continuous-Time Spiking Neural Networks with Differentiable Spike-Time
 * Discretization"):
 *
 *   LIF model and spike kernel K(t) ............ App. A, Eq. (LIF_model_TTFS),
 *                                                  Table "tab:kernel" (rows tau_v != tau_I,
 *                                                  (tau, tau), (inf, tau), (inf, inf))
 *   exact spike time (sort + interval candidates) App. A, Eq. (timing_exact), Alg. 1
 *   exact spike-time gradients .................. implicit function theorem on
 *                                                  v(t) = V_th over the causal set (App. A)
 *   multi-spike DSTD (reset of v, current kept) . App. "multi-spikes", Eq. (Vmem_multiSpikes)
 *   DSTD grid T_m = T_first + m*dt - t_offset .. App. B.1
 *   DSTD event weights s_jm ..................... Eq. (DSTD_kernel), Table "tab:DSTD_kernels"
 *   weighted events w^_im = sum_j w_ij s_jm ..... App. B.1 (definition of w^)
 *   DSTD candidate times and min selection ...... Table "tab:timing_DSTD", Eq. (timing_DSTD);
 *                                                  the closed-form rows as printed, with the
 *                                                  principal branch W_0 for (tau, tau)
 *
 * Every quantity is computed in double precision from its plain definition.
 * Inputs are double; callers pass the float32 values the GPU sees, widened
 * exactly, or fp64 values for finite-difference pins.
 *
 * Readings where the paper is silent (listed in the design notes):
 *  - M intervals, M+1 grid points T_0..T_M; the grid is passed as (t0, dt, M),
 *    the random t_offset of Alg. 2 is folded into t0 by the caller.
 *  - Eq. (DSTD_kernel) is applied literally at the grid ends: an input in
 *    [T_{-1}, T_0) keeps only its weight at T_0, an input in [T_M, T_{M+1})
 *    keeps only its weight at T_M; everything else (including +inf = silent)
 *    contributes nothing.
 *  - The last candidate interval is [T_M, t_max) (t_max = +inf by default):
 *    Eq. (timing_DSTD) leaves T_{M+1} undefined; the exact method's analogue
 *    uses +inf for the interval after the last input.
 *  - "Reaches the threshold" means v >= V_th; the interval is half-open.
 *  - The kernel is symmetric in (tau_v, tau_I); the canonical order puts the
 *    larger (possibly infinite) constant first. A time constant of +inf
 *    selects the (inf, tau) / (inf, inf) rows, equal finite constants the
 *    (tau, tau) row.
 *
 * The only non-closed-form step is the root of v^(t) = V_th inside an
 * interval for general (tau_v, tau_I) (Table "tab:timing_DSTD" gives closed
 * forms only for special ratios). Inside one interval v^ is a combination of
 * two exponentials, so its derivative has at most one zero; the interval is
 * split there into monotone pieces and the first rising piece that reaches
 * V_th is bisected to full double precision.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Rows of the tables, by the pair of time constants.                        */
/* ------------------------------------------------------------------------ */
enum { ROW_GENERAL = 0, ROW_EQUAL = 1, ROW_INF_TAU = 2, ROW_INF_INF = 3 };

static int row_of(double tv, double ti) {
    if (isinf(tv) && isinf(ti)) return ROW_INF_INF;
    if (isinf(tv) || isinf(ti)) return ROW_INF_TAU;
    if (tv == ti) return ROW_EQUAL;
    return ROW_GENERAL;
}

/* the finite constant of an (inf, tau) pair */
static double finite_of(double tv, double ti) { return isinf(tv) ? ti : tv; }

/* ------------------------------------------------------------------------ */
/* Spike kernel K(t), Table "tab:kernel".                                    */
/* ------------------------------------------------------------------------ */
static double kern(double tv, double ti, double t) {
    if (t < 0.0) return 0.0; /* Heaviside factor */
    switch (row_of(tv, ti)) {
        case ROW_INF_INF: return t;
        case ROW_INF_TAU: { double tau = finite_of(tv, ti); return tau * (1.0 - exp(-t / tau)); }
        case ROW_EQUAL: return t * exp(-t / tv);
        default: {
            double c = tv * ti / (tv - ti);
            return c * (exp(-t / tv) - exp(-t / ti));
        }
    }
}

double oracle_kernel(double tau_v, double tau_i, double t) { return kern(tau_v, tau_i, t); }

/* ------------------------------------------------------------------------ */
/* DSTD kernel K_DSTD, Table "tab:DSTD_kernels", and its derivative with      */
/* respect to its argument (D = dt).                                         */
/* ------------------------------------------------------------------------ */
static double kdstd(double tv, double ti, double D, double t) {
    int row = row_of(tv, ti);
    if (row == ROW_INF_INF) return (t < 0.0) ? (t + D) / D : (D - t) / D;
    if (row == ROW_INF_TAU) {
        double tau = finite_of(tv, ti), den = 1.0 - exp(-D / tau);
        if (t < 0.0) return (-exp(-D / tau) + exp(t / tau)) / den;
        return (1.0 - exp((t - D) / tau)) / den;
    }
    if (row == ROW_EQUAL) {
        if (t < 0.0) return (t + D) / D * exp(t / tv);
        return (D - t) / D * exp(t / tv);
    }
    double den = exp(-D / tv) - exp(-D / ti);
    if (t >= 0.0)
        return (exp((t - D) / tv) - exp((t - D) / ti)) / den;
    return (-exp(-D / ti) * exp(t / tv) + exp(-D / tv) * exp(t / ti)) / den;
}

static double kdstd_dt(double tv, double ti, double D, double t) {
    int row = row_of(tv, ti);
    if (row == ROW_INF_INF) return (t < 0.0) ? 1.0 / D : -1.0 / D;
    if (row == ROW_INF_TAU) {
        double tau = finite_of(tv, ti), den = 1.0 - exp(-D / tau);
        if (t < 0.0) return exp(t / tau) / tau / den;
        return -exp((t - D) / tau) / tau / den;
    }
    if (row == ROW_EQUAL) {
        if (t < 0.0) return exp(t / tv) * (1.0 / D + (t + D) / (D * tv));
        return exp(t / tv) * (-1.0 / D + (D - t) / (D * tv));
    }
    double den = exp(-D / tv) - exp(-D / ti);
    if (t >= 0.0)
        return (exp((t - D) / tv) / tv - exp((t - D) / ti) / ti) / den;
    return (-exp(-D / ti) * exp(t / tv) / tv + exp(-D / tv) * exp(t / ti) / ti) / den;
}

double oracle_kdstd(double tau_v, double tau_i, double dt, double t) { return kdstd(tau_v, tau_i, dt, t); }

static double kern_dt(double tv, double ti, double t);

/* Grid point T_m (App. B.1 with t_offset folded into t0). */
static double grid(double t0, double dt, int m) { return t0 + (double)m * dt; }

/*
 * Eq. (DSTD_kernel) taken literally: s_jm = K_DSTD(t_j - T_m) when
 * T_{m-1} <= t_j < T_{m+1}, else 0, for m = 0..M. Every m is tested; the
 * nonzero ones (at most two, the compact support of App. B.3) are returned.
 */
static int events_literal(double t, double t0, double dt, int M, double tv, double ti,
                          int *m_out, double *s_out, double *ds_out) {
    int n = 0;
    for (int m = 0; m <= M; ++m) {
        double lo = grid(t0, dt, m - 1), hi = grid(t0, dt, m + 1);
        if (lo <= t && t < hi) {
            double arg = t - grid(t0, dt, m);
            if (n < 2) {
                m_out[n] = m;
                s_out[n] = kdstd(tv, ti, dt, arg);
                ds_out[n] = kdstd_dt(tv, ti, dt, arg);
            }
            ++n;
        }
    }
    return n;
}

/* Dense event tensor s[b][m][j] for small cases (pins). */
void oracle_dstd_events(double tau_v, double tau_i, int M, double t0, double dt,
                        int64_t B, int64_t N_in, const double *t_in, double *s, double *ds) {
    memset(s, 0, sizeof(double) * (size_t)(B * (M + 1) * N_in));
    if (ds) memset(ds, 0, sizeof(double) * (size_t)(B * (M + 1) * N_in));
    for (int64_t b = 0; b < B; ++b)
        for (int64_t j = 0; j < N_in; ++j) {
            int mm[2]; double sv[2], dv[2];
            int n = events_literal(t_in[b * N_in + j], t0, dt, M, tau_v, tau_i, mm, sv, dv);
            for (int k = 0; k < n && k < 2; ++k) {
                s[(b * (M + 1) + mm[k]) * N_in + j] = sv[k];
                if (ds) ds[(b * (M + 1) + mm[k]) * N_in + j] = dv[k];
            }
        }
}

/* ------------------------------------------------------------------------ */
/* Candidate solve inside one interval.                                      */
/*                                                                           */
/* On an interval the potential is v(t) = c*(a*exp(-(t-tr)/tv)               */
/*  - b*exp(-(t-tr)/ti)), the general-tau analogue of the a_iq, b_iq prefix   */
/* sums of Tables "tab:spike_timing" / "tab:timing_DSTD" (weights times       */
/* exp(T/tau)), written relative to a reference time tr so the exponentials  */
/* stay in range.                                                            */
/* ------------------------------------------------------------------------ */
typedef struct { double tv, ti, c, theta, tr, a, b; int row; } piece_t;

static void piece_init(piece_t *p, double tv, double ti, double theta, double tr) {
    p->tv = tv; p->ti = ti; p->theta = theta; p->tr = tr; p->a = 0.0; p->b = 0.0;
    p->row = row_of(tv, ti);
    p->c = (p->row == ROW_GENERAL) ? tv * ti / (tv - ti) : 0.0;
}

/*
 * Add a weight w arriving at time T to the prefix sums a, b of Tables
 * "tab:spike_timing" / "tab:timing_DSTD" (shifted frame s = T - tr):
 *   general  : a += w e^{s/tv},            b += w e^{s/ti}
 *   (tau,tau): a += w e^{s/tau},           b += w (s/tau) e^{s/tau}
 *   (inf,tau): a += w e^{s/tau},           b += w
 *   (inf,inf): a += w s,                   b += w
 */
static void piece_add(piece_t *p, double w, double T) {
    double s = T - p->tr;
    switch (p->row) {
        case ROW_INF_INF: p->a += w * s; p->b += w; break;
        case ROW_INF_TAU: { double tau = finite_of(p->tv, p->ti);
                            p->a += w * exp(s / tau); p->b += w; break; }
        case ROW_EQUAL: p->a += w * exp(s / p->tv); p->b += w * (s / p->tv) * exp(s / p->tv); break;
        default: p->a += w * exp(s / p->tv); p->b += w * exp(s / p->ti); break;
    }
}

/* the potential on the current piece, from the prefix sums:
 *   general  : c (a e^{-s/tv} - b e^{-s/ti})
 *   (tau,tau): e^{-s/tau} (s a - tau b)
 *   (inf,tau): tau (b - a e^{-s/tau})
 *   (inf,inf): b s - a                                                    */
static double pv(const piece_t *p, double t) {
    double s = t - p->tr;
    switch (p->row) {
        case ROW_INF_INF: return p->b * s - p->a;
        case ROW_INF_TAU: { double tau = finite_of(p->tv, p->ti);
                            return tau * (p->b - p->a * exp(-s / tau)); }
        case ROW_EQUAL: return exp(-s / p->tv) * (s * p->a - p->tv * p->b);
        default: return p->c * (p->a * exp(-s / p->tv) - p->b * exp(-s / p->ti));
    }
}

static double pdv(const piece_t *p, double t) {
    double s = t - p->tr;
    switch (p->row) {
        case ROW_INF_INF: return p->b;
        case ROW_INF_TAU: { double tau = finite_of(p->tv, p->ti); return p->a * exp(-s / tau); }
        case ROW_EQUAL: return exp(-s / p->tv) * (p->a * (1.0 - s / p->tv) + p->b);
        default: return p->c * (-p->a / p->tv * exp(-s / p->tv) + p->b / p->ti * exp(-s / p->ti));
    }
}

/* value at hi; at hi = +inf the decaying rows vanish, (inf, tau) tends to
   tau b and (inf, inf) to +-inf with the sign of b (-a when b = 0) */
static double pv_end(const piece_t *p, double hi) {
    if (!isinf(hi)) return pv(p, hi);
    switch (p->row) {
        case ROW_INF_INF: return (p->b > 0.0) ? INFINITY : (p->b < 0.0) ? -INFINITY : -p->a;
        case ROW_INF_TAU: return finite_of(p->tv, p->ti) * p->b;
        default: return 0.0;
    }
}

/*
 * Principal branch W_0 of the Lambert W function (w e^w = x, w >= -1) for
 * x >= -1/e: the series in p = sqrt(2 (e x + 1)) about the branch point (or
 * log-based guesses) refined by Halley's iteration.
 */
double oracle_lambert_w0(double x) {
    const double E = 2.718281828459045235360287;
    if (!(x >= -1.0 / E)) return NAN;
    if (x == 0.0) return 0.0;
    double w;
    if (x < -0.3) {
        double p = sqrt(fmax(0.0, 2.0 * (E * x + 1.0)));
        w = -1.0 + p - p * p / 3.0 + 11.0 / 72.0 * p * p * p - 43.0 / 540.0 * p * p * p * p;
        if (p < 1e-5) return w; /* the series is exact to rounding there */
    } else if (x < 3.0) {
        w = log1p(x) * (1.0 - 0.5 * log1p(log1p(x)) / (1.0 + log1p(x)));
    } else {
        double l = log(x);
        w = l - log(l);
    }
    for (int it = 0; it < 100; ++it) {
        double e = exp(w), f = w * e - x;
        double wn = w - f / (e * (w + 1.0) - (w + 2.0) * f / (2.0 * w + 2.0));
        if (!isfinite(wn)) break;
        if (fabs(wn - w) <= 4e-16 * (1.0 + fabs(wn))) { w = wn; break; }
        w = wn;
    }
    return w;
}

/*
 * Candidate of one interval from Table "tab:timing_DSTD" (shifted frame), for
 * the closed-form rows; NAN where the formula has no real value:
 *   (tau,tau): tau [b/a - W_0(-(V_th/tau)/a e^{b/a})]   (a > 0)
 *   (inf,tau): tau ln[a / (b - V_th/tau)]
 *   (inf,inf): (V_th + a) / b
 */
static double candidate(const piece_t *p) {
    double th = p->theta;
    switch (p->row) {
        case ROW_INF_INF: return (p->b > 0.0) ? (th + p->a) / p->b : NAN;
        case ROW_INF_TAU: {
            double tau = finite_of(p->tv, p->ti), den = p->b - th / tau;
            return (p->a > 0.0 && den > 0.0) ? tau * log(p->a / den) : NAN;
        }
        case ROW_EQUAL: {
            if (!(p->a > 0.0)) return NAN;
            double r = p->b / p->a;
            double z = -(th / p->tv) / p->a * exp(r);
            double w = oracle_lambert_w0(z);
            return isnan(w) ? NAN : p->tv * (r - w);
        }
        default: return NAN;
    }
}

/*
 * First t in [lo, hi) with v(t) >= theta. Returns 1 and sets *root when it
 * exists. *peak receives sup v over [lo, hi] (for the ambiguity margin).
 */
static int first_crossing_closed(const piece_t *p, double lo, double hi, double *root,
                                 double *peak);

static int first_crossing(const piece_t *p, double lo, double hi, double *root, double *peak) {
    if (p->row != ROW_GENERAL) return first_crossing_closed(p, lo, hi, root, peak);
    double th = p->theta;
    /* critical point of v: exp(-kappa*s) = a*ti/(b*tv), kappa = 1/ti - 1/tv */
    double kappa = 1.0 / p->ti - 1.0 / p->tv;
    double tc = NAN;
    double ratio = (p->b != 0.0) ? (p->a * p->ti) / (p->b * p->tv) : -1.0;
    if (ratio > 0.0) {
        tc = p->tr - log(ratio) / kappa;
        if (!(tc > lo && tc < hi)) tc = NAN;
    }
    double v_lo = pv(p, lo), v_hi = pv_end(p, hi);
    double pk = fmax(v_lo, v_hi);
    if (!isnan(tc)) pk = fmax(pk, pv(p, tc));
    *peak = pk;

    if (v_lo >= th) { *root = lo; return 1; }
    double e0[2], e1[2];
    int np = 0;
    if (!isnan(tc)) { e0[0] = lo; e1[0] = tc; e0[1] = tc; e1[1] = hi; np = 2; }
    else { e0[0] = lo; e1[0] = hi; np = 1; }
    for (int k = 0; k < np; ++k) {
        double a = e0[k], b = e1[k];
        double fa = pv(p, a) - th;
        double fb = pv_end(p, b) - th;
        if (fa >= 0.0) { *root = a; return 1; }
        if (fb < 0.0) continue; /* piece stays below threshold */
        if (isinf(b)) continue; /* v -> 0 < theta at +inf: unreachable */
        /* f(a) < 0 <= f(b) on a monotone piece: bisect */
        for (int it = 0; it < 400; ++it) {
            double mid = 0.5 * (a + b);
            if (!(mid > a && mid < b)) break;
            if (pv(p, mid) - th >= 0.0) b = mid; else a = mid;
        }
        if (b >= hi) return 0; /* the crossing is exactly at hi: next interval */
        *root = b;
        return 1;
    }
    return 0;
}

/*
 * Closed-form rows: the potential's only critical point is the maximum of
 * (tau, tau) at s = tau (1 + b/a) (a > 0); the (inf, .) rows are monotone.
 * The first time in [lo, hi) with v >= V_th is lo itself when v(lo) >= V_th,
 * else the table's candidate when it lies in [lo, hi) (for (tau, tau) the
 * W_0 branch is the crossing on the rising side, i.e. the first one).
 */
static int first_crossing_closed(const piece_t *p, double lo, double hi, double *root,
                                 double *peak) {
    double th = p->theta;
    double v_lo = pv(p, lo), v_hi = pv_end(p, hi);
    double pk = fmax(v_lo, v_hi);
    if (p->row == ROW_EQUAL && p->a > 0.0) {
        double sc = p->tr + p->tv * (1.0 + p->b / p->a);
        if (sc > lo && sc < hi) pk = fmax(pk, pv(p, sc));
    }
    *peak = pk;
    if (v_lo >= th) { *root = lo; return 1; }
    double c = candidate(p);
    if (isnan(c)) return 0;
    double t = p->tr + c;
    if (t >= lo && t < hi) { *root = t; return 1; }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* DSTD forward for one sample: Eq. (DSTD), App. B.1, Table "tab:timing_DSTD" */
/* and Eq. (timing_DSTD).                                                    */
/* ------------------------------------------------------------------------ */
typedef struct {
    double tv, ti, theta, t0, dt, t_max;
    int M;
} prm_t;

static void canon(prm_t *p, double tau_m, double tau_s) {
    /* K is symmetric in (tau_v, tau_I); keep tau_v > tau_I */
    p->tv = fmax(tau_m, tau_s);
    p->ti = fmin(tau_m, tau_s);
}

/* per-neuron scan over the M+1 DSTD intervals given w^[0..M] */
static void dstd_scan(const prm_t *p, const double *wh, double *t_out, double *slope,
                      int *q_out, double *margin, double *v_at_T) {
    piece_t pc;
    piece_init(&pc, p->tv, p->ti, p->theta, p->t0);
    double pre = INFINITY; /* min over earlier intervals of theta - peak */
    for (int q = 0; q <= p->M; ++q) {
        double Tq = grid(p->t0, p->dt, q);
        /* prefix sums a_iq, b_iq of Table "tab:timing_DSTD", shifted frame */
        piece_add(&pc, wh[q], Tq);
        double hi = (q < p->M) ? grid(p->t0, p->dt, q + 1) : p->t_max;
        if (v_at_T) v_at_T[q] = pv(&pc, Tq);
        double root, peak;
        int hit = first_crossing(&pc, Tq, hi, &root, &peak);
        if (hit) {
            *t_out = root;
            *slope = pdv(&pc, root);
            *q_out = q;
            double m = pre;
            m = fmin(m, fabs(peak - p->theta));
            m = fmin(m, fabs(pv(&pc, Tq) - p->theta));
            if (q < p->M) m = fmin(m, fabs(pv(&pc, hi) - p->theta));
            if (margin) *margin = m;
            return;
        }
        pre = fmin(pre, p->theta - peak);
    }
    *t_out = INFINITY;
    *slope = 0.0;
    *q_out = -1;
    if (margin) *margin = pre;
}

typedef struct { int n; int m[2]; double s[2]; double ds[2]; } ev_t;

static void sample_events(const prm_t *p, const double *t_row, int64_t N_in, ev_t *ev) {
    for (int64_t j = 0; j < N_in; ++j) {
        ev_t e;
        int n = events_literal(t_row[j], p->t0, p->dt, p->M, p->tv, p->ti, e.m, e.s, e.ds);
        e.n = n > 2 ? 2 : n;
        ev[j] = e;
    }
}

/*
 * Forward of one dense layer.
 *   t_in [B][N_in] (+inf = silent), W [N_out][N_in] (w_ij: j -> i)
 * Outputs (double): t_out [B][N_out] (+inf = no spike), slope = dv^/dt at
 * t_out, q_idx = interval index (-1 = none), margin (distance of the
 * decision-relevant potentials from V_th), vabs = sum over m <= q* of
 * |K(t_out - T_m)| * sum_j |w_ij s_jm| (scale of the terms forming v^(t_out)),
 * emass = sum over m <= q* (all m for a silent neuron) of sum_j |w_ij s_jm|
 * (the event mass that v^ and its derivatives are formed from; with
 * |K'| <= 1 it bounds the scale of the terms of the slope),
 * what (optional) [B][M+1][N_out] = weighted events.
 * vabs, emass and what are conditioning / inspection outputs for the tests.
 */
void oracle_dstd_forward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                         double t_max, int64_t B, int64_t N_in, int64_t N_out,
                         const double *t_in, const double *W,
                         double *t_out, double *slope, int32_t *q_idx, double *margin,
                         double *vabs, double *emass, double *what) {
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)(N_in > 0 ? N_in : 1));
        double *wh = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        double *wabs = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        sample_events(&p, t_in + b * N_in, N_in, ev);
        for (int64_t i = 0; i < N_out; ++i) {
            for (int m = 0; m <= M; ++m) { wh[m] = 0.0; wabs[m] = 0.0; }
            const double *wr = W + i * N_in;
            /* w^_im = sum_j w_ij s_jm over the nonzero s_jm */
            for (int64_t j = 0; j < N_in; ++j)
                for (int k = 0; k < ev[j].n; ++k) {
                    wh[ev[j].m[k]] += wr[j] * ev[j].s[k];
                    wabs[ev[j].m[k]] += fabs(wr[j] * ev[j].s[k]);
                }
            if (what)
                for (int m = 0; m <= M; ++m) what[(b * (M + 1) + m) * N_out + i] = wh[m];
            double to, sl, mg; int q;
            dstd_scan(&p, wh, &to, &sl, &q, &mg, NULL);
            int64_t o = b * N_out + i;
            t_out[o] = to; slope[o] = sl; q_idx[o] = q;
            if (margin) margin[o] = mg;
            if (vabs) {
                double va = 0.0;
                for (int m = 0; m <= (q < 0 ? -1 : q); ++m)
                    va += fabs(kern(p.tv, p.ti, to - grid(t0, dt, m))) * wabs[m];
                vabs[o] = va;
            }
            if (emass) {
                double em = 0.0;
                for (int m = 0; m <= (q < 0 ? M : q); ++m) em += wabs[m];
                emass[o] = em;
            }
        }
        free(ev); free(wh); free(wabs);
    }
}

/* Scan only, from given weighted events w^ [B][M+1][N_out] (pins the solver). */
void oracle_dstd_scan(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                      double t_max, int64_t B, int64_t N_out, const double *what,
                      double *t_out, double *slope, int32_t *q_idx, double *margin,
                      double *v_at_T /* [B][M+1][N_out] or NULL */) {
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        double *wh = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        double *vt = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        for (int64_t i = 0; i < N_out; ++i) {
            for (int m = 0; m <= M; ++m) { wh[m] = what[(b * (M + 1) + m) * N_out + i]; vt[m] = NAN; }
            double to, sl, mg; int q;
            dstd_scan(&p, wh, &to, &sl, &q, &mg, vt);
            int64_t o = b * N_out + i;
            t_out[o] = to; slope[o] = sl; q_idx[o] = q;
            if (margin) margin[o] = mg;
            if (v_at_T) for (int m = 0; m <= M; ++m) v_at_T[(b * (M + 1) + m) * N_out + i] = vt[m];
        }
        free(wh); free(vt);
    }
}

/*
 * Backward of one dense layer. The DSTD spike time solves v^(t) = V_th with
 * v^(t) = sum_{m<=q*} w^_m K(t - T_m) (App. B.1); the interval index q* is
 * piecewise constant, so by the implicit-function theorem
 *   d t / d w^_m = -K(t - T_m) / v^'(t)   for m <= q*,  0 otherwise,
 * which is what reverse-mode differentiation of the closed-form candidates of
 * Table "tab:timing_DSTD" yields as well (each candidate is that root).
 * Chain rule through w^_im = sum_j w_ij s_jm and s_jm = K_DSTD(t_j - T_m):
 *   dL/dw_ij = sum_b sum_m G[b,m,i] s_jm,   dL/dt_j = sum_m sum_i G[b,m,i] w_ij ds_jm/dt_j
 * with G[b,m,i] = -g_bi K(t_bi - T_m) / slope_bi. Non-fired neurons (q < 0)
 * contribute nothing. grad_W is [N_out][N_in], grad_t_in is [B][N_in].
 */
void oracle_dstd_backward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                          double t_max, int64_t B, int64_t N_in, int64_t N_out,
                          const double *t_in, const double *W,
                          const double *t_out, const double *slope, const int32_t *q_idx,
                          const double *grad_t_out,
                          int64_t n_isel, const int64_t *isel, double *grad_W,
                          int64_t n_bsel, const int64_t *bsel, double *grad_t_in,
                          double *grad_W_abs, double *grad_t_in_abs,
                          const double *rho, const double *delta,
                          double *grad_W_err, double *grad_t_in_err) {
    /* grad_W rows are computed for the n_isel neurons listed in isel (all when
       n_isel < 0) and stored as [n_isel][N_in]; grad_t_in rows likewise for the
       samples in bsel, stored as [n_bsel][N_in]. The optional *_abs outputs
       receive the sum of the absolute values of the terms of each gradient
       element (its conditioning, used to judge rounding).
       Error weights (test infrastructure): given per neuron a relative error
       rho of the slope and an absolute error delta of the spike time, the
       factor G[b,m,i] = gamma K(t - T_m) of a term moves by at most
       |gamma| (rho K(t - T_m) + delta |K'(t - T_m)|) to first order. The
       optional *_err outputs (rho, delta and both outputs given together)
       receive each element's sum over its terms of that bound times the
       term's other factors in absolute value. */
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
    int64_t ni = n_isel < 0 ? N_out : n_isel;
    int64_t nb = n_bsel < 0 ? B : n_bsel;
    int want_err = rho && delta;
    size_t ng = (size_t)(B * N_out * (M + 1) > 0 ? B * N_out * (M + 1) : 1);
    ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)(B * N_in > 0 ? B * N_in : 1));
    double *G = (double *)calloc(ng, sizeof(double));
    double *GE = want_err ? (double *)calloc(ng, sizeof(double)) : NULL;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        sample_events(&p, t_in + b * N_in, N_in, ev + b * N_in);
        for (int64_t i = 0; i < N_out; ++i) {
            int64_t o = b * N_out + i;
            int q = q_idx[o];
            if (q < 0 || grad_t_out[o] == 0.0) continue;
            double gam = -grad_t_out[o] / slope[o];
            for (int m = 0; m <= q; ++m) {
                double u = t_out[o] - grid(t0, dt, m);
                G[o * (M + 1) + m] = gam * kern(p.tv, p.ti, u);
                if (GE)
                    GE[o * (M + 1) + m] = fabs(gam) * (rho[o] * fabs(kern(p.tv, p.ti, u)) +
                                                       delta[o] * fabs(kern_dt(p.tv, p.ti, u)));
            }
        }
    }
    if (grad_t_in) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t r = 0; r < nb; ++r) {
            int64_t b = n_bsel < 0 ? r : bsel[r];
            for (int64_t j = 0; j < N_in; ++j) {
                const ev_t *e = ev + b * N_in + j;
                double acc = 0.0, aabs = 0.0, aerr = 0.0;
                for (int k = 0; k < e->n; ++k)
                    for (int64_t i = 0; i < N_out; ++i) {
                        int64_t g = (b * N_out + i) * (M + 1) + e->m[k];
                        double term = G[g] * W[i * N_in + j] * e->ds[k];
                        acc += term;
                        aabs += fabs(term);
                        if (GE) aerr += GE[g] * fabs(W[i * N_in + j] * e->ds[k]);
                    }
                grad_t_in[r * N_in + j] = acc;
                if (grad_t_in_abs) grad_t_in_abs[r * N_in + j] = aabs;
                if (GE && grad_t_in_err) grad_t_in_err[r * N_in + j] = aerr;
            }
        }
    }
    if (grad_W) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t r = 0; r < ni; ++r) {
            int64_t i = n_isel < 0 ? r : isel[r];
            for (int64_t j = 0; j < N_in; ++j) {
                double acc = 0.0, aabs = 0.0, aerr = 0.0;
                for (int64_t b = 0; b < B; ++b) {
                    const ev_t *e = ev + b * N_in + j;
                    for (int k = 0; k < e->n; ++k) {
                        int64_t g = (b * N_out + i) * (M + 1) + e->m[k];
                        double term = G[g] * e->s[k];
                        acc += term;
                        aabs += fabs(term);
                        if (GE) aerr += GE[g] * fabs(e->s[k]);
                    }
                }
                grad_W[r * N_in + j] = acc;
                if (grad_W_abs) grad_W_abs[r * N_in + j] = aabs;
                if (GE && grad_W_err) grad_W_err[r * N_in + j] = aerr;
            }
        }
    }
    free(ev);
    free(G);
    free(GE);
}

/* ------------------------------------------------------------------------ */
/* Exact continuous-time LIF spike times (App. A, Eq. (timing_exact), Alg. 1) */
/* ------------------------------------------------------------------------ */
typedef struct { double t; double w; } tw_t;

static int cmp_tw(const void *x, const void *y) {
    double a = ((const tw_t *)x)->t, b = ((const tw_t *)y)->t;
    return (a > b) - (a < b);
}

/* K'(t), the derivative of each row of Table "tab:kernel" with respect to its
   argument, for t >= 0 (the jump of the Heaviside factor at 0 is not part of
   it; at t = 0 this is the right derivative). */
static double kern_dt(double tv, double ti, double t) {
    if (t < 0.0) return 0.0;
    switch (row_of(tv, ti)) {
        case ROW_INF_INF: return 1.0;                                   /* d/dt t */
        case ROW_INF_TAU: return exp(-t / finite_of(tv, ti));          /* d/dt tau (1 - e^{-t/tau}) */
        case ROW_EQUAL: return exp(-t / tv) * (1.0 - t / tv);           /* d/dt t e^{-t/tau} */
        default: {
            double c = tv * ti / (tv - ti);
            return c * (exp(-t / ti) / ti - exp(-t / tv) / tv);        /* d/dt c (e^{-t/tv} - e^{-t/ti}) */
        }
    }
}

/*
 * Sort the presynaptic spikes ascending; on [t~_k, t~_{k+1}) the potential is
 * sum_{j<=k} w_j K(t - t~_j); take the first interval whose candidate lies in
 * it (t~_{N+1} = t_max, +inf by default). Non-finite inputs are silent.
 *
 * Optional outputs (NULL to skip):
 *  k_out  : position (0-based, ascending order of the finite inputs) of the
 *           left end of the crossing interval, -1 when the neuron is silent.
 *           Simultaneous spikes add up before their interval is tested, so
 *           this is the last position of a group of equal times: the causal
 *           set of the spike is exactly the inputs with t_j <= t~_k.
 *  margin : distance of the firing decision from the threshold, as for the
 *           DSTD scan: min over earlier intervals of (V_th - peak), and at the
 *           crossing interval |peak - V_th|, |v(t~_k) - V_th| and
 *           |v(t~_{k+1}) - V_th| (finite right end); silent neurons get the
 *           min over all intervals of (V_th - peak).
 *  vabs   : sum over the causal set of |w_j K(t - t_j)| at the spike (the
 *           magnitude of the terms of v(t) = V_th, for rounding estimates).
 */
void oracle_exact_forward(double tau_m, double tau_s, double theta, double t_max,
                          int64_t B, int64_t N_in, int64_t N_out,
                          const double *t_in, const double *W, double *t_out, double *slope,
                          int32_t *k_out, double *margin, double *vabs, double *emass) {
    /* emass (optional): sum over the causal set of |w_j| (all finite inputs
       for a silent neuron); with |K'| <= 1 it bounds the terms of the slope */
    double tv = fmax(tau_m, tau_s), ti = fmin(tau_m, tau_s);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        tw_t *s = (tw_t *)malloc(sizeof(tw_t) * (size_t)(N_in > 0 ? N_in : 1));
        for (int64_t i = 0; i < N_out; ++i) {
            int64_t n = 0;
            for (int64_t j = 0; j < N_in; ++j) {
                double t = t_in[b * N_in + j];
                if (isfinite(t)) { s[n].t = t; s[n].w = W[i * N_in + j]; ++n; }
            }
            qsort(s, (size_t)n, sizeof(tw_t), cmp_tw);
            double to = INFINITY, sl = 0.0, pre = INFINITY, mg = INFINITY, va = 0.0, em = 0.0;
            int32_t kk = -1;
            if (n > 0) {
                piece_t pc;
                piece_init(&pc, tv, ti, theta, s[0].t);
                for (int64_t k = 0; k < n; ++k) {
                    piece_add(&pc, s[k].w, s[k].t);
                    double lo = s[k].t;
                    double hi = (k + 1 < n) ? s[k + 1].t : t_max;
                    if (!(hi > lo)) continue; /* simultaneous spikes add up first */
                    if (lo >= t_max) break;
                    if (hi > t_max) hi = t_max;
                    double root, peak;
                    int hit = first_crossing(&pc, lo, hi, &root, &peak);
                    if (hit) {
                        to = root; sl = pdv(&pc, root); kk = (int32_t)k;
                        mg = fmin(pre, fabs(peak - theta));
                        mg = fmin(mg, fabs(pv(&pc, lo) - theta));
                        if (!isinf(hi)) mg = fmin(mg, fabs(pv(&pc, hi) - theta));
                        for (int64_t j = 0; j <= k; ++j) {
                            va += fabs(s[j].w * kern(tv, ti, root - s[j].t));
                            em += fabs(s[j].w);
                        }
                        break;
                    }
                    pre = fmin(pre, theta - peak);
                }
            }
            if (kk < 0) {
                mg = pre;
                for (int64_t j = 0; j < n; ++j) em += fabs(s[j].w);
            }
            if (emass) emass[b * N_out + i] = em;
            t_out[b * N_out + i] = to;
            slope[b * N_out + i] = sl;
            if (k_out) k_out[b * N_out + i] = kk;
            if (margin) margin[b * N_out + i] = mg;
            if (vabs) vabs[b * N_out + i] = va;
        }
        free(s);
    }
}

static int cmp_d(const void *x, const void *y) {
    double a = *(const double *)x, b = *(const double *)y;
    return (a > b) - (a < b);
}

/*
 * Gradients of the exact spike times (App. A, Eq. (timing_exact)) by the
 * implicit function theorem on v_i(t_i) = V_th with
 * v_i(t) = sum_{j in S_i} w_ij K(t - t_j), S_i = {j : t_j <= t~_k} the causal
 * set of the crossing interval k (the candidate of the selected interval is
 * that root, and the min over intervals is piecewise constant):
 *   d t_i / d w_ij = -K(t_i - t_j) / v'(t_i)
 *   d t_i / d t_j  =  w_ij K'(t_i - t_j) / v'(t_i)
 * so with g = dL/dt_out and gamma = -g / slope:
 *   grad_W[i][j]    = sum_b gamma_bi K(t_bi - t_bj)          (j in S_bi)
 *   grad_t_in[b][j] = -sum_i gamma_bi W_ij K'(t_bi - t_bj)   (j in S_bi)
 * Silent neurons (k < 0) and g = 0 contribute nothing; non-finite inputs get
 * zero gradient. *_abs (optional) receive the sums of |terms|.
 */
void oracle_exact_backward(double tau_m, double tau_s, int64_t B, int64_t N_in, int64_t N_out,
                           const double *t_in, const double *W, const double *t_out,
                           const double *slope, const int32_t *k_idx, const double *grad_t_out,
                           double *grad_W, double *grad_t_in, double *grad_W_abs,
                           double *grad_t_in_abs, const double *rho, const double *delta,
                           double *grad_W_err, double *grad_t_in_err) {
    /* Error weights (test infrastructure; rho, delta [B][N_out] and both
       outputs given together): with a relative slope error rho and a spike
       time error delta, gamma K(t - t_j) moves by at most
       |gamma| (rho K + delta |K'|) and gamma K'(t - t_j) by at most
       |gamma| (rho |K'| + delta (1/tau_v + 1/tau_I)), the last factor bounding
       |K''| on every row. *_err receive each element's sum of these bounds
       times the term's other factors in absolute value. */
    int want_err = rho && delta && grad_W_err && grad_t_in_err;
    double k2 = 1.0 / fmax(tau_m, tau_s) + 1.0 / fmin(tau_m, tau_s);
    double tv = fmax(tau_m, tau_s), ti = fmin(tau_m, tau_s);
    double *gam = (double *)calloc((size_t)(B * N_out > 0 ? B * N_out : 1), sizeof(double));
    double *tl = (double *)calloc((size_t)(B * N_out > 0 ? B * N_out : 1), sizeof(double));
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        double *ts = (double *)malloc(sizeof(double) * (size_t)(N_in > 0 ? N_in : 1));
        int64_t n = 0;
        for (int64_t j = 0; j < N_in; ++j)
            if (isfinite(t_in[b * N_in + j])) ts[n++] = t_in[b * N_in + j];
        qsort(ts, (size_t)n, sizeof(double), cmp_d);
        for (int64_t i = 0; i < N_out; ++i) {
            int64_t o = b * N_out + i;
            int32_t k = k_idx[o];
            if (k < 0 || k >= n || grad_t_out[o] == 0.0) continue;
            gam[o] = -grad_t_out[o] / slope[o];
            tl[o] = ts[k];
        }
        free(ts);
    }
    if (grad_W) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t i = 0; i < N_out; ++i)
            for (int64_t j = 0; j < N_in; ++j) {
                double acc = 0.0, aabs = 0.0, aerr = 0.0;
                for (int64_t b = 0; b < B; ++b) {
                    int64_t o = b * N_out + i;
                    double t = t_in[b * N_in + j];
                    if (gam[o] == 0.0 || !isfinite(t) || !(t <= tl[o])) continue;
                    double term = gam[o] * kern(tv, ti, t_out[o] - t);
                    acc += term;
                    aabs += fabs(term);
                    if (want_err)
                        aerr += fabs(gam[o]) * (rho[o] * fabs(kern(tv, ti, t_out[o] - t)) +
                                                delta[o] * fabs(kern_dt(tv, ti, t_out[o] - t)));
                }
                grad_W[i * N_in + j] = acc;
                if (grad_W_abs) grad_W_abs[i * N_in + j] = aabs;
                if (want_err) grad_W_err[i * N_in + j] = aerr;
            }
    }
    if (grad_t_in) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t j = 0; j < N_in; ++j) {
                double acc = 0.0, aabs = 0.0, aerr = 0.0, t = t_in[b * N_in + j];
                if (isfinite(t))
                    for (int64_t i = 0; i < N_out; ++i) {
                        int64_t o = b * N_out + i;
                        if (gam[o] == 0.0 || !(t <= tl[o])) continue;
                        double kd = kern_dt(tv, ti, t_out[o] - t);
                        double term = -gam[o] * W[i * N_in + j] * kd;
                        acc += term;
                        aabs += fabs(term);
                        if (want_err)
                            aerr += fabs(gam[o] * W[i * N_in + j]) * (rho[o] * fabs(kd) + delta[o] * k2);
                    }
                grad_t_in[b * N_in + j] = acc;
                if (grad_t_in_abs) grad_t_in_abs[b * N_in + j] = aabs;
                if (want_err) grad_t_in_err[b * N_in + j] = aerr;
            }
    }
    free(gam);
    free(tl);
}

/* ------------------------------------------------------------------------ */
/* Multi-spike DSTD (App. "multi-spikes", Eq. (Vmem_multiSpikes) and the      */
/* DSTD form after it).                                                      */
/*                                                                           */
/* Each input neuron j may fire F_in times; every input spike gets its own   */
/* events s_jm^f and the weighted events sum them. After an output spike at  */
/* t_k the membrane potential is reset to 0 and the synaptic current is not, */
/* so from t_k on                                                            */
/*   v(t) = I(t_k) K(t - t_k) + sum_{t_k < T_q <= t} w^_q K(t - T_q),        */
/*   I(t_k) = sum_{T_q <= t_k} w^_q e^{-(t_k - T_q)/tau_I}.                  */
/* The spikes are the successive first crossings of V_th (several may fall   */
/* in one interval); the first F_out are kept.                               */
/* ------------------------------------------------------------------------ */

/* current at time t from the events at T_0..T_q (T_q <= t) */
static double ms_current(const prm_t *p, const double *wh, int q, double t) {
    double I = 0.0;
    for (int m = 0; m <= q; ++m) I += wh[m] * exp(-(t - grid(p->t0, p->dt, m)) / p->ti);
    return I;
}

/* coefficient of w^_m in v_k(t_k): K(t_k - T_m) for T_m after the previous
   spike (m > q_prev), e^{-(t_prev - T_m)/tau_I} K(t_k - t_prev) for T_m at or
   before it (m <= q_prev), 0 after t_k (m > q_k); q_prev = -1 for k = 0 */
static double ms_coef(const prm_t *p, int m, double tk, int qk, double tprev, int qprev) {
    if (m > qk) return 0.0;
    double Tm = grid(p->t0, p->dt, m);
    if (m > qprev) return kern(p->tv, p->ti, tk - Tm);
    return exp(-(tprev - Tm) / p->ti) * kern(p->tv, p->ti, tk - tprev);
}

/* scan of one neuron with reset; outputs per spike k < F (unset spikes:
   t = +inf, slope 0, q -1, cur 0, margin min over the rest of the grid) */
static void ms_scan(const prm_t *p, const double *wh, const double *wabs, int F, double *t_out,
                    double *slope, int32_t *q_out, double *cur, double *margin, double *vabs) {
    for (int k = 0; k < F; ++k) {
        t_out[k] = INFINITY; slope[k] = 0.0; q_out[k] = -1; cur[k] = 0.0;
        if (margin) margin[k] = INFINITY;
        if (vabs) vabs[k] = 0.0;
    }
    int nk = 0, qprev = -1;
    double tprev = -INFINITY, pre = INFINITY;
    piece_t pc;
    piece_init(&pc, p->tv, p->ti, p->theta, p->t0);
    for (int q = 0; q <= p->M && nk < F; ++q) {
        double Tq = grid(p->t0, p->dt, q);
        piece_add(&pc, wh[q], Tq);
        double hi = (q < p->M) ? grid(p->t0, p->dt, q + 1) : p->t_max;
        double lo = Tq > tprev ? Tq : tprev;
        while (nk < F) {
            double root, peak;
            if (!(hi > lo) || !first_crossing(&pc, lo, hi, &root, &peak)) {
                if (hi > lo) pre = fmin(pre, p->theta - peak);
                break;
            }
            double mg = fmin(pre, fabs(peak - p->theta));
            mg = fmin(mg, fabs(pv(&pc, lo) - p->theta));
            if (q < p->M) mg = fmin(mg, fabs(pv(&pc, hi) - p->theta));
            t_out[nk] = root;
            slope[nk] = pdv(&pc, root);
            q_out[nk] = q;
            cur[nk] = ms_current(p, wh, q, root);
            if (margin) margin[nk] = mg;
            if (vabs) {
                double va = 0.0;
                for (int m = 0; m <= q; ++m)
                    va += wabs[m] * fabs(ms_coef(p, m, root, q, tprev, qprev));
                vabs[nk] = va;
            }
            ++nk;
            /* reset: v = 0 at root, the current carries on */
            tprev = root;
            qprev = q;
            piece_init(&pc, p->tv, p->ti, p->theta, root);
            piece_add(&pc, cur[nk - 1], root);
            pre = INFINITY;
            lo = root;
        }
    }
    if (margin && nk < F) margin[nk] = pre;
}

/*
 * Forward: t_in [B][N_in][F_in] (non-finite = no spike), W [N_out][N_in];
 * per output spike [B][N_out][F_out]: t_out (+inf = none), slope, q_idx
 * (-1 = none), cur = I(t_k) (the current at the spike, which carries over the
 * reset), and optionally margin, vabs, and dprev = d t_k / d t_{k-1} through
 * the reset (0 for k = 0):
 *   d t_k / d t_{k-1} = I(t_{k-1}) (K(d)/tau_I + K'(d)) / slope_k,  d = t_k - t_{k-1}.
 */
void oracle_ms_forward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                       double t_max, int64_t B, int64_t N_in, int64_t F_in, int64_t N_out,
                       int64_t F_out, const double *t_in, const double *W, double *t_out,
                       double *slope, int32_t *q_idx, double *cur, double *margin, double *vabs,
                       double *dprev) {
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
    int64_t NV = N_in * F_in;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)(NV > 0 ? NV : 1));
        double *wh = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        double *wabs = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        sample_events(&p, t_in + b * NV, NV, ev); /* every input spike */
        for (int64_t i = 0; i < N_out; ++i) {
            for (int m = 0; m <= M; ++m) { wh[m] = 0.0; wabs[m] = 0.0; }
            const double *wr = W + i * N_in;
            for (int64_t v = 0; v < NV; ++v)
                for (int k = 0; k < ev[v].n; ++k) {
                    wh[ev[v].m[k]] += wr[v / F_in] * ev[v].s[k];
                    wabs[ev[v].m[k]] += fabs(wr[v / F_in] * ev[v].s[k]);
                }
            int64_t o = (b * N_out + i) * F_out;
            ms_scan(&p, wh, wabs, (int)F_out, t_out + o, slope + o, q_idx + o, cur + o,
                    margin ? margin + o : NULL, vabs ? vabs + o : NULL);
            if (dprev)
                for (int64_t k = 0; k < F_out; ++k) {
                    dprev[o + k] = 0.0;
                    if (k == 0 || q_idx[o + k] < 0) continue;
                    double d = t_out[o + k] - t_out[o + k - 1];
                    dprev[o + k] = cur[o + k - 1] * (kern(p.tv, p.ti, d) / p.ti + kern_dt(p.tv, p.ti, d)) /
                                   slope[o + k];
                }
        }
        free(ev); free(wh); free(wabs);
    }
}

/*
 * Backward by the implicit function theorem on each spike's v_k(t_k) = V_th,
 * with the intervals fixed: F_k depends on w^ and, through the reset, on
 * t_{k-1} (dF_k/dt_{k-1} = -I(t_{k-1}) (K(d)/tau_I + K'(d))). Adjoints run
 * from the last spike back: gbar_k = g_k + gbar_{k+1} (d t_{k+1} / d t_k),
 * gamma_k = -gbar_k / slope_k, and dL/dw^_m = sum_k gamma_k dF_k/dw^_m with
 * the coefficients of ms_coef; then dW and dt_in through the events as in the
 * single-spike backward (every input spike has its own events and slope
 * derivative). grad_t_in is [B][N_in][F_in]; *_abs (optional) get the sums
 * of |terms|.
 */
void oracle_ms_backward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                        double t_max, int64_t B, int64_t N_in, int64_t F_in, int64_t N_out,
                        int64_t F_out, const double *t_in, const double *W, const double *t_out,
                        const double *slope, const int32_t *q_idx, const double *cur,
                        const double *grad_t_out, double *grad_W, double *grad_t_in,
                        double *grad_W_abs, double *grad_t_in_abs) {
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
    int64_t NV = N_in * F_in;
    ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)(B * NV > 0 ? B * NV : 1));
    double *G = (double *)calloc((size_t)(B * N_out * (M + 1) > 0 ? B * N_out * (M + 1) : 1),
                                 sizeof(double));
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        sample_events(&p, t_in + b * NV, NV, ev + b * NV);
        double *gb = (double *)malloc(sizeof(double) * (size_t)(F_out > 0 ? F_out : 1));
        for (int64_t i = 0; i < N_out; ++i) {
            int64_t o = (b * N_out + i) * F_out;
            int K = 0;
            while (K < F_out && q_idx[o + K] >= 0) ++K;
            for (int k = K - 1; k >= 0; --k) {
                gb[k] = grad_t_out[o + k];
                if (k + 1 < K) {
                    double d = t_out[o + k + 1] - t_out[o + k];
                    double dFdprev = -cur[o + k] * (kern(p.tv, p.ti, d) / p.ti + kern_dt(p.tv, p.ti, d));
                    gb[k] += gb[k + 1] * (-dFdprev / slope[o + k + 1]);
                }
            }
            double *Gi = G + (b * N_out + i) * (M + 1);
            for (int k = 0; k < K; ++k) {
                double gam = -gb[k] / slope[o + k];
                double tprev = k > 0 ? t_out[o + k - 1] : -INFINITY;
                int qprev = k > 0 ? q_idx[o + k - 1] : -1;
                for (int m = 0; m <= q_idx[o + k]; ++m)
                    Gi[m] += gam * ms_coef(&p, m, t_out[o + k], q_idx[o + k], tprev, qprev);
            }
        }
        free(gb);
    }
    if (grad_t_in) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b)
            for (int64_t v = 0; v < NV; ++v) {
                const ev_t *e = ev + b * NV + v;
                double acc = 0.0, aabs = 0.0;
                for (int k = 0; k < e->n; ++k)
                    for (int64_t i = 0; i < N_out; ++i) {
                        double term = G[(b * N_out + i) * (M + 1) + e->m[k]] * W[i * N_in + v / F_in] * e->ds[k];
                        acc += term;
                        aabs += fabs(term);
                    }
                grad_t_in[b * NV + v] = acc;
                if (grad_t_in_abs) grad_t_in_abs[b * NV + v] = aabs;
            }
    }
    if (grad_W) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int64_t i = 0; i < N_out; ++i)
            for (int64_t j = 0; j < N_in; ++j) {
                double acc = 0.0, aabs = 0.0;
                for (int64_t b = 0; b < B; ++b)
                    for (int64_t f = 0; f < F_in; ++f) {
                        const ev_t *e = ev + b * NV + j * F_in + f;
                        for (int k = 0; k < e->n; ++k) {
                            double term = G[(b * N_out + i) * (M + 1) + e->m[k]] * e->s[k];
                            acc += term;
                            aabs += fabs(term);
                        }
                    }
                grad_W[i * N_in + j] = acc;
                if (grad_W_abs) grad_W_abs[i * N_in + j] = aabs;
            }
    }
    free(ev);
    free(G);
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Convolutional DSTD-LIF layer.                                             */
/*                                                                           */
/* A conv layer is a dense layer whose weight matrix is the convolution's    */
/* (sparse, shared) connectivity, so w^_im = sum_j w_ij s_jm of App. B.1      */
/* holds with j ranging over the receptive field of output neuron i. Inputs  */
/* are NCHW [B][C_in][H][W]; W is [C_out][C_in][KH][KW]; outputs NCHW.        */
/* pool_in = 2 averages the input events over 2x2 windows before the         */
/* convolution, pool_in = 0 averages them over the whole map (global pool),   */
/* pool_in = 1 uses them as they are. Averaging events is linear, so it is    */
/* the same as averaging the synaptic input currents (reading: the paper's    */
/* own nets down-sample with stride-2 convolutions, Table "tab:architectures",*/
/* and do not define spike pooling).                                         */
/* ------------------------------------------------------------------------ */
typedef struct {
    int C_in, H, W, C_out, KH, KW, stride, pad, pool;
    int Hp, Wp, Ho, Wo, P; /* pooled input map, output map, pool size */
} cgeom_t;

static void cgeom(cgeom_t *g, int C_in, int H, int W, int C_out, int KH, int KW, int stride,
                  int pad, int pool) {
    g->C_in = C_in; g->H = H; g->W = W; g->C_out = C_out; g->KH = KH; g->KW = KW;
    g->stride = stride; g->pad = pad; g->pool = pool;
    if (pool == 2) { g->Hp = H / 2; g->Wp = W / 2; g->P = 4; }
    else if (pool == 0) { g->Hp = 1; g->Wp = 1; g->P = H * W; }
    else { g->Hp = H; g->Wp = W; g->P = 1; }
    g->Ho = (g->Hp + 2 * pad - KH) / stride + 1;
    g->Wo = (g->Wp + 2 * pad - KW) / stride + 1;
}

/* raw input pixels (y, x) that pool into pooled cell (py, px) */
static int pool_cells(const cgeom_t *g, int py, int px, int *ys, int *xs) {
    int n = 0;
    if (g->pool == 2) {
        for (int dy = 0; dy < 2; ++dy)
            for (int dx = 0; dx < 2; ++dx) { ys[n] = 2 * py + dy; xs[n] = 2 * px + dx; ++n; }
    } else if (g->pool == 0) {
        for (int y = 0; y < g->H; ++y)
            for (int x = 0; x < g->W; ++x) { ys[n] = y; xs[n] = x; ++n; }
    } else { ys[0] = py; xs[0] = px; n = 1; }
    return n;
}

void oracle_conv_forward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                         double t_max, int64_t B, int C_in, int H, int Wd, int C_out, int KH,
                         int KW, int stride, int pad, int pool,
                         const double *t_in, const double *W,
                         double *t_out, double *slope, int32_t *q_idx, double *margin, double *vabs,
                         double *emass) {
    /* margin, vabs and emass as for oracle_dstd_forward */
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
    cgeom_t g;
    cgeom(&g, C_in, H, Wd, C_out, KH, KW, stride, pad, pool);
    int64_t nin = (int64_t)C_in * H * Wd;
    int64_t nout = (int64_t)C_out * g.Ho * g.Wo;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < B; ++b) {
        ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)nin);
        double *wh = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        double *wabs = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        int *ys = (int *)malloc(sizeof(int) * (size_t)(H * Wd));
        int *xs = (int *)malloc(sizeof(int) * (size_t)(H * Wd));
        sample_events(&p, t_in + b * nin, nin, ev);
        for (int co = 0; co < C_out; ++co)
            for (int oy = 0; oy < g.Ho; ++oy)
                for (int ox = 0; ox < g.Wo; ++ox) {
                    for (int m = 0; m <= M; ++m) { wh[m] = 0.0; wabs[m] = 0.0; }
                    for (int ci = 0; ci < C_in; ++ci)
                        for (int ky = 0; ky < KH; ++ky)
                            for (int kx = 0; kx < KW; ++kx) {
                                int py = oy * stride + ky - pad, px = ox * stride + kx - pad;
                                if (py < 0 || py >= g.Hp || px < 0 || px >= g.Wp) continue;
                                double w = W[((co * C_in + ci) * KH + ky) * KW + kx] / g.P;
                                int nc = pool_cells(&g, py, px, ys, xs);
                                for (int r = 0; r < nc; ++r) {
                                    const ev_t *e = ev + ((int64_t)ci * H + ys[r]) * Wd + xs[r];
                                    for (int k = 0; k < e->n; ++k) {
                                        wh[e->m[k]] += w * e->s[k];
                                        wabs[e->m[k]] += fabs(w * e->s[k]);
                                    }
                                }
                            }
                    double to, sl, mg; int q;
                    dstd_scan(&p, wh, &to, &sl, &q, &mg, NULL);
                    int64_t o = b * nout + ((int64_t)co * g.Ho + oy) * g.Wo + ox;
                    t_out[o] = to; slope[o] = sl; q_idx[o] = q;
                    if (margin) margin[o] = mg;
                    if (vabs) {
                        double va = 0.0;
                        for (int m = 0; m <= (q < 0 ? -1 : q); ++m)
                            va += fabs(kern(p.tv, p.ti, to - grid(t0, dt, m))) * wabs[m];
                        vabs[o] = va;
                    }
                    if (emass) {
                        double em = 0.0;
                        for (int m = 0; m <= (q < 0 ? M : q); ++m) em += wabs[m];
                        emass[o] = em;
                    }
                }
        free(ev); free(wh); free(wabs); free(ys); free(xs);
    }
}

/* Backward of the conv layer: the dense-layer chain rule over the conv's
   connectivity (and through the linear event pooling). */
void oracle_conv_backward(double tau_m, double tau_s, double theta, int M, double t0, double dt,
                          double t_max, int64_t B, int C_in, int H, int Wd, int C_out, int KH,
                          int KW, int stride, int pad, int pool,
                          const double *t_in, const double *W,
                          const double *t_out, const double *slope, const int32_t *q_idx,
                          const double *grad_t_out, double *grad_W, double *grad_t_in,
                          double *grad_W_abs, double *grad_t_in_abs,
                          const double *rho, const double *delta,
                          double *grad_W_err, double *grad_t_in_err) {
    /* The optional *_abs outputs (NULL to skip) receive, per gradient element,
       the sum of the absolute values of its terms (its conditioning). The
       optional error weights rho, delta [B][C_out][Ho][Wo] and *_err outputs
       are those of oracle_dstd_backward (all four given together). */
    prm_t p;
    canon(&p, tau_m, tau_s);
    p.theta = theta; p.M = M; p.t0 = t0; p.dt = dt; p.t_max = t_max;
    (void)theta;
    cgeom_t g;
    cgeom(&g, C_in, H, Wd, C_out, KH, KW, stride, pad, pool);
    int64_t nin = (int64_t)C_in * H * Wd;
    int64_t nout = (int64_t)C_out * g.Ho * g.Wo;
    int64_t nw = (int64_t)C_out * C_in * KH * KW;
    int nth = 1;
#ifdef _OPENMP
    nth = omp_get_max_threads();
#endif
    int want_err = rho && delta && grad_W_err && grad_t_in_err;
    double *dWp = (double *)calloc((size_t)(nw * nth), sizeof(double));
    double *dWa = (double *)calloc((size_t)(nw * nth), sizeof(double));
    double *dWe = (double *)calloc((size_t)(nw * nth), sizeof(double));
    memset(grad_t_in, 0, sizeof(double) * (size_t)(B * nin));
    if (grad_t_in_abs) memset(grad_t_in_abs, 0, sizeof(double) * (size_t)(B * nin));
    if (want_err) memset(grad_t_in_err, 0, sizeof(double) * (size_t)(B * nin));
#pragma omp parallel
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double *dWl = dWp + (int64_t)tid * nw;
        double *dWal = dWa + (int64_t)tid * nw;
        double *dWel = dWe + (int64_t)tid * nw;
        ev_t *ev = (ev_t *)malloc(sizeof(ev_t) * (size_t)nin);
        double *G = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        double *GE = (double *)malloc(sizeof(double) * (size_t)(M + 1));
        int *ys = (int *)malloc(sizeof(int) * (size_t)(H * Wd));
        int *xs = (int *)malloc(sizeof(int) * (size_t)(H * Wd));
#pragma omp for schedule(dynamic, 1)
        for (int64_t b = 0; b < B; ++b) {
            sample_events(&p, t_in + b * nin, nin, ev);
            double *dt_row = grad_t_in + b * nin;
            double *dta_row = grad_t_in_abs ? grad_t_in_abs + b * nin : NULL;
            double *dte_row = want_err ? grad_t_in_err + b * nin : NULL;
            for (int co = 0; co < C_out; ++co)
                for (int oy = 0; oy < g.Ho; ++oy)
                    for (int ox = 0; ox < g.Wo; ++ox) {
                        int64_t o = b * nout + ((int64_t)co * g.Ho + oy) * g.Wo + ox;
                        int q = q_idx[o];
                        if (q < 0 || grad_t_out[o] == 0.0) continue;
                        double gam = -grad_t_out[o] / slope[o];
                        for (int m = 0; m <= M; ++m) {
                            double u = t_out[o] - grid(t0, dt, m);
                            G[m] = (m <= q) ? gam * kern(p.tv, p.ti, u) : 0.0;
                            GE[m] = (m <= q && want_err)
                                        ? fabs(gam) * (rho[o] * fabs(kern(p.tv, p.ti, u)) +
                                                       delta[o] * fabs(kern_dt(p.tv, p.ti, u)))
                                        : 0.0;
                        }
                        for (int ci = 0; ci < C_in; ++ci)
                            for (int ky = 0; ky < KH; ++ky)
                                for (int kx = 0; kx < KW; ++kx) {
                                    int py = oy * stride + ky - pad, px = ox * stride + kx - pad;
                                    if (py < 0 || py >= g.Hp || px < 0 || px >= g.Wp) continue;
                                    int64_t widx = ((int64_t)(co * C_in + ci) * KH + ky) * KW + kx;
                                    double w = W[widx];
                                    int nc = pool_cells(&g, py, px, ys, xs);
                                    for (int r = 0; r < nc; ++r) {
                                        int64_t jin = ((int64_t)ci * H + ys[r]) * Wd + xs[r];
                                        const ev_t *e = ev + jin;
                                        for (int k = 0; k < e->n; ++k) {
                                            double tw = G[e->m[k]] * e->s[k] / g.P;
                                            double tt = G[e->m[k]] * w * e->ds[k] / g.P;
                                            dWl[widx] += tw;
                                            dWal[widx] += fabs(tw);
                                            dt_row[jin] += tt;
                                            if (dta_row) dta_row[jin] += fabs(tt);
                                            if (want_err) {
                                                dWel[widx] += GE[e->m[k]] * fabs(e->s[k]) / g.P;
                                                dte_row[jin] += GE[e->m[k]] * fabs(w * e->ds[k]) / g.P;
                                            }
                                        }
                                    }
                                }
                    }
        }
        free(ev); free(G); free(GE); free(ys); free(xs);
    }
    for (int64_t k = 0; k < nw; ++k) {
        double s = 0.0, a = 0.0, e = 0.0;
        for (int t = 0; t < nth; ++t) {
            s += dWp[(int64_t)t * nw + k];
            a += dWa[(int64_t)t * nw + k];
            e += dWe[(int64_t)t * nw + k];
        }
        grad_W[k] = s;
        if (grad_W_abs) grad_W_abs[k] = a;
        if (want_err) grad_W_err[k] = e;
    }
    free(dWp);
    free(dWa);
    free(dWe);
}
