// dstd_internal.h -- device-side building blocks shared by the DSTD-LIF
// kernels (gfx950). Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

namespace dstd {

constexpr int kWave = 64;  // CDNA wavefront width

// The rows of Table "tab:kernel" this library evaluates: the general row
// (tau_v != tau_I, both finite) and the three closed-form limits.
enum KernelKind : int {
    kGeneral = 0,  // K = c (e^{-u/tv} - e^{-u/ti})
    kEqual = 1,    // (tau, tau):  K = u e^{-u/tau}
    kInfTau = 2,   // (inf, tau):  K = tau (1 - e^{-u/tau})
    kInfInf = 3,   // (inf, inf):  K = u
};

// Kernels take the row as a compile-time hint KS: a KernelKind when the
// launcher knows it (the general row gets code without the other rows'
// branches), kAnyKind to switch on LifConst::kind at run time.
constexpr int kAnyKind = -1;

// Layer constants, computed once per call on the host in double precision and
// rounded to fp32. The kernel K (Table "tab:kernel") is symmetric in the time
// constants; tv >= ti is the canonical order (an infinite constant is tv; the
// finite one of the (inf, tau) row is ti, as is the common one of (tau, tau)).
// Every case keeps the state form v(T_q + u) = V e^{-u/tv} + I K(u) with the
// current decaying as e^{-u/ti}; a 1/inf is stored as 0 (e^0 = 1).
struct LifConst {
    int kind;              // KernelKind
    float tv, ti;          // time constants, tv >= ti (tv may be +inf)
    float inv_tv, inv_ti;  // 1/tv, 1/ti (0 for an infinite constant)
    float c;               // tv*ti/(tv - ti)
    float kappa;           // 1/ti - 1/tv > 0
    float alpha, beta;     // exp(-dt/tv), exp(-dt/ti): one-interval decays
    float k_dt;            // K(dt)
    float inv_em1;         // 1/expm1(-kappa*dt)  (< 0)
    float theta;           // V_th
    float t0, dt;          // grid T_m = t0 + m*dt
    float last_len;        // t_max - T_M (may be +inf)
    float slope_floor;     // smallest slope used in the backward pass
    int M;                 // intervals; M+1 grid points
    // fp64 copies for the O(M) recurrences (state propagation over all
    // intervals), so their rounding does not grow with M
    double alpha_d, beta_d, k_dt_d;
    // e^{-kappa*len} for len = dt and for the last interval: the interior
    // maximum u* of v lies inside [0, len) iff e^{-kappa u*} is in (this, 1)
    float r_lo_dt, r_lo_last;
    // closed-form rows: 1/dt, and for (inf, tau) e^{-dt/tau} and
    // 1/(1 - e^{-dt/tau})
    float inv_dt, e_mdt, inv_D;
    // the scan's interval filter in fp64: max K on [0, dt] and on the last
    // interval, and theta / 1.0001 (the filter's margin)
    double kmax_dt_d, kmax_last_d, theta_lo_d;
    // max K over the whole window [0, t_max - T_0] (+inf where K grows
    // without bound): with no further input, v never exceeds
    // max(V, 0) + max(I, 0) kpeak_d
    double kpeak_d;
    // curvature bound of one interval of length dt: dt^2/8 times 1/tv^2 and
    // times max |K''| on [0, dt] (the filter of the intervals before T_M)
    double curv_v_d, curv_i_d;
    int twice;  // general row with tv = 2 ti exactly: closed-form crossing
};

template <int KS> __device__ __forceinline__ int kind_of(const LifConst &C) {
    return (KS >= 0) ? KS : C.kind;
}

struct LifConst;
template <int KS> __device__ __forceinline__ int kind_of(const LifConst &C);

// Event rows in LDS / G tables: row r holds grid point m = r - 1, so the
// dropped halves of inputs at the grid ends land in the two zero rows
// r = 0 (m = -1) and r = M + 2 (m = M + 1).
__device__ __forceinline__ int rows_of(const LifConst &C) { return C.M + 3; }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

template <typename WT> struct WLoad;
template <> struct WLoad<float> {
    static __device__ __forceinline__ float get(const float *p, int64_t k) { return p[k]; }
};
template <> struct WLoad<uint16_t> {
    static __device__ __forceinline__ float get(const uint16_t *p, int64_t k) { return bf16_to_f32(p[k]); }
};

// K(u), u >= 0 (Table "tab:kernel"). General row: c (e^{-u/tv} - e^{-u/ti})
// = -c e^{-u/tv} expm1(-kappa u), written with expm1 so small u keeps full
// relative precision; likewise tau (1 - e^{-u/tau}) = -tau expm1(-u/tau).
template <int KS = kAnyKind>
__device__ __forceinline__ float kern(const LifConst &C, float u) {
    switch (kind_of<KS>(C)) {
        case kEqual: return u * expf(-u * C.inv_ti);
        case kInfTau: return -C.ti * expm1f(-u * C.inv_ti);
        case kInfInf: return u;
        default: return -C.c * expf(-u * C.inv_tv) * expm1f(-C.kappa * u);
    }
}

// DSTD events of one input spike (Eq. (DSTD_kernel), Table "tab:DSTD_kernels"),
// in forms without cancellation, with q = floor((t - t0)/dt),
// x = t - T_q in [0, dt), y = dt - x:
//   general : L = e^{x/tv} expm1(-kappa y) / expm1(-kappa dt)      (at T_q)
//             R = e^{-y/ti} expm1(-kappa x) / expm1(-kappa dt)     (at T_{q+1})
//   (tau,tau): L = (y/dt) e^{x/tau},   R = (x/dt) e^{-y/tau}
//   (inf,tau): L = (1 - e^{-y/tau}) / D,  R = e^{-dt/tau} (e^{x/tau} - 1) / D,
//              D = 1 - e^{-dt/tau}
//   (inf,inf): L = y/dt,  R = x/dt
// and their derivatives with respect to t. `row` = q + 1 (the LDS row of T_q),
// or -1 when the input contributes nothing (non-finite or out of
// [T_0 - dt, T_M + dt)). Halves that fall outside the grid are zeroed.
struct Event { int row; float L, R, dL, dR; };

// Event row of an input spike time (q + 1), or -1 if it has no events.
__device__ __forceinline__ int bin_row(const LifConst &C, float t) {
    if (!isfinite(t)) return -1;
    float qf = floorf((t - C.t0) / C.dt);
    if (!(qf >= -1.f && qf <= static_cast<float>(C.M))) return -1;
    return static_cast<int>(qf) + 1;
}

template <int KS = kAnyKind>
__device__ __forceinline__ Event bin_event(const LifConst &C, float t) {
    const int kind = kind_of<KS>(C);
    Event e{-1, 0.f, 0.f, 0.f, 0.f};
    const int row = bin_row(C, t);
    if (row < 0) return e;
    float rel = t - C.t0;
    int q = row - 1;
    float qf = static_cast<float>(q);
    float x = fmaf(-qf, C.dt, rel);
    x = fminf(fmaxf(x, 0.f), C.dt);
    float y = C.dt - x;
    if (kind == kEqual) {
        const float ex = expf(x * C.inv_ti), ey = expf(-y * C.inv_ti);
        e.L = y * C.inv_dt * ex;
        e.R = x * C.inv_dt * ey;
        e.dL = ex * C.inv_dt * fmaf(y, C.inv_ti, -1.f);
        e.dR = ey * C.inv_dt * fmaf(x, C.inv_ti, 1.f);
    } else if (kind == kInfTau) {
        const float ey = expf(-y * C.inv_ti);
        e.L = -expm1f(-y * C.inv_ti) * C.inv_D;
        e.R = C.e_mdt * expm1f(x * C.inv_ti) * C.inv_D;
        e.dR = ey * C.inv_ti * C.inv_D;
        e.dL = -e.dR;
    } else if (kind == kInfInf) {
        e.L = y * C.inv_dt;
        e.R = x * C.inv_dt;
        e.dL = -C.inv_dt;
        e.dR = C.inv_dt;
    } else {
        float ex = expf(x * C.inv_tv);
        float ey = expf(-y * C.inv_ti);
        float my = expm1f(-C.kappa * y);
        float mx = expm1f(-C.kappa * x);
        e.L = ex * my * C.inv_em1;
        e.R = ey * mx * C.inv_em1;
        e.dL = ex * (my * C.inv_tv + C.kappa * (1.f + my)) * C.inv_em1;
        e.dR = ey * (mx * C.inv_ti - C.kappa * (1.f + mx)) * C.inv_em1;
    }
    if (q < 0) { e.L = 0.f; e.dL = 0.f; }
    if (q >= C.M) { e.R = 0.f; e.dR = 0.f; }
    e.row = q + 1;
    return e;
}

// Per-sample lists of the inputs with events, sorted by event row, as
// structure-of-arrays (each array [B][stride]); rs[b][r] (r = 0..M+3) is the
// start of event row r in sample b's list (rs[b][M+3] = its length).
struct SortedEv { int *j; int *r; float *L; float *R; int64_t stride; int *rs; };

// Potential inside one interval, relative to its left grid point:
//   v(u) = V e^{-u/tv} + I K(u)
// where V = v(T_q) and I is the synaptic current just after the event at T_q
// (the state-space form of v^(t) = sum_{m<=q} w^_m K(t - T_m)).
struct Seg { float V, I; };

template <int KS = kAnyKind>
__device__ __forceinline__ void seg_eval(const LifConst &C, const Seg &s, float u, float &f,
                                         float &fp) {
    const int kind = kind_of<KS>(C);
    if (kind == kEqual) {  // v = (V + I u) e^{-u/tau}
        const float e = expf(-u * C.inv_ti);
        const float a = fmaf(s.I, u, s.V);
        f = a * e - C.theta;
        fp = e * fmaf(-a, C.inv_ti, s.I);
        return;
    }
    if (kind == kInfTau) {  // v = V + I tau (1 - e^{-u/tau})
        f = fmaf(s.I, -C.ti * expm1f(-u * C.inv_ti), s.V) - C.theta;
        fp = s.I * expf(-u * C.inv_ti);
        return;
    }
    if (kind == kInfInf) {  // v = V + I u
        f = fmaf(s.I, u, s.V) - C.theta;
        fp = s.I;
        return;
    }
    float ev = expf(-u * C.inv_tv);
    float em = expm1f(-C.kappa * u);
    float K = -C.c * ev * em;
    float Kp = C.c * ev * (C.kappa + em * C.inv_ti);  // K'(u)
    f = fmaf(s.V, ev, s.I * K) - C.theta;
    fp = fmaf(-s.V * C.inv_tv, ev, s.I * Kp);
}

// v - theta and its first two u-derivatives on one segment, from the
// hardware exponential (relative error ~1e-6): good enough to home in on a
// root, not to place it. Rows with a root solve only: general and (tau, tau).
//   general:    v'' = V e^{-u/tv}/tv^2 + I c (e^{-u/tv}/tv^2 - e^{-u/ti}/ti^2)
//   (tau, tau): v'' = -(e^{-u/tau}/tau) (I + v')  with v' = e^{-u/tau} (I - a/tau)
template <int KS = kAnyKind>
__device__ __forceinline__ void seg_eval_fast(const LifConst &C, const Seg &s, float u, float &f,
                                              float &fp, float &fpp) {
    if (kind_of<KS>(C) == kEqual) {
        const float e = __expf(-u * C.inv_ti);
        const float a = fmaf(s.I, u, s.V);
        const float d = fmaf(-a, C.inv_ti, s.I);
        f = a * e - C.theta;
        fp = e * d;
        fpp = -(e * C.inv_ti) * (s.I + d);
        return;
    }
    const float ev = __expf(-u * C.inv_tv);
    const float ei = __expf(-u * C.inv_ti);
    const float av = ev * C.inv_tv, ai = ei * C.inv_ti;
    f = fmaf(s.V, ev, s.I * C.c * (ev - ei)) - C.theta;
    fp = fmaf(-s.V, av, s.I * C.c * (ai - av));
    fpp = fmaf(s.V * C.inv_tv, av, s.I * C.c * fmaf(av, C.inv_tv, -ai * C.inv_ti));
}

// First root of v(u) = theta on [0, hi] given f(0) < 0 <= f(hi) = fhi (the
// only root there: v has at most one extremum per interval, and [0, hi]
// either ends at it or past the crossing). Halley iteration on the fast
// evaluation, started at the regula-falsi point and kept inside the bracket
// (bisection where a step leaves it), until |v - theta| <= 1e-6 theta or a
// step falls below 3e-5 of u; the cubic convergence puts that iterate within
// the fast evaluation's own error of the root. One Newton step on the exact evaluation then places the root
// to fp32 precision; the slope is the exact v' there, carried over the step
// with the fast v''.
template <int KS = kAnyKind>
__device__ __forceinline__ float seg_root(const LifConst &C, const Seg &s, float hi, float fhi,
                                          float &slope) {
    const float f0 = s.V - C.theta;  // f(0) < 0
    const float top = hi;
    float lo = 0.f;
    float u = (fhi > f0) ? hi * (-f0 / (fhi - f0)) : 0.5f * hi;
    if (!(u > 0.f && u < hi)) u = 0.5f * hi;
    float f, fp, fpp = 0.f;
    for (int it = 0; it < 40; ++it) {
        seg_eval_fast<KS>(C, s, u, f, fp, fpp);
        // at the fast evaluation's resolution: stepping further only follows
        // its rounding (an exact zero would also collapse the bracket onto u)
        if (fabsf(f) <= 1e-6f * C.theta) break;
        if (f < 0.f) lo = u; else hi = u;
        // Halley: u - 2 f f' / (2 f'^2 - f f'')
        const float den = fmaf(2.f * fp, fp, -f * fpp);
        float un = (fp > 0.f && den > 0.f) ? u - (2.f * f * fp) * __builtin_amdgcn_rcpf(den)
                                           : 0.5f * (lo + hi);
        if (!(un > lo && un < hi)) un = 0.5f * (lo + hi);
        const float step = un - u;
        u = un;
        const float tol = 3e-5f * fmaxf(u, 1e-6f * C.dt);
        if (fabsf(step) <= tol || hi - lo <= 0.25f * tol) break;
    }
    float fe, fpe;
    seg_eval<KS>(C, s, u, fe, fpe);
    float un = (fpe > 0.f) ? u - fe / fpe : u;
    un = fminf(fmaxf(un, 0.f), top);
    slope = fmaf(un - u, fpp, fpe);
    return un;
}

// Scan gradient of one neuron, G[m] = dL/dw^_m = gamma K(t - T_m) for
// 0 <= m <= q (implicit-function theorem on v^(t) = theta), from the
// per-neuron triple gamma = -g / slope (slope floored at 1e-12 theta),
// u = t - T_q (difference taken in fp64) and q; q = -1 where no gradient
// flows (silent neuron or g = 0).
// Synfire-chain training terms inside a backward call (App. C.1): the
// temporal penalty's dT/dt joins the gradient of every firing neuron; dq
// (workspace, one float per weight row) receives -gamma_q * scale * (number
// of silent neurons the row feeds) and is added where dW is written.
struct Synfire {
    int on;
    float gh, gt, th, tt, gq, scale;
    float *dq;
};

// d T / d t of a firing neuron: 2 scale (gamma_head (t - t_head) below the
// window, gamma_tail (t - t_tail) above it), 0 inside
__device__ __forceinline__ float synfire_dt(const Synfire &s, float t) {
    float d = 0.f;
    if (t < s.th) d = 2.f * s.gh * (t - s.th);
    else if (t > s.tt) d = 2.f * s.gt * (t - s.tt);
    return s.scale * d;
}

struct GradPrep { float gam, uq; int q; };

__device__ __forceinline__ GradPrep grad_prep(const LifConst &C, float t, float slope, int q,
                                              float g) {
    GradPrep r{0.f, 0.f, -1};
    if (q < 0 || g == 0.f) return r;
    const double T_q = fma(static_cast<double>(q), static_cast<double>(C.dt), static_cast<double>(C.t0));
    r.gam = -g / fmaxf(slope, C.slope_floor);
    r.uq = static_cast<float>(fmax(static_cast<double>(t) - T_q, 0.0));
    r.q = q;
    return r;
}

// G[m] from the triple: t - T_m = (t - T_q) + (q - m) dt is formed with one
// rounding from non-negative terms, and K(u) keeps full relative precision
// (expm1 form), so no per-neuron recurrence over the grid is needed.
template <int KS = kAnyKind>
__device__ __forceinline__ float g_at(const LifConst &C, float gam, float uq, int q, int m) {
    if (m < 0 || m > q) return 0.f;
    return gam * kern<KS>(C, fmaf(static_cast<float>(q - m), C.dt, uq));
}

// G of one neuron at the grid points m_c = m0 + c * step, c = 0..N-1 (rows of
// a strided staging pattern; entries outside 0 <= m_c <= q are 0). The
// largest m_c <= q is evaluated directly; the smaller ones follow from the
// recurrence K(u + s) = a_s K(u) + K(s) e^{-u/ti}, e^{-(u+s)/ti} =
// b_s e^{-u/ti} (s = step * dt), whose terms are all positive.
struct GStep { float a, b, k; };  // e^{-s/tv}, e^{-s/ti}, K(s)

template <int KS = kAnyKind>
__device__ __forceinline__ GStep g_step(const LifConst &C, int step) {
    const float s = static_cast<float>(step) * C.dt;
    return GStep{expf(-s * C.inv_tv), expf(-s * C.inv_ti), kern<KS>(C, s)};
}

template <int N, int KS = kAnyKind>
__device__ __forceinline__ void g_strided(const LifConst &C, const GStep &gs, float gam, float uq,
                                          int q, int m0, int step, float *out) {
    // highest c with m_c <= q (-1: none)
    const int c_top = (q < m0) ? -1 : min(N - 1, (q - m0) / step);
    const float u_top = fmaf(static_cast<float>(q - (m0 + max(c_top, 0) * step)), C.dt, uq);
    float K, E;  // K(u_top), e^{-u_top/ti}
    if (kind_of<KS>(C) == kGeneral) {
        const float ev = expf(-u_top * C.inv_tv);
        const float em = expm1f(-C.kappa * u_top);
        K = -C.c * ev * em;
        E = ev * (1.f + em);
    } else {
        K = kern<KS>(C, u_top);
        E = expf(-u_top * C.inv_ti);
    }
#pragma unroll
    for (int c = N - 1; c >= 0; --c) {
        if (c < c_top) {
            K = fmaf(gs.a, K, gs.k * E);
            E *= gs.b;
        }
        out[c] = (c <= c_top && m0 + c * step >= 0) ? gam * K : 0.f;
    }
}

// Crossing test of one interval [0, len) of the state form v(u) = V e^{-u/tv}
// + I K(u) (V = v at the interval's start, I the current just after its
// input), for a neuron that has not fired before it. vn_d is v at the
// interval's end carried by the fp64 recurrence (used unless `last`); the
// last interval's end value is evaluated at len, or taken as the limit of an
// open interval (len = +inf). kmax = max K on [0, len] (fp64), r_lo =
// e^{-kappa len} (general row). On a crossing returns true with the fp32
// segment, the bracket end hi (0: fires at u = 0, only through rounding) and
// v - theta there.
// The bound filter of a segment of any length (the last interval, the
// free-decay tail, the exact and multi-spike walks): v(u) <= max(V,0) +
// max(I,0) kmax, tested on the fp64 state against theta with a 1e-4 margin
// (only segments that pass are analysed; kmax is +inf on an open interval
// of the (inf, inf) row, where I = 0 must not give inf * 0).
__device__ __forceinline__ bool seg_may_cross(const LifConst &C, double Vd, double Id,
                                              double kmax) {
    const double vpos = fmax(Vd, 0.0);
    const double ub = (Id > 0.0) ? fma(Id, kmax, vpos) : vpos;
    return ub >= C.theta_lo_d;
}

// The filter of an interval of length dt (before T_M) from its two ends: on
// [0, dt] the linear interpolation of v(0) = V and v(dt) = vn lies below
// max(V, vn), and v exceeds it by at most dt^2/8 max(-v''), where
// |v''| <= |V| / tv^2 + |I| max |K''|. Every interval whose maximum reaches
// theta_lo passes; the ones hovering below theta do not.
__device__ __forceinline__ bool seg_may_cross_dt(const LifConst &C, double Vd, double Id,
                                                 double vn_d) {
    const double ub = fma(fabs(Id), C.curv_i_d, fma(fabs(Vd), C.curv_v_d, fmax(Vd, vn_d)));
    return ub >= C.theta_lo_d;
}

// The analysis of an interval that passed the filter.
template <int KS = kAnyKind>
__device__ __forceinline__ bool seg_cross(const LifConst &C, double Vd, double Id, double vn_d,
                                          bool last, float len, float r_lo, Seg &sf, float &hi,
                                          float &fhi) {
    const int kind = kind_of<KS>(C);
    const Seg s{static_cast<float>(Vd), static_cast<float>(Id)};
    const bool fin = !last || isfinite(len);
    float vend = -INFINITY;
    if (!last) {
        vend = static_cast<float>(vn_d);
    } else if (fin) {
        float f, fp;
        seg_eval<KS>(C, s, len, f, fp);
        vend = f + C.theta;
    } else if (kind == kInfTau) {
        // open interval: v rises to V + I tau (never reached)
        const float lim = fmaf(s.I, C.ti, s.V);
        if (s.I > 0.f && lim > C.theta) vend = lim;
    } else if (kind == kInfInf) {
        if (s.I > 0.f) vend = INFINITY;  // v = V + I u grows without bound
    }
    if (s.V >= C.theta) {  // only through rounding: v is continuous
        sf = s; hi = 0.f;
        return true;
    }
    if (vend >= C.theta) {
        sf = s; hi = len; fhi = vend - C.theta;
        return true;
    }
    if (kind == kEqual) {
        // interior maximum of (V + I u) e^{-u/tau} at u* = tau - V/I (I > 0),
        // where v = I tau e^{-u*/tau} <= I tau
        if (s.I > 0.f && s.I * C.ti * 1.0001f >= C.theta) {
            const float us = C.ti - s.V / s.I;
            if (us > 0.f && us < len) {
                const float vs = s.I * C.ti * expf(-us * C.inv_ti);
                if (vs >= C.theta) { sf = s; hi = us; fhi = vs - C.theta; return true; }
            }
        }
    } else if (kind == kGeneral && s.I > 0.f) {
        // interior maximum: v'(u*) = 0 with e^{-kappa u*} = (ti/tv)(1 + V/(c I))
        const float r = (C.ti * C.inv_tv) * (1.f + s.V / (C.c * s.I));
        // v(u*) = e^{-u*/tv} (V + c I (1 - r)) <= V + c I (1 - r): the
        // maximum is evaluated only if this bound reaches theta
        if (r > r_lo && r < 1.f && fmaf(s.I * C.c, 1.f - r, s.V) * 1.0001f >= C.theta) {
            const float us = -logf(r) / C.kappa;
            float f, fp;
            seg_eval<KS>(C, s, us, f, fp);
            if (f >= 0.f) { sf = s; hi = us; fhi = f; return true; }
        }
    }
    return false;
}

template <int KS = kAnyKind>
__device__ __forceinline__ bool seg_test(const LifConst &C, double Vd, double Id, double vn_d,
                                         bool last, float len, double kmax, float r_lo, Seg &sf,
                                         float &hi, float &fhi) {
    return seg_may_cross(C, Vd, Id, kmax) &&
           seg_cross<KS>(C, Vd, Id, vn_d, last, len, r_lo, sf, hi, fhi);
}

// Spike time inside the crossing interval found by seg_test: u with v(u) =
// theta on [0, hi] and the slope v'(u). The closed-form rows of Table
// "tab:timing_DSTD" are solved directly; the general row by seg_root.
template <int KS = kAnyKind>
__device__ __forceinline__ void seg_solve(const LifConst &C, const Seg &sf, float hi, float fhi,
                                          float &u, float &sl) {
    const int kind = kind_of<KS>(C);
    if (hi > 0.f && kind == kInfInf) {
        // Table "tab:timing_DSTD", row (inf, inf): V + I u = theta, I > 0
        u = fminf((C.theta - sf.V) / sf.I, hi);
        sl = sf.I;
    } else if (hi > 0.f && kind == kInfTau) {
        // row (inf, tau): V + I tau (1 - e^{-u/tau}) = theta, I > 0
        u = fminf(-C.ti * log1pf(-(C.theta - sf.V) / (sf.I * C.ti)), hi);
        sl = sf.I * expf(-u * C.inv_ti);
    } else if (hi > 0.f && kind == kGeneral && C.twice) {
        // Table "tab:timing_DSTD", row (2tau, tau): with x = e^{-u/(2tau)}
        // the segment is v = A x - B x^2 (A = V + cI, B = cI, c = 2tau), so
        // v = theta is a quadratic in x; the crossing is the root below 1
        // nearest to it (the larger root for B > 0), in its stable form
        const float Bq = C.c * sf.I, Aq = sf.V + Bq;
        const float sq = sqrtf(fmaxf(fmaf(Aq, Aq, -4.f * Bq * C.theta), 0.f));
        const float x = (Bq > 0.f) ? (Aq + sq) / (2.f * Bq) : 2.f * C.theta / (Aq + sq);
        u = fminf(fmaxf(-C.tv * logf(x), 0.f), hi);
        const float xu = expf(-u * C.inv_tv);
        sl = fmaf(-Aq * xu, C.inv_tv, Bq * xu * xu * C.inv_ti);
    } else if (hi > 0.f) {
        u = seg_root<KS>(C, sf, hi, fhi, sl);
    } else {
        float f;
        u = 0.f;
        seg_eval<KS>(C, sf, 0.f, f, sl);
    }
}

// Interval scan of one neuron (Table "tab:timing_DSTD", Eq. (timing_DSTD)):
// weighted events arrive in grid order through step(); the earliest interval
// whose candidate lies inside it is kept. The state (v at T_q, current after
// the event at T_q) is propagated in fp64: over M intervals fp32 rounding of
// the recurrence would grow with M. Interval tests use the fp32-rounded state.
// Only the crossing interval and its bracket are located here; the root is
// solved once in finish(), with all lanes of the wave together.
template <int KS = kAnyKind>
struct Scan {
    double Vd = 0.0, Id = 0.0;
    int qf = -1;
    Seg sf{0.f, 0.f};
    float hi = 0.f, fhi = 0.f;  // bracket end of the crossing and v - theta there
    bool tl = false;            // the bracket is on the free-decay tail from T_qf

    // grid point q: w^_q enters the current, and the interval after T_q
    // (kLast: the last one, [T_M, t_max)) is tested. The filter runs on every
    // lane; one branch covers the lanes still searching that pass it.
    template <bool kLast>
    __device__ __forceinline__ void step_k(const LifConst &C, int q, float w) {
        Id += static_cast<double>(w);
        const double vn_d = fma(Vd, C.alpha_d, Id * C.k_dt_d);
        // one branch: the filter is evaluated on every lane (no short circuit)
        const bool go = (qf < 0) & (kLast ? seg_may_cross(C, Vd, Id, C.kmax_last_d)
                                          : seg_may_cross_dt(C, Vd, Id, vn_d));
        if (go) {
            if (seg_cross<KS>(C, Vd, Id, vn_d, kLast, kLast ? C.last_len : C.dt,
                              kLast ? C.r_lo_last : C.r_lo_dt, sf, hi, fhi))
                qf = q;
        }
        Vd = vn_d;
        Id *= C.beta_d;
    }

    __device__ __forceinline__ void step(const LifConst &C, int q, float w) {
        if (q == C.M) step_k<true>(C, q, w);
        else step_k<false>(C, q, w);
    }

    __device__ __forceinline__ bool found() const { return qf >= 0; }

    // No input arrives at grid points q0 .. M (the state is v at T_q0 and the
    // current before the empty event there): from T_q0 to t_max v is one free
    // decay, v(T_q0 + u) = V e^{-u/tv} + I K(u), the same function the
    // remaining intervals would be tested on one by one. Its first crossing,
    // if any, is bracketed once by the interval analysis applied to the whole
    // segment; finish() then solves it there and names the interval that
    // holds it. Lanes that have found their interval are unchanged.
    __device__ __forceinline__ void tail(const LifConst &C, int q0) {
        if (qf >= 0 || !seg_may_cross(C, Vd, Id, C.kpeak_d)) return;
        const float len = fmaf(static_cast<float>(C.M - q0), C.dt, C.last_len);  // +inf stays
        const float r_lo = (kind_of<KS>(C) == kGeneral && len < INFINITY) ? expf(-C.kappa * len) : 0.f;
        if (seg_cross<KS>(C, Vd, Id, 0.0, true, len, r_lo, sf, hi, fhi)) {
            qf = q0;
            tl = true;
        }
    }

    __device__ __forceinline__ void finish(const LifConst &C, float &t_out, float &slope,
                                           int &q_out) const {
        t_out = INFINITY;
        slope = 0.f;
        q_out = qf;
        if (qf < 0) return;
        float u, sl;
        seg_solve<KS>(C, sf, hi, fhi, u, sl);
        t_out = static_cast<float>(fma(static_cast<double>(qf), static_cast<double>(C.dt),
                                       static_cast<double>(C.t0)) + static_cast<double>(u));
        slope = sl;
        if (tl) q_out = qf + min(static_cast<int>(u * C.inv_dt), C.M - qf);
    }
};

// W [rows][cols] -> WT [cols][rows], one 32 x 32 tile through a padded LDS
// tile (kThreads threads, a multiple of 32).
template <typename WT, int kThreads>
__device__ void transpose_tile(int rows, int cols, const WT *__restrict__ in, WT *__restrict__ out,
                               int tile, WT (*buf)[33]) {
    const int ntx = (cols + 31) / 32;
    const int c0 = (tile % ntx) * 32, r0 = (tile / ntx) * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int k = ty; k < 32; k += kThreads / 32) {
        const int r = r0 + k, c = c0 + tx;
        if (r < rows && c < cols) buf[k][tx] = in[static_cast<int64_t>(r) * cols + c];
    }
    __syncthreads();
    for (int k = ty; k < 32; k += kThreads / 32) {
        const int c = c0 + k, r = r0 + tx;
        if (r < rows && c < cols) out[static_cast<int64_t>(c) * rows + r] = buf[tx][k];
    }
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// The chip hands workgroup b to XCD b % 8 (eight XCDs, each with its own L2).
// xcd_block maps the hardware block index to a logical one such that each
// XCD takes one contiguous range of logical blocks: neighbouring output
// positions then share an L2, and the partial cache lines their lanes write
// (one channel each, NCHW) merge there instead of in HBM.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_block(int bid, int nb) {
    const int x = bid % kXcds, i = bid / kXcds;
    const int per = nb / kXcds, rem = nb % kXcds;
    return x * per + min(x, rem) + i;
}

// Eight per-lane values, each summed over the 64 lanes of the wave; the
// totals come back scattered: every lane of the group 8k .. 8k+7 holds the
// total of v[k]. Each halving step exchanges half of the values still held:
// lanes l and l+32 (permlane32 swap: v[k] stays in the low half, v[k+4] in
// the high half), then the 16-lane rows (permlane16 swap), then lanes l and
// l^8 (DPP rotate by 8 within a row); the 8-lane groups finish with DPP quad
// permutes and the half-row mirror. 18 VALU where eight butterflies take 96.
// The summation order is fixed, so the totals are deterministic. Needs all
// 64 lanes active.
template <int kCtrl>
__device__ __forceinline__ float dpp_c(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum8(const float (&v)[8], int lane) {
    float s[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[k]), __float_as_uint(v[k + 4]),
                                                        false, false);
        s[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    // lanes 0-31: v[0..3] over lane pairs (l, l+32); lanes 32-63: v[4..7]
    float t[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(s[k]), __float_as_uint(s[k + 2]),
                                                        false, false);
        t[k] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    // rows 0..3 of 16 lanes: t[0] holds v[0], v[2], v[4], v[6]; t[1] holds
    // v[1], v[3], v[5], v[7]
    const bool hi = (lane & 8) != 0;
    const float keep = hi ? t[1] : t[0], send = hi ? t[0] : t[1];
    float u = keep + dpp_c<0x128>(send);  // row_ror:8
    u += dpp_c<0xB1>(u);                  // quad_perm [1,0,3,2]
    u += dpp_c<0x4E>(u);                  // quad_perm [2,3,0,1]
    u += dpp_c<0x141>(u);                 // row_half_mirror
    return u;
}

// Raw buffer access: a per-lane byte offset plus a wave-uniform (scalar)
// byte offset. Every caller keeps both offsets inside `bytes` (indices are
// clamped); the descriptor's range check is only a backstop.
constexpr int kBufWord3 = 0x00020000;  // gfx9 raw-buffer descriptor, word 3
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), static_cast<short>(0),
                                             static_cast<int>(bytes), kBufWord3);
}
template <typename WT> struct BufLoad;
template <> struct BufLoad<float> {
    static __device__ __forceinline__ float get(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
        // the builtin returns the 32 bits as an integer: reinterpret, not convert
        return __int_as_float(static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0)));
    }
};
template <> struct BufLoad<uint16_t> {
    static __device__ __forceinline__ float get(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
        return bf16_to_f32(static_cast<uint16_t>(__builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0)));
    }
};

// N consecutive weights (N = 1, 2 or 4) with one buffer load: fp32 as 4N
// bytes, bf16 as 2N bytes, widened to fp32.
template <typename WT, int N> struct BufLoadN;
template <int N> struct BufLoadN<float, N> {
    static __device__ __forceinline__ void get(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                               float (&out)[N]) {
        if constexpr (N == 4) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
#pragma unroll
            for (int c = 0; c < 4; ++c) out[c] = __int_as_float(static_cast<int>(v[c]));
        } else if constexpr (N == 2) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
            out[0] = __int_as_float(static_cast<int>(v[0]));
            out[1] = __int_as_float(static_cast<int>(v[1]));
        } else {
            out[0] = BufLoad<float>::get(r, voff, soff);
        }
    }
};
template <int N> struct BufLoadN<uint16_t, N> {
    static __device__ __forceinline__ void get(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                               float (&out)[N]) {
        if constexpr (N == 4) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const uint32_t u = static_cast<uint32_t>(v[c]);
                out[2 * c] = __uint_as_float(u << 16);
                out[2 * c + 1] = __uint_as_float(u & 0xffff0000u);
            }
        } else if constexpr (N == 2) {
            const uint32_t u = static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
            out[0] = __uint_as_float(u << 16);
            out[1] = __uint_as_float(u & 0xffff0000u);
        } else {
            out[0] = BufLoad<uint16_t>::get(r, voff, soff);
        }
    }
};

// Reads through the constant address space: with a wave-uniform address the
// compiler emits scalar (SMEM) loads, batched into s_load_dwordx16 when
// consecutive. Only for data that no kernel in flight writes.
typedef __attribute__((address_space(4))) const int cint_t;
typedef __attribute__((address_space(4))) const float cflt_t;
typedef __attribute__((address_space(4))) const double cdbl_t;
__device__ __forceinline__ cint_t *as_const(const int *p) { return (cint_t *)p; }
__device__ __forceinline__ cflt_t *as_const(const float *p) { return (cflt_t *)p; }
__device__ __forceinline__ cdbl_t *as_const(const double *p) { return (cdbl_t *)p; }

}  // namespace dstd
