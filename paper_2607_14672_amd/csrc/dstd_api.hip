// dstd_api.hip -- C ABI of the DSTD-LIF library: argument validation (host
// only, before anything is enqueued), layer constants, workspace layout and
// kernel dispatch. The contract of every entry point is documented in
// include/dstd_lif.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "../../include/dstd_lif.h"
#include "dstd_internal.h"
#include "dstd_kernels.h"

using dstd::LifConst;

namespace {

thread_local char g_err[512] = "";

dstd_status fail(dstd_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

// Host validation of the layer parameters (no device access).
dstd_status check_params(const dstd_lif_params *p, int32_t allowed_flags = 0) {
    if (!p) return fail(DSTD_ERR_NULL, "params is NULL");
    // each time constant is > 0, finite or +inf (the closed-form rows)
    if (!(p->tau_m > 0.f) || !(p->tau_s > 0.f))
        return fail(DSTD_ERR_PARAM, "time constants must be > 0 or +inf (tau_m=%g tau_s=%g)",
                    (double)p->tau_m, (double)p->tau_s);
    if (isfinite(p->tau_m) && isfinite(p->tau_s) && p->tau_m != p->tau_s) {
        double tmax = std::max((double)p->tau_m, (double)p->tau_s);
        if (fabs((double)p->tau_m - (double)p->tau_s) <= 1e-3 * tmax)
            return fail(DSTD_ERR_UNSUPPORTED,
                        "tau_m and tau_s differ by less than 1e-3 relative without being equal: "
                        "use equal constants (the (tau, tau) row) or separate them further");
    }
    if (!(isfinite(p->threshold) && p->threshold > 0.f))
        return fail(DSTD_ERR_PARAM, "threshold must be finite and > 0");
    if (p->M < 1) return fail(DSTD_ERR_PARAM, "M must be >= 1 (got %d)", p->M);
    if (p->M > DSTD_MAX_M)
        return fail(DSTD_ERR_UNSUPPORTED, "M = %d exceeds DSTD_MAX_M = %d", p->M, DSTD_MAX_M);
    if (!(isfinite(p->dt) && p->dt > 0.f)) return fail(DSTD_ERR_PARAM, "dt must be finite and > 0");
    if (!isfinite(p->t0)) return fail(DSTD_ERR_PARAM, "t0 must be finite");
    double TM = (double)p->t0 + (double)p->M * (double)p->dt;
    if (isnan(p->t_max) || !((double)p->t_max > TM))
        return fail(DSTD_ERR_PARAM, "t_max must be > T_M = t0 + M*dt (got %g, T_M = %g)",
                    (double)p->t_max, TM);
    if ((p->flags & ~allowed_flags) != 0) {
        const int32_t extra = p->flags & ~allowed_flags;
        if (extra & (DSTD_FLAG_CONTRACT_SPARSE | DSTD_FLAG_CONTRACT_MFMA))
            return fail(DSTD_ERR_UNSUPPORTED, "the contraction flags apply to dense layers only");
        if (extra & DSTD_FLAG_CONV_KEEP)
            return fail(DSTD_ERR_UNSUPPORTED, "DSTD_FLAG_CONV_KEEP applies to the conv forward only");
        if (extra & DSTD_FLAG_CONV_REUSE)
            return fail(DSTD_ERR_UNSUPPORTED, "DSTD_FLAG_CONV_REUSE applies to the conv backward only");
        return fail(DSTD_ERR_PARAM, "unknown flags 0x%x", (unsigned)p->flags);
    }
    if ((p->flags & DSTD_FLAG_CONTRACT_SPARSE) && (p->flags & DSTD_FLAG_CONTRACT_MFMA))
        return fail(DSTD_ERR_PARAM, "DSTD_FLAG_CONTRACT_SPARSE and _MFMA exclude each other");
    return DSTD_OK;
}

constexpr int32_t kDenseFlags = DSTD_FLAG_CONTRACT_SPARSE | DSTD_FLAG_CONTRACT_MFMA;

// The dense forward's contraction: the event-sparse VALU kernels, or the
// dense bf16 MFMA product of the event matrix and W (bf16 weights only). The
// automatic choice is by shape, from measured times on MI355X (the dense
// product does (M+1)/2 times the method's work, so it wins only for small M
// on large layers).
bool mfma_shape_auto(int M, int64_t B, int64_t N_in, int64_t N_out) {
    return M <= dstd::kMfmaAutoMaxM && N_out >= 1024 && N_in >= 1024 && B * N_out >= (int64_t)1 << 18;
}

// could this call take the MFMA path (the workspace query does not know the
// weight type, so it reserves room whenever it could)
bool mfma_possible(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out) {
    if (p->flags & DSTD_FLAG_CONTRACT_SPARSE) return false;
    if (p->flags & DSTD_FLAG_CONTRACT_MFMA) return true;
    return mfma_shape_auto(p->M, B, N_in, N_out);
}

size_t mfma_ws_events(int64_t B, int64_t N_in) { return align_up((size_t)(B * N_in) * 16); }
size_t mfma_ws_bytes(int M, int64_t B, int64_t N_in, int64_t N_out) {
    if (B * N_out == 0) return 0;
    return mfma_ws_events(B, N_in) + align_up((size_t)B * (size_t)(M + 1) * (size_t)N_out * sizeof(float));
}

// Row of Table "tab:kernel" for the canonical pair tv >= ti (tv may be inf).
int kind_of(double tv, double ti) {
    if (isinf(ti)) return dstd::kInfInf;
    if (isinf(tv)) return dstd::kInfTau;
    if (tv == ti) return dstd::kEqual;
    return dstd::kGeneral;
}

// K(u), u >= 0 (u may be +inf for the (inf, tau) row's limit)
double kern_d(int kind, double tv, double ti, double u) {
    switch (kind) {
        case dstd::kEqual: return u * exp(-u / ti);
        case dstd::kInfTau: return -ti * expm1(-u / ti);
        case dstd::kInfInf: return u;
        default: {
            double c = tv * ti / (tv - ti), kap = 1.0 / ti - 1.0 / tv;
            return -c * exp(-u / tv) * expm1(-kap * u);
        }
    }
}

LifConst make_const(const dstd_lif_params *p) {
    double tv = std::max((double)p->tau_m, (double)p->tau_s);
    double ti = std::min((double)p->tau_m, (double)p->tau_s);
    const int kind = kind_of(tv, ti);
    double dt = p->dt;
    // K's maximum on [0, len] sits at min(len, peak): the general row peaks
    // at ln(tv/ti)/kappa, (tau, tau) at tau; the other rows increase
    double kap = (kind == dstd::kGeneral) ? 1.0 / ti - 1.0 / tv : 0.0;
    double upk = (kind == dstd::kGeneral) ? log(tv / ti) / kap
                 : (kind == dstd::kEqual) ? ti : INFINITY;
    double TM = (double)p->t0 + (double)p->M * dt;
    double last = isinf(p->t_max) ? INFINITY : (double)p->t_max - TM;
    LifConst C{};
    C.kind = kind;
    C.tv = (float)tv;
    C.ti = (float)ti;
    C.inv_tv = (float)(1.0 / tv);  // 0 for an infinite constant
    C.inv_ti = (float)(1.0 / ti);
    C.c = (kind == dstd::kGeneral) ? (float)(tv * ti / (tv - ti)) : 0.f;
    C.kappa = (float)kap;
    C.alpha = (float)exp(-dt / tv);
    C.beta = (float)exp(-dt / ti);
    C.k_dt = (float)kern_d(kind, tv, ti, dt);
    C.inv_em1 = (kind == dstd::kGeneral) ? (float)(1.0 / expm1(-kap * dt)) : 0.f;
    C.kmax_dt_d = kern_d(kind, tv, ti, std::min(dt, upk));
    C.kmax_last_d = kern_d(kind, tv, ti, std::min(last, upk));
    C.theta_lo_d = (double)p->threshold / 1.0001;
    C.kpeak_d = kern_d(kind, tv, ti, std::min((double)p->M * dt + last, upk));
    // max |K''| on [0, dt]: general row c |e^{-u/tv}/tv^2 - e^{-u/ti}/ti^2|
    // <= c / ti^2; (tau, tau) e^{-u/tau} |u/tau^2 - 2/tau| <= 2/tau + dt/tau^2;
    // (inf, tau) e^{-u/tau}/tau <= 1/tau; (inf, inf) 0
    const double kpp = (kind == dstd::kGeneral) ? tv / (ti * (tv - ti))
                       : (kind == dstd::kEqual) ? 2.0 / ti + dt / (ti * ti)
                       : (kind == dstd::kInfTau) ? 1.0 / ti : 0.0;
    C.curv_v_d = dt * dt / 8.0 * (isinf(tv) ? 0.0 : 1.0 / (tv * tv));
    C.curv_i_d = dt * dt / 8.0 * kpp;
    C.twice = (kind == dstd::kGeneral && tv == 2.0 * ti) ? 1 : 0;
    C.inv_dt = (float)(1.0 / dt);
    C.e_mdt = (float)exp(-dt / ti);
    C.inv_D = (kind == dstd::kInfTau) ? (float)(-1.0 / expm1(-dt / ti)) : 0.f;
    C.theta = p->threshold;
    C.t0 = p->t0;
    C.dt = p->dt;
    C.last_len = (float)last;
    C.slope_floor = 1e-12f * p->threshold;
    C.M = p->M;
    C.alpha_d = exp(-dt / tv);
    C.beta_d = exp(-dt / ti);
    C.k_dt_d = kern_d(kind, tv, ti, dt);
    C.r_lo_dt = (float)exp(-kap * dt);
    C.r_lo_last = isinf(last) ? 0.f : (float)exp(-kap * last);
    return C;
}

dstd_status check_dims(int64_t B, int64_t N_in, int64_t N_out) {
    if (B < 0 || N_in < 0 || N_out < 0)
        return fail(DSTD_ERR_SHAPE, "sizes must be >= 0 (B=%lld N_in=%lld N_out=%lld)",
                    (long long)B, (long long)N_in, (long long)N_out);
    const int64_t lim = (int64_t)1 << 24;
    if (N_in >= lim || N_out >= lim)
        return fail(DSTD_ERR_SHAPE, "N_in and N_out must be < 2^24");
    if (B > 65535)
        return fail(DSTD_ERR_SHAPE, "B = %lld exceeds the supported batch (65535)", (long long)B);
    if (N_in * N_out * 4 >= ((int64_t)1 << 31))
        return fail(DSTD_ERR_SHAPE, "N_in * N_out = %lld exceeds 2^29 weights",
                    (long long)(N_in * N_out));
    return DSTD_OK;
}

struct DenseWs {
    size_t row, L, R, gam, uq, q, part, dq, wt, sj, sr, sL, sR, nvalid, rs, total;
    int64_t sstride;
};

DenseWs dense_ws_layout(int M, int64_t B, int64_t N_in, int64_t N_out, bool backward) {
    DenseWs w{};
    size_t off = 0;
    size_t n = (size_t)(B * N_in);
    if (!backward && B * N_out == 0) return w;  // the forward enqueues nothing
    // transposed weights (room for fp32) and the row-sorted event records of
    // every sample: both passes walk them (the backward for dt_in)
    w.wt = off; off += align_up((size_t)N_in * (size_t)N_out * sizeof(float));
    // sorted event lists: per sample N_in records; the last sample's list
    // is padded so batched reads past its end stay in the allocation
    w.sstride = N_in;
    size_t ns = n + dstd::kSortPad;
    w.sj = off; off += align_up(ns * sizeof(int));
    w.sr = off; off += align_up(ns * sizeof(int));
    w.sL = off; off += align_up(ns * sizeof(float));
    w.sR = off; off += align_up(ns * sizeof(float));
    w.nvalid = off; off += align_up((size_t)B * sizeof(int));
    w.rs = off; off += align_up((size_t)B * (M + 4) * sizeof(int));
    if (backward) {
        // per-input events for the dW reduction, gradient triples, dW partials
        w.row = off; off += align_up(n * sizeof(int));
        w.L = off; off += align_up(n * sizeof(float));
        w.R = off; off += align_up(n * sizeof(float));
        w.gam = off; off += align_up((size_t)B * (size_t)N_out * sizeof(float));
        w.uq = off; off += align_up((size_t)B * (size_t)N_out * sizeof(float));
        w.q = off; off += align_up((size_t)B * (size_t)N_out * sizeof(int));
        w.dq = off; off += align_up((size_t)N_out * sizeof(float));  // dead-neuron term per row
        dstd::DwPlan dp = dstd::plan_dw(B, N_in, N_out, M);
        w.part = off;
        if (dp.nsplit > 1) off += align_up((size_t)dp.nsplit * (size_t)N_out * (size_t)N_in * sizeof(float));
    }
    w.total = off;
    return w;
}

dstd_status check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (need == 0) return DSTD_OK;
    if (!ws) return fail(DSTD_ERR_NULL, "workspace is NULL (%zu bytes needed)", need);
    if (((uintptr_t)ws) % kAlign != 0) return fail(DSTD_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (ws_bytes < need)
        return fail(DSTD_ERR_WORKSPACE, "workspace too small: %zu < %zu bytes", ws_bytes, need);
    return DSTD_OK;
}

dstd_status hip_status(hipError_t e, const char *what) {
    if (e == hipSuccess) return DSTD_OK;
    return fail(DSTD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

template <typename T> T *at(void *ws, size_t off) {
    return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}


// Host validation of a conv layer; fills the derived geometry.
dstd_status check_conv(const dstd_conv_shape *cs, int64_t B, int M, dstd::ConvGeom *g) {
    if (!cs) return fail(DSTD_ERR_NULL, "conv shape is NULL");
    if (B < 0) return fail(DSTD_ERR_SHAPE, "B must be >= 0");
    if (cs->C_in < 1 || cs->H < 1 || cs->W < 1 || cs->C_out < 1)
        return fail(DSTD_ERR_SHAPE, "C_in, H, W and C_out must be >= 1");
    if (cs->C_in > (1 << 20) || cs->C_out > (1 << 20))
        return fail(DSTD_ERR_SHAPE, "C_in and C_out must be <= 2^20");
    if (cs->KH < 1 || cs->KW < 1 || cs->KH > dstd::kConvMaxK || cs->KW > dstd::kConvMaxK)
        return fail(DSTD_ERR_UNSUPPORTED, "kernel size %dx%d: 1..%d supported", cs->KH, cs->KW,
                    dstd::kConvMaxK);
    if (cs->stride < 1 || cs->pad < 0 || cs->pad >= std::max(cs->KH, cs->KW) + 1)
        return fail(DSTD_ERR_SHAPE, "need stride >= 1 and 0 <= pad <= max(KH, KW)");
    if (cs->pool_in != 0 && cs->pool_in != 1 && cs->pool_in != 2)
        return fail(DSTD_ERR_PARAM, "pool_in must be 0, 1 or 2 (got %d)", cs->pool_in);
    if (cs->pool_in == 2 && (cs->H % 2 != 0 || cs->W % 2 != 0))
        return fail(DSTD_ERR_SHAPE, "2x2 event pooling needs even H and W (got %dx%d)", cs->H, cs->W);
    dstd::ConvGeom &G = *g;
    G.C_in = cs->C_in; G.H = cs->H; G.W = cs->W; G.C_out = cs->C_out;
    G.KH = cs->KH; G.KW = cs->KW; G.stride = cs->stride; G.pad = cs->pad; G.pool = cs->pool_in;
    if (G.pool == 2) { G.Hp = G.H / 2; G.Wp = G.W / 2; G.P = 4; }
    else if (G.pool == 0) { G.Hp = 1; G.Wp = 1; G.P = G.H * G.W; }
    else { G.Hp = G.H; G.Wp = G.W; G.P = 1; }
    const int64_t ho = ((int64_t)G.Hp + 2 * G.pad - G.KH) / G.stride + 1;
    const int64_t wo = ((int64_t)G.Wp + 2 * G.pad - G.KW) / G.stride + 1;
    if ((int64_t)G.Hp + 2 * G.pad < G.KH || (int64_t)G.Wp + 2 * G.pad < G.KW || ho < 1 || wo < 1)
        return fail(DSTD_ERR_SHAPE, "kernel larger than the padded input map");
    G.Ho = (int)ho; G.Wo = (int)wo;
    const int64_t pc = (int64_t)G.P * G.C_in;
    const int64_t lim = (int64_t)1 << 30;
    const int64_t nw = (int64_t)G.KH * G.KW * G.C_in * G.C_out;
    if (pc * G.Wp >= lim || (int64_t)G.C_in * G.H * G.W >= lim || nw * 4 >= lim ||
        (int64_t)G.C_out * G.Ho * G.Wo >= lim)
        return fail(DSTD_ERR_SHAPE, "conv layer too large (per-sample sizes must stay below 2^30)");
    if (B * G.Hp >= ((int64_t)1 << 31) || B * G.Ho * G.Wo >= ((int64_t)1 << 31))
        return fail(DSTD_ERR_SHAPE, "batch too large for this map size");
    if ((int64_t)(M + 3) * G.Wp + 256 > 16384)
        return fail(DSTD_ERR_UNSUPPORTED, "(M + 3) * W_p = %lld exceeds the cell-row sort's LDS "
                    "table (16128 buckets)", (long long)(M + 3) * G.Wp);
    G.PC = (int)pc;
    G.inv_P = (float)(1.0 / G.P);
    G.dv_pch = dstd::fast_div((uint32_t)(G.Wp * G.P));
    G.dv_w = dstd::fast_div((uint32_t)G.W);
    G.dv_cin = dstd::fast_div((uint32_t)G.C_in);
    G.dv_p = dstd::fast_div((uint32_t)G.P);
    G.dv_kw = dstd::fast_div((uint32_t)G.KW);
    G.dv_pc = dstd::fast_div((uint32_t)G.PC);
    return DSTD_OK;
}

struct ConvWs {
    size_t wt, key, L, R, off;                        // both passes
    size_t px, src, P, dL, dR;                        // backward sort extras
    size_t row, eL, eR, crlive, gam, uq, q, rend, part, zlive, dq;   // backward
    size_t total;
};

ConvWs conv_ws_layout(int M, const dstd::ConvGeom &g, int64_t B, bool backward) {
    ConvWs w{};
    size_t off = 0;
    const size_t n = (size_t)B * g.Hp * g.Wp * g.PC;  // inputs (cell-major)
    const size_t nw = (size_t)g.KH * g.KW * g.C_in * g.C_out;
    const size_t nout = (size_t)B * g.Ho * g.Wo * g.C_out;
    const int R = M + 3;
    if (B == 0 && !backward) return w;
    // weights / P and the records sorted per cell row; batched reads may run
    // past the last record by up to kSortPad slots
    w.wt = off; off += align_up(nw * sizeof(float));
    const size_t nr = n + dstd::kSortPad;
    w.key = off; off += align_up(nr * sizeof(int));
    w.L = off; off += align_up(nr * sizeof(float));
    w.R = off; off += align_up(nr * sizeof(float));
    w.off = off; off += align_up((size_t)B * g.Hp * (size_t)dstd::conv_off_stride(R, g) * sizeof(int));
    if (backward) {
        w.px = off; off += align_up(nr * sizeof(int));
        w.src = off; off += align_up(nr * sizeof(int));
        w.P = off; off += align_up(nr * (size_t)(g.KH * g.KW) * sizeof(float));
        w.dL = off; off += align_up(nr * sizeof(float));
        w.dR = off; off += align_up(nr * sizeof(float));
        w.row = off; off += align_up(n * sizeof(int));
        w.eL = off; off += align_up(n * sizeof(float));
        w.eR = off; off += align_up(n * sizeof(float));
        w.crlive = off; off += align_up((size_t)B * g.Hp * sizeof(int));
        w.gam = off; off += align_up(nout * sizeof(float));
        w.uq = off; off += align_up(nout * sizeof(float));
        w.q = off; off += align_up(nout * sizeof(int));
        w.rend = off; off += align_up((size_t)B * g.Ho * g.Wo * sizeof(int));
        w.dq = off; off += align_up((size_t)g.C_out * sizeof(float));  // dead-neuron term per channel
        dstd::ConvDwPlan dp = dstd::plan_conv_dw(g, B, M);
        w.part = off; off += align_up((size_t)dp.nsplit * nw * sizeof(float));
        w.zlive = off; off += align_up((size_t)dp.nsplit * sizeof(int));
    }
    w.total = off;
    return w;
}

// Synfire terms of a backward call (NULL: off).
dstd_status check_synfire(const dstd_synfire_params *sp) {
    if (!sp) return DSTD_OK;
    const float g[3] = {sp->gamma_head, sp->gamma_tail, sp->gamma_q};
    for (float v : g)
        if (!(isfinite(v) && v >= 0.f))
            return fail(DSTD_ERR_PARAM, "synfire gammas must be finite and >= 0");
    if (!isfinite(sp->t_head) || !isfinite(sp->t_tail))
        return fail(DSTD_ERR_PARAM, "synfire t_head and t_tail must be finite");
    if (!(isfinite(sp->scale) && sp->scale > 0.f))
        return fail(DSTD_ERR_PARAM, "synfire scale must be finite and > 0");
    return DSTD_OK;
}

dstd::Synfire make_synfire(const dstd_synfire_params *sp, float *dq) {
    dstd::Synfire f{};
    if (!sp) return f;
    f.on = 1;
    f.gh = sp->gamma_head;
    f.gt = sp->gamma_tail;
    f.th = sp->t_head;
    f.tt = sp->t_tail;
    f.gq = sp->gamma_q;
    f.scale = sp->scale;
    f.dq = dq;
    return f;
}

dstd_status dense_backward(const dstd_lif_params *p, const dstd_synfire_params *sp, int64_t B,
                           int64_t N_in, int64_t N_out, const float *t_in, const void *W,
                           dstd_dtype w_dtype, const float *t_out, const float *slope,
                           const int32_t *q_idx, const float *grad_t_out, float *grad_W,
                           float *grad_t_in, void *ws, size_t ws_bytes, void *stream);
dstd_status conv_backward(const dstd_lif_params *p, const dstd_synfire_params *sp,
                          const dstd_conv_shape *cs, int64_t B, const float *t_in, const void *W,
                          dstd_dtype w_dtype, const float *t_out, const float *slope,
                          const int32_t *q_idx, const float *grad_t_out, float *grad_W,
                          float *grad_t_in, void *ws, size_t ws_bytes, void *stream);

}  // namespace

extern "C" {

const char *dstd_status_string(dstd_status s) {
    switch (s) {
        case DSTD_OK: return "ok";
        case DSTD_ERR_NULL: return "null pointer";
        case DSTD_ERR_SHAPE: return "invalid shape";
        case DSTD_ERR_PARAM: return "invalid parameter";
        case DSTD_ERR_UNSUPPORTED: return "unsupported";
        case DSTD_ERR_WORKSPACE: return "workspace too small or misaligned";
        case DSTD_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char *dstd_last_error(void) { return g_err; }

int32_t dstd_version(void) { return 100; }

size_t dstd_lif_forward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                       int64_t N_out) {
    if (check_params(p, kDenseFlags) != DSTD_OK || check_dims(B, N_in, N_out) != DSTD_OK) return 0;
    size_t need = (p->flags & DSTD_FLAG_CONTRACT_MFMA) ? 0 : dense_ws_layout(p->M, B, N_in, N_out, false).total;
    if (mfma_possible(p, B, N_in, N_out)) need = std::max(need, mfma_ws_bytes(p->M, B, N_in, N_out));
    return need;
}

size_t dstd_lif_backward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                        int64_t N_out) {
    if (check_params(p, kDenseFlags) != DSTD_OK || check_dims(B, N_in, N_out) != DSTD_OK) return 0;
    return dense_ws_layout(p->M, B, N_in, N_out, true).total;
}

dstd_status dstd_lif_forward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                             const float *t_in, const void *W, dstd_dtype w_dtype, float *t_out,
                             float *slope, int32_t *q_idx, void *ws, size_t ws_bytes,
                             void *stream) {
    dstd_status s = check_params(p, kDenseFlags);
    if (s != DSTD_OK) return s;
    if ((s = check_dims(B, N_in, N_out)) != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if ((p->flags & DSTD_FLAG_CONTRACT_MFMA) && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_UNSUPPORTED, "the MFMA contraction takes bf16 weights");
    if (B * N_out > 0 && (!t_out || !slope || !q_idx))
        return fail(DSTD_ERR_NULL, "t_out, slope and q_idx are required");
    if (B * N_in > 0 && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (N_in * N_out > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    const bool mfma = w_dtype == DSTD_BF16 && mfma_possible(p, B, N_in, N_out);
    if (mfma) {
        if ((s = check_ws(ws, ws_bytes, mfma_ws_bytes(p->M, B, N_in, N_out))) != DSTD_OK) return s;
        if (B * N_out == 0) return DSTD_OK;
        LifConst C = make_const(p);
        hipError_t e = dstd::launch_forward_mfma(
            C, B, N_in, N_out, static_cast<const uint16_t *>(W), ws,
            at<float>(ws, mfma_ws_events(B, N_in)), t_in, t_out, slope, q_idx,
            static_cast<hipStream_t>(stream));
        return hip_status(e, "forward (MFMA) launch");
    }
    DenseWs L = dense_ws_layout(p->M, B, N_in, N_out, false);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    if (B * N_out == 0) return DSTD_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    LifConst C = make_const(p);
    dstd::SortedEv srt{at<int>(ws, L.sj), at<int>(ws, L.sr), at<float>(ws, L.sL),
                       at<float>(ws, L.sR), L.sstride, at<int>(ws, L.rs)};
    hipError_t e = dstd::launch_forward(C, B, N_in, N_out, W, w_dtype == DSTD_BF16, at<void>(ws, L.wt),
                                        srt, at<int>(ws, L.nvalid), t_in, t_out, slope, q_idx, st);
    return hip_status(e, "forward launch");
}

}  // extern "C"

// Scratch of the allocation-free forward: one array per GPU, reserved when the
// library's code object is loaded there and kept until the process ends. In
// host code `scratch` only names the symbol; its device address comes from
// hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) unsigned char scratch[DSTD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
void *g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;

dstd_status scratch_for_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(DSTD_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(DSTD_ERR_UNSUPPORTED, "device index %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(DSTD_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return DSTD_OK;
}

}  // namespace

extern "C" {

dstd_status dstd_lif_forward_noalloc(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                     int64_t N_out, const float *t_in, const void *W,
                                     dstd_dtype w_dtype, float *t_out, float *slope,
                                     int32_t *q_idx, void *stream) {
    // host validation first: nothing touches the device before the sizes pass
    dstd_status s = check_params(p, kDenseFlags);
    if (s != DSTD_OK) return s;
    if ((s = check_dims(B, N_in, N_out)) != DSTD_OK) return s;
    const size_t need = dstd_lif_forward_workspace_size(p, B, N_in, N_out);
    if (need > (size_t)DSTD_NOALLOC_SCRATCH_BYTES)
        return fail(DSTD_ERR_WORKSPACE,
                    "layer needs %zu bytes of scratch; the allocation-free forward holds %zu "
                    "(use dstd_lif_forward with a caller workspace)",
                    need, (size_t)DSTD_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    if (need > 0 && (s = scratch_for_current_device(&ws)) != DSTD_OK) return s;
    // the forward's kernels write every scratch word they read: nothing to clear
    return dstd_lif_forward(p, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx, ws,
                            need > 0 ? (size_t)DSTD_NOALLOC_SCRATCH_BYTES : 0, stream);
}

dstd_status dstd_lif_backward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                              const float *t_in, const void *W, dstd_dtype w_dtype,
                              const float *t_out, const float *slope, const int32_t *q_idx,
                              const float *grad_t_out, float *grad_W, float *grad_t_in, void *ws,
                              size_t ws_bytes, void *stream) {
    return dense_backward(p, nullptr, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx,
                          grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream);
}

dstd_status dstd_lif_backward_synfire(const dstd_lif_params *p, const dstd_synfire_params *sp,
                                      int64_t B, int64_t N_in, int64_t N_out, const float *t_in,
                                      const void *W, dstd_dtype w_dtype, const float *t_out,
                                      const float *slope, const int32_t *q_idx,
                                      const float *grad_t_out, float *grad_W, float *grad_t_in,
                                      void *ws, size_t ws_bytes, void *stream) {
    return dense_backward(p, sp, B, N_in, N_out, t_in, W, w_dtype, t_out, slope, q_idx,
                          grad_t_out, grad_W, grad_t_in, ws, ws_bytes, stream);
}

}  // extern "C"

namespace {

dstd_status dense_backward(const dstd_lif_params *p, const dstd_synfire_params *sp, int64_t B,
                           int64_t N_in, int64_t N_out, const float *t_in, const void *W,
                           dstd_dtype w_dtype, const float *t_out, const float *slope,
                           const int32_t *q_idx, const float *grad_t_out, float *grad_W,
                           float *grad_t_in, void *ws, size_t ws_bytes, void *stream) {
    // the contraction flags select the forward's kernels; the backward takes them as given
    dstd_status s = check_params(p, kDenseFlags);
    if (s != DSTD_OK) return s;
    if ((s = check_synfire(sp)) != DSTD_OK) return s;
    if ((s = check_dims(B, N_in, N_out)) != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * N_out > 0 && (!t_out || !slope || !q_idx || !grad_t_out))
        return fail(DSTD_ERR_NULL, "t_out, slope, q_idx and grad_t_out are required");
    if (B * N_in > 0 && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (grad_t_in && N_in * N_out > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    DenseWs L = dense_ws_layout(p->M, B, N_in, N_out, true);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    // Empty sizes need no special case: with B == 0 the dW kernel writes
    // zeros; dt_in is zeroed by the event sort and only inputs with events
    // are written after that (no memset is used, so the call stays safe to
    // capture in a graph).
    LifConst C = make_const(p);
    dstd::DenseBwdWs bw;
    bw.row = at<int>(ws, L.row);
    bw.L = at<float>(ws, L.L);
    bw.R = at<float>(ws, L.R);
    bw.srt = dstd::SortedEv{at<int>(ws, L.sj), at<int>(ws, L.sr), at<float>(ws, L.sL),
                            at<float>(ws, L.sR), L.sstride, at<int>(ws, L.rs)};
    bw.n_valid = at<int>(ws, L.nvalid);
    bw.wt = at<void>(ws, L.wt);
    bw.gam = at<float>(ws, L.gam);
    bw.uq = at<float>(ws, L.uq);
    bw.q = at<int>(ws, L.q);
    bw.part = at<float>(ws, L.part);
    e = dstd::launch_backward(C, B, N_in, N_out, W, w_dtype == DSTD_BF16, t_in, t_out, slope,
                              q_idx, grad_t_out, bw, grad_W, grad_t_in,
                              make_synfire(sp, at<float>(ws, L.dq)), st);
    return hip_status(e, "backward launch");
}

}  // namespace

extern "C" {

dstd_status dstd_softmax_ce_grad(int64_t B, int64_t N, const float *t_out, const int32_t *labels,
                                 float tau_soft, float t_cap, float *grad_t, float *loss,
                                 void *stream) {
    if (B < 0 || B > 65535 || N < 1 || N >= (1 << 24))
        return fail(DSTD_ERR_SHAPE, "need 0 <= B <= 65535 and 1 <= N < 2^24");
    if (!(isfinite(tau_soft) && tau_soft > 0.f)) return fail(DSTD_ERR_PARAM, "tau_soft must be > 0");
    if (!isfinite(t_cap)) return fail(DSTD_ERR_PARAM, "t_cap must be finite");
    if (!loss || (B > 0 && (!t_out || !labels || !grad_t)))
        return fail(DSTD_ERR_NULL, "t_out, labels, grad_t and loss are required");
    hipError_t e = dstd::launch_softmax_ce(B, N, t_out, labels, tau_soft, t_cap, grad_t, loss,
                                           static_cast<hipStream_t>(stream));
    return hip_status(e, "softmax_ce launch");
}

dstd_status dstd_mse_grad(int64_t B, int64_t N, const float *t_out, const float *target,
                          float *grad_t, float *loss, void *stream) {
    if (B < 0 || B > 65535 || N < 1 || N >= (1 << 24))
        return fail(DSTD_ERR_SHAPE, "need 0 <= B <= 65535 and 1 <= N < 2^24");
    if (!loss || (B > 0 && (!t_out || !target || !grad_t)))
        return fail(DSTD_ERR_NULL, "t_out, target, grad_t and loss are required");
    hipError_t e = dstd::launch_mse(B, N, t_out, target, grad_t, loss,
                                    static_cast<hipStream_t>(stream));
    return hip_status(e, "mse launch");
}

size_t dstd_lif_conv_forward_workspace_size(const dstd_lif_params *p, const dstd_conv_shape *cs,
                                            int64_t B) {
    dstd::ConvGeom g;
    if (check_params(p, DSTD_FLAG_CONV_KEEP) != DSTD_OK || check_conv(cs, B, p->M, &g) != DSTD_OK)
        return 0;
    // a forward that keeps its sort for the backward needs the backward's size
    return conv_ws_layout(p->M, g, B, (p->flags & DSTD_FLAG_CONV_KEEP) != 0).total;
}

size_t dstd_lif_conv_backward_workspace_size(const dstd_lif_params *p, const dstd_conv_shape *cs,
                                             int64_t B) {
    dstd::ConvGeom g;
    if (check_params(p, DSTD_FLAG_CONV_REUSE) != DSTD_OK || check_conv(cs, B, p->M, &g) != DSTD_OK)
        return 0;
    return conv_ws_layout(p->M, g, B, true).total;
}

dstd_status dstd_lif_conv_forward(const dstd_lif_params *p, const dstd_conv_shape *cs, int64_t B,
                                  const float *t_in, const void *W, dstd_dtype w_dtype,
                                  float *t_out, float *slope, int32_t *q_idx, void *ws,
                                  size_t ws_bytes, void *stream) {
    dstd_status s = check_params(p, DSTD_FLAG_CONV_KEEP);
    if (s != DSTD_OK) return s;
    dstd::ConvGeom g;
    if ((s = check_conv(cs, B, p->M, &g)) != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B > 0 && (!t_in || !W || !t_out || !slope || !q_idx))
        return fail(DSTD_ERR_NULL, "t_in, W, t_out, slope and q_idx are required");
    // keeping the sort for the backward needs the backward's workspace
    const bool keep = (p->flags & DSTD_FLAG_CONV_KEEP) != 0;
    ConvWs L = conv_ws_layout(p->M, g, B, keep);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    if (B == 0) return DSTD_OK;
    LifConst C = make_const(p);
    dstd::ConvSorted srt{at<int>(ws, L.key), at<float>(ws, L.L), at<float>(ws, L.R),
                         at<int>(ws, L.off), nullptr, nullptr, nullptr, nullptr, nullptr};
    dstd::CellEv ev{nullptr, nullptr, nullptr, nullptr};
    if (keep) {
        srt.px = at<int>(ws, L.px);
        srt.src = at<int>(ws, L.src);
        srt.dL = at<float>(ws, L.dL);
        srt.dR = at<float>(ws, L.dR);
        ev = dstd::CellEv{at<int>(ws, L.row), at<float>(ws, L.eL), at<float>(ws, L.eR),
                          at<int>(ws, L.crlive)};
    }
    hipError_t e = dstd::launch_conv_forward(C, g, B, W, w_dtype == DSTD_BF16, at<float>(ws, L.wt),
                                             srt, ev, t_in, t_out, slope, q_idx,
                                             static_cast<hipStream_t>(stream));
    return hip_status(e, "conv forward launch");
}

dstd_status dstd_lif_conv_backward(const dstd_lif_params *p, const dstd_conv_shape *cs, int64_t B,
                                   const float *t_in, const void *W, dstd_dtype w_dtype,
                                   const float *t_out, const float *slope, const int32_t *q_idx,
                                   const float *grad_t_out, float *grad_W, float *grad_t_in,
                                   void *ws, size_t ws_bytes, void *stream) {
    return conv_backward(p, nullptr, cs, B, t_in, W, w_dtype, t_out, slope, q_idx, grad_t_out,
                         grad_W, grad_t_in, ws, ws_bytes, stream);
}

dstd_status dstd_lif_conv_backward_synfire(const dstd_lif_params *p, const dstd_synfire_params *sp,
                                           const dstd_conv_shape *cs, int64_t B,
                                           const float *t_in, const void *W, dstd_dtype w_dtype,
                                           const float *t_out, const float *slope,
                                           const int32_t *q_idx, const float *grad_t_out,
                                           float *grad_W, float *grad_t_in, void *ws,
                                           size_t ws_bytes, void *stream) {
    return conv_backward(p, sp, cs, B, t_in, W, w_dtype, t_out, slope, q_idx, grad_t_out,
                         grad_W, grad_t_in, ws, ws_bytes, stream);
}

size_t dstd_synfire_penalty_workspace_size(int64_t B, int64_t rows, int64_t spatial) {
    if (B < 0 || rows < 0 || spatial < 0) return 0;
    const int64_t n_tb = dstd::synfire_value_blocks(B * rows * spatial);
    return align_up((size_t)(rows + n_tb) * sizeof(float));
}

dstd_status dstd_synfire_penalty(const dstd_synfire_params *sp, int64_t B, int64_t rows,
                                 int64_t spatial, int64_t row_len, const float *t_out,
                                 const void *W, dstd_dtype w_dtype, float *value, void *ws,
                                 size_t ws_bytes, void *stream) {
    if (!sp || !value) return fail(DSTD_ERR_NULL, "synfire parameters and value are required");
    dstd_status s = check_synfire(sp);
    if (s != DSTD_OK) return s;
    if (B < 0 || rows < 0 || spatial < 0 || row_len < 0)
        return fail(DSTD_ERR_SHAPE, "sizes must be >= 0");
    const int64_t lim = (int64_t)1 << 31;
    if (B > 0 && rows > 0 && spatial > 0 && B * rows * spatial >= lim)
        return fail(DSTD_ERR_SHAPE, "B * rows * spatial must be < 2^31");
    if (rows > 0 && row_len > 0 && rows * row_len >= lim)
        return fail(DSTD_ERR_SHAPE, "rows * row_len must be < 2^31");
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * rows * spatial > 0 && !t_out) return fail(DSTD_ERR_NULL, "t_out is NULL");
    if (rows * row_len > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    if ((s = check_ws(ws, ws_bytes, dstd_synfire_penalty_workspace_size(B, rows, spatial))) != DSTD_OK)
        return s;
    hipError_t e = dstd::launch_synfire_value(make_synfire(sp, nullptr), B, rows, spatial, row_len,
                                              t_out, W, w_dtype == DSTD_BF16,
                                              static_cast<float *>(ws), value,
                                              static_cast<hipStream_t>(stream));
    return hip_status(e, "synfire value launch");
}

}  // extern "C"

namespace {

dstd_status conv_backward(const dstd_lif_params *p, const dstd_synfire_params *sp,
                          const dstd_conv_shape *cs, int64_t B, const float *t_in, const void *W,
                          dstd_dtype w_dtype, const float *t_out, const float *slope,
                          const int32_t *q_idx, const float *grad_t_out, float *grad_W,
                          float *grad_t_in, void *ws, size_t ws_bytes, void *stream) {
    dstd_status s = check_params(p, DSTD_FLAG_CONV_REUSE);
    if (s != DSTD_OK) return s;
    if ((s = check_synfire(sp)) != DSTD_OK) return s;
    dstd::ConvGeom g;
    if ((s = check_conv(cs, B, p->M, &g)) != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B > 0 && (!t_in || !t_out || !slope || !q_idx || !grad_t_out))
        return fail(DSTD_ERR_NULL, "t_in, t_out, slope, q_idx and grad_t_out are required");
    if (grad_t_in && B > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    if (grad_t_in && g.C_out > dstd::kConvMaxCoutDt)
        return fail(DSTD_ERR_UNSUPPORTED, "grad_t_in of a conv layer needs C_out <= %d",
                    dstd::kConvMaxCoutDt);
    ConvWs L = conv_ws_layout(p->M, g, B, true);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    LifConst C = make_const(p);
    dstd::ConvBwdWs bw;
    bw.row = at<int>(ws, L.row);
    bw.L = at<float>(ws, L.eL);
    bw.R = at<float>(ws, L.eR);
    bw.gam = at<float>(ws, L.gam);
    bw.uq = at<float>(ws, L.uq);
    bw.q = at<int>(ws, L.q);
    bw.rend = at<int>(ws, L.rend);
    bw.crlive = at<int>(ws, L.crlive);
    bw.part = at<float>(ws, L.part);
    bw.zlive = at<int>(ws, L.zlive);
    bw.wt = at<float>(ws, L.wt);
    bw.srt = dstd::ConvSorted{at<int>(ws, L.key), at<float>(ws, L.L), at<float>(ws, L.R),
                              at<int>(ws, L.off), at<int>(ws, L.px), at<int>(ws, L.src),
                              at<float>(ws, L.P), at<float>(ws, L.dL), at<float>(ws, L.dR)};
    const bool reuse = (p->flags & DSTD_FLAG_CONV_REUSE) != 0;
    // With B == 0 the dW kernel still runs (one empty split) and writes zeros.
    hipError_t e = dstd::launch_conv_backward(C, g, B, W, w_dtype == DSTD_BF16, t_in, t_out, slope,
                                              q_idx, grad_t_out, bw, grad_W, grad_t_in,
                                              make_synfire(sp, at<float>(ws, L.dq)), reuse,
                                              static_cast<hipStream_t>(stream));
    return hip_status(e, "conv backward launch");
}

}  // namespace

// ------------------------------------------------------------------ exact --
namespace {

// The exact path uses tau_m, tau_s, threshold, t_max and flags; the grid
// fields (M, t0, dt) do not apply and are not read.
dstd_status check_exact(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                        dstd_lif_params *q) {
    if (!p) return fail(DSTD_ERR_NULL, "params is NULL");
    *q = *p;
    q->M = 1;
    q->t0 = 0.f;
    q->dt = 1.f;
    q->t_max = INFINITY;
    dstd_status s = check_params(q);
    if (s != DSTD_OK) return s;
    if (isnan(p->t_max)) return fail(DSTD_ERR_PARAM, "t_max must not be NaN");
    if ((s = check_dims(B, N_in, N_out)) != DSTD_OK) return s;
    if (N_in > dstd::kExactMaxIn)
        return fail(DSTD_ERR_UNSUPPORTED, "the exact path sorts at most %d inputs per sample (N_in = %lld)",
                    dstd::kExactMaxIn, (long long)N_in);
    return DSTD_OK;
}

struct ExactWs {
    size_t wt, j, t, len, r_lo, alpha, beta, kl, kmax, n, P, PT, total;
};

ExactWs exact_ws_layout(int64_t B, int64_t N_in, int64_t N_out, bool backward) {
    ExactWs w{};
    size_t off = 0;
    if (backward) {
        w.P = off; off += align_up((size_t)B * (size_t)N_out * 4 * sizeof(float));
        w.PT = off; off += align_up((size_t)B * (size_t)N_out * 4 * sizeof(float));
    } else if (B * N_out > 0) {
        const size_t ns = (size_t)(B * N_in) + dstd::kExactPad;
        w.wt = off; off += align_up((size_t)N_in * (size_t)N_out * sizeof(float));
        w.j = off; off += align_up(ns * sizeof(int));
        w.t = off; off += align_up(ns * sizeof(float));
        w.len = off; off += align_up(ns * sizeof(float));
        w.r_lo = off; off += align_up(ns * sizeof(float));
        w.alpha = off; off += align_up(ns * sizeof(double));
        w.beta = off; off += align_up(ns * sizeof(double));
        w.kl = off; off += align_up(ns * sizeof(double));
        w.kmax = off; off += align_up(ns * sizeof(float));
        w.n = off; off += align_up((size_t)B * sizeof(int));
    }
    w.total = off;
    return w;
}

}  // namespace

extern "C" {

size_t dstd_exact_forward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                         int64_t N_out) {
    dstd_lif_params q;
    if (check_exact(p, B, N_in, N_out, &q) != DSTD_OK) return 0;
    return exact_ws_layout(B, N_in, N_out, false).total;
}

size_t dstd_exact_backward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                          int64_t N_out) {
    dstd_lif_params q;
    if (check_exact(p, B, N_in, N_out, &q) != DSTD_OK) return 0;
    return exact_ws_layout(B, N_in, N_out, true).total;
}

dstd_status dstd_exact_forward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                               const float *t_in, const void *W, dstd_dtype w_dtype, float *t_out,
                               float *slope, int32_t *k_idx, void *ws, size_t ws_bytes,
                               void *stream) {
    dstd_lif_params q;
    dstd_status s = check_exact(p, B, N_in, N_out, &q);
    if (s != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * N_out > 0 && (!t_out || !slope || !k_idx))
        return fail(DSTD_ERR_NULL, "t_out, slope and k_idx are required");
    if (B * N_in > 0 && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (N_in * N_out > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    ExactWs L = exact_ws_layout(B, N_in, N_out, false);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    if (B * N_out == 0) return DSTD_OK;
    LifConst C = make_const(&q);
    dstd::ExactRecs rec{at<int>(ws, L.j), at<float>(ws, L.t), at<float>(ws, L.len),
                        at<float>(ws, L.r_lo), at<float>(ws, L.kmax), at<double>(ws, L.alpha),
                        at<double>(ws, L.beta), at<double>(ws, L.kl), at<int>(ws, L.n), N_in};
    hipError_t e = dstd::launch_exact_forward(C, B, N_in, N_out, W, w_dtype == DSTD_BF16,
                                              at<void>(ws, L.wt), rec, t_in, p->t_max, t_out,
                                              slope, k_idx, static_cast<hipStream_t>(stream));
    return hip_status(e, "exact forward launch");
}

dstd_status dstd_exact_backward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                                const float *t_in, const void *W, dstd_dtype w_dtype,
                                const float *t_out, const float *slope, const int32_t *k_idx,
                                const float *grad_t_out, float *grad_W, float *grad_t_in,
                                void *ws, size_t ws_bytes, void *stream) {
    dstd_lif_params q;
    dstd_status s = check_exact(p, B, N_in, N_out, &q);
    if (s != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * N_out > 0 && (!t_out || !slope || !k_idx || !grad_t_out))
        return fail(DSTD_ERR_NULL, "t_out, slope, k_idx and grad_t_out are required");
    if (B * N_in > 0 && (grad_W || grad_t_in) && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (grad_t_in && N_in * N_out > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    ExactWs L = exact_ws_layout(B, N_in, N_out, true);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    LifConst C = make_const(&q);
    // B == 0: the dW kernel still runs and writes zeros; N_out == 0: the
    // dt_in kernel sums nothing and writes zeros
    hipError_t e = dstd::launch_exact_backward(
        C, B, N_in, N_out, W, w_dtype == DSTD_BF16, t_in, p->t_max, t_out, slope, k_idx,
        grad_t_out, at<float4>(ws, L.P), at<float4>(ws, L.PT), grad_W, grad_t_in,
        static_cast<hipStream_t>(stream));
    return hip_status(e, "exact backward launch");
}

}  // extern "C"

// ------------------------------------------------------------------- skip --
namespace {

dstd_status check_skip(int64_t B, int64_t C1, int64_t C2, int64_t HW) {
    if (B < 0 || C1 < 0 || C2 < 0 || HW < 0)
        return fail(DSTD_ERR_SHAPE, "sizes must be >= 0 (B=%lld C1=%lld C2=%lld HW=%lld)",
                    (long long)B, (long long)C1, (long long)C2, (long long)HW);
    if (B > 65535) return fail(DSTD_ERR_SHAPE, "B = %lld exceeds 65535", (long long)B);
    if ((C1 + C2) * HW >= ((int64_t)1 << 30))
        return fail(DSTD_ERR_SHAPE, "(C1 + C2) * HW must be below 2^30 per sample");
    return DSTD_OK;
}

}  // namespace

extern "C" {

dstd_status dstd_skip_delay_concat(int64_t B, int64_t C1, int64_t C2, int64_t HW, const float *t1,
                                   float delay, const float *t2, float *out, void *stream) {
    dstd_status s = check_skip(B, C1, C2, HW);
    if (s != DSTD_OK) return s;
    if (!isfinite(delay)) return fail(DSTD_ERR_PARAM, "delay must be finite");
    if (B * (C1 + C2) * HW == 0) return DSTD_OK;
    if (!out || (C1 * HW > 0 && !t1) || (C2 * HW > 0 && !t2))
        return fail(DSTD_ERR_NULL, "t1, t2 and out are required");
    hipError_t e = dstd::launch_skip_concat(B, C1 * HW, C2 * HW, t1, delay, t2, out,
                                            static_cast<hipStream_t>(stream));
    return hip_status(e, "skip concat launch");
}

dstd_status dstd_skip_delay_concat_backward(int64_t B, int64_t C1, int64_t C2, int64_t HW,
                                            const float *g, float *g1, int32_t accumulate,
                                            float *g2, void *stream) {
    dstd_status s = check_skip(B, C1, C2, HW);
    if (s != DSTD_OK) return s;
    if (accumulate != 0 && accumulate != 1) return fail(DSTD_ERR_PARAM, "accumulate must be 0 or 1");
    if (B * (C1 + C2) * HW == 0) return DSTD_OK;
    if (!g) return fail(DSTD_ERR_NULL, "g is NULL");
    hipError_t e = dstd::launch_skip_split(B, C1 * HW, C2 * HW, g, g1, accumulate, g2,
                                           static_cast<hipStream_t>(stream));
    return hip_status(e, "skip split launch");
}

}  // extern "C"

// ------------------------------------------------------------- multispike --
namespace {

dstd_status check_ms(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t F_in,
                     int64_t N_out, int64_t F_out) {
    dstd_status s = check_params(p);
    if (s != DSTD_OK) return s;
    if (p->M > dstd::kMsMaxM)
        return fail(DSTD_ERR_UNSUPPORTED, "multi-spike layers support M <= %d (got %d)",
                    dstd::kMsMaxM, p->M);
    if (F_in < 1 || F_out < 1 || F_in > dstd::kMsMaxF || F_out > dstd::kMsMaxF)
        return fail(DSTD_ERR_SHAPE, "F_in and F_out must be in [1, %d]", dstd::kMsMaxF);
    if ((s = check_dims(B, N_in * F_in, N_out)) != DSTD_OK) return s;
    if (N_out * F_out >= ((int64_t)1 << 24) || N_out >= ((int64_t)1 << 22) ||
        B * N_out * (p->M + 1) >= ((int64_t)1 << 31))
        return fail(DSTD_ERR_SHAPE, "N_out (< 2^22), N_out * F_out (< 2^24) or B * N_out * (M + 1) "
                    "(< 2^31) too large");
    return DSTD_OK;
}

struct MsWs { size_t row, L, R, dL, dR, wt, G, part, sj, sr, sL, sR, nvalid, rs, total; };

// forward: the records of every input spike sorted by event row (as the TTFS
// forward's lists) and W^T; backward: per-spike events, W^T and G
MsWs ms_ws_layout(int M, int64_t B, int64_t N_in, int64_t F_in, int64_t N_out, bool backward) {
    MsWs w{};
    size_t off = 0;
    const size_t n = (size_t)(B * N_in * F_in);
    if (backward) {
        w.row = off; off += align_up(n * sizeof(int));
        w.L = off; off += align_up(n * sizeof(float));
        w.R = off; off += align_up(n * sizeof(float));
        w.dL = off; off += align_up(n * sizeof(float));
        w.dR = off; off += align_up(n * sizeof(float));
        w.G = off; off += align_up((size_t)B * (size_t)(M + 1) * (size_t)N_out * sizeof(float));
        const int S = dstd::ms_dw_splits(M, B, N_in, N_out);
        w.part = off;
        if (S > 1) off += align_up((size_t)S * (size_t)N_in * (size_t)N_out * sizeof(float));
    } else {
        const size_t ns = n + dstd::kSortPad;
        w.sj = off; off += align_up(ns * sizeof(int));
        w.sr = off; off += align_up(ns * sizeof(int));
        w.sL = off; off += align_up(ns * sizeof(float));
        w.sR = off; off += align_up(ns * sizeof(float));
        w.nvalid = off; off += align_up((size_t)B * sizeof(int));
        w.rs = off; off += align_up((size_t)B * (M + 4) * sizeof(int));
    }
    w.wt = off; off += align_up((size_t)N_in * (size_t)N_out * sizeof(float));
    w.total = off;
    return w;
}

}  // namespace

extern "C" {

size_t dstd_lif_multispike_forward_workspace_size(const dstd_lif_params *p, int64_t B,
                                                  int64_t N_in, int64_t F_in, int64_t N_out,
                                                  int64_t F_out) {
    if (check_ms(p, B, N_in, F_in, N_out, F_out) != DSTD_OK) return 0;
    if (B * N_out == 0) return 0;
    return ms_ws_layout(p->M, B, N_in, F_in, N_out, false).total;
}

size_t dstd_lif_multispike_backward_workspace_size(const dstd_lif_params *p, int64_t B,
                                                   int64_t N_in, int64_t F_in, int64_t N_out,
                                                   int64_t F_out) {
    if (check_ms(p, B, N_in, F_in, N_out, F_out) != DSTD_OK) return 0;
    return ms_ws_layout(p->M, B, N_in, F_in, N_out, true).total;
}

dstd_status dstd_lif_multispike_forward(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                        int64_t F_in, int64_t N_out, int64_t F_out,
                                        const float *t_in, const void *W, dstd_dtype w_dtype,
                                        float *t_out, float *slope, int32_t *q_idx, float *cur,
                                        void *ws, size_t ws_bytes, void *stream) {
    dstd_status s = check_ms(p, B, N_in, F_in, N_out, F_out);
    if (s != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * N_out == 0) return DSTD_OK;
    if (!t_out || !slope || !q_idx || !cur)
        return fail(DSTD_ERR_NULL, "t_out, slope, q_idx and cur are required");
    if (N_in > 0 && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (N_in > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    MsWs L = ms_ws_layout(p->M, B, N_in, F_in, N_out, false);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    LifConst C = make_const(p);
    dstd::SortedEv srt{at<int>(ws, L.sj), at<int>(ws, L.sr), at<float>(ws, L.sL),
                       at<float>(ws, L.sR), N_in * F_in, at<int>(ws, L.rs)};
    hipError_t e = dstd::launch_ms_forward(C, B, N_in, F_in, N_out, F_out, W,
                                           w_dtype == DSTD_BF16, at<void>(ws, L.wt), srt,
                                           at<int>(ws, L.nvalid), t_in, t_out, slope, q_idx, cur,
                                           static_cast<hipStream_t>(stream));
    return hip_status(e, "multi-spike forward launch");
}

dstd_status dstd_lif_multispike_backward(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                         int64_t F_in, int64_t N_out, int64_t F_out,
                                         const float *t_in, const void *W, dstd_dtype w_dtype,
                                         const float *t_out, const float *slope,
                                         const int32_t *q_idx, const float *cur,
                                         const float *grad_t_out, float *grad_W,
                                         float *grad_t_in, void *ws, size_t ws_bytes,
                                         void *stream) {
    dstd_status s = check_ms(p, B, N_in, F_in, N_out, F_out);
    if (s != DSTD_OK) return s;
    if (w_dtype != DSTD_F32 && w_dtype != DSTD_BF16)
        return fail(DSTD_ERR_PARAM, "unknown weight dtype %d", (int)w_dtype);
    if (B * N_out > 0 && (!t_out || !slope || !q_idx || !cur || !grad_t_out))
        return fail(DSTD_ERR_NULL, "t_out, slope, q_idx, cur and grad_t_out are required");
    if (B * N_in > 0 && !t_in) return fail(DSTD_ERR_NULL, "t_in is NULL");
    if (grad_t_in && N_in * N_out > 0 && !W) return fail(DSTD_ERR_NULL, "W is NULL");
    MsWs L = ms_ws_layout(p->M, B, N_in, F_in, N_out, true);
    if ((s = check_ws(ws, ws_bytes, L.total)) != DSTD_OK) return s;
    LifConst C = make_const(p);
    dstd::MsEvents ev{at<int>(ws, L.row), at<float>(ws, L.L), at<float>(ws, L.R),
                      at<float>(ws, L.dL), at<float>(ws, L.dR)};
    // B == 0: the dW kernel still runs and writes zeros; N_out == 0: dt_in
    // sums nothing and writes zeros
    hipError_t e = dstd::launch_ms_backward(C, B, N_in, F_in, N_out, F_out, W,
                                            w_dtype == DSTD_BF16, at<void>(ws, L.wt), ev, t_in,
                                            t_out, slope, q_idx, cur, grad_t_out,
                                            at<float>(ws, L.G), at<float>(ws, L.part), grad_W,
                                            grad_t_in,
                                            static_cast<hipStream_t>(stream));
    return hip_status(e, "multi-spike backward launch");
}

}  // extern "C"
