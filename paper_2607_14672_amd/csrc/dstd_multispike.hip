// dstd_multispike.hip -- multi-spike DSTD for a dense layer on gfx950 (App.
// "multi-spikes", Eq. (Vmem_multiSpikes) and its DSTD form).
//
// Every input neuron may fire F_in times; each input spike gets its own
// events, and the weighted events sum them. An output neuron fires each time
// v reaches V_th; v is then reset to 0 while the synaptic current carries on,
// so after a spike at T_q + u0 the rest of interval q is the segment
// v(u) = I K(u - u0) (V = 0, I the current at the spike). The first F_out
// spikes are kept. The spikes of one neuron are sequential (each depends on
// the previous one through the reset); neurons and samples are independent.
//
// Kernels:
//  ms_prep_kernel: events of every input spike (row, L, R, dL/dt, dR/dt),
//    once per call, and the transposed weights; the backward role also
//    builds G[b][m][i] = dL/dw^_im from the neuron's spikes (adjoints through
//    the reset chain, implicit function theorem per spike).
//  ms_fwd_kernel: the TTFS forward's walk over the sample's input spikes
//    sorted by event row (the records are input spikes), closing grid points
//    into a scan with reset that solves each crossing at once.
//  ms_dw_kernel / ms_dtin_kernel: the event contractions with G read from
//    memory (lanes over neurons, so G rows are coalesced).
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"
#include "dstd_walk.h"
#include "dstd_rows.h"

namespace dstd {

namespace {

constexpr int kMsPrepThreads = 256;
constexpr int kMsWaves = 4;  // waves per dW / dt_in block (one input each)
constexpr int kMsGReg = 8;   // spikes per neuron whose G terms are summed in registers

// K(u) in fp64 for the state carried after a reset (Table "tab:kernel")
__device__ __forceinline__ double kern_d64(const LifConst &C, double u) {
    const double tv = C.tv, ti = C.ti;
    switch (C.kind) {
        case kEqual: return u * exp(-u / ti);
        case kInfTau: return -ti * expm1(-u / ti);
        case kInfInf: return u;
        default: {
            const double c = tv * ti / (tv - ti), kap = 1.0 / ti - 1.0 / tv;
            return -c * exp(-u / tv) * expm1(-kap * u);
        }
    }
}

// Setup roles by block: [0, n_ev) events of kMsPrepThreads input spikes,
// [n_ev, n_ev + n_tr) one 32 x 32 tile of W^T each, then (backward) G of
// kMsPrepThreads neurons each.
template <typename WT, int KS>
__global__ __launch_bounds__(kMsPrepThreads) void ms_prep_kernel(
    LifConst C, int64_t n_spk, int n_ev, int n_tr, int N_in, int N_out, const float *__restrict__ t_in,
    MsEvents ev, const WT *__restrict__ W, WT *__restrict__ Wt, MsGrad gr) {
    __shared__ WT buf[32][33];
    const int blk = blockIdx.x;
    if (blk < n_ev) {
        const int64_t x = static_cast<int64_t>(blk) * kMsPrepThreads + threadIdx.x;
        if (x < n_spk) {
            const Event e = bin_event<KS>(C, t_in[x]);
            ev.row[x] = e.row;
            ev.L[x] = e.L;
            ev.R[x] = e.R;
            ev.dL[x] = e.dL;
            ev.dR[x] = e.dR;
        }
        return;
    }
    if (blk < n_ev + n_tr) {
        transpose_tile<WT, kMsPrepThreads>(N_out, N_in, W, Wt, blk - n_ev, buf);
        return;
    }
    // G of one neuron (b, i): gbar_k = g_k + gbar_{k+1} d t_{k+1}/d t_k,
    // gamma_k = -gbar_k / slope_k, G[m] = sum_k gamma_k c_k(m) with
    //   c_k(m) = K(t_k - T_m)                                 q_{k-1} < m <= q_k
    //          = e^{-(t_{k-1} - T_m)/tau_I} K(t_k - t_{k-1})  m <= q_{k-1}
    const int64_t o = static_cast<int64_t>(blk - n_ev - n_tr) * kMsPrepThreads + threadIdx.x;
    if (o >= gr.n) return;
    const int64_t b = o / N_out, i = o - b * N_out;
    const int F = gr.F;
    const int64_t so = o * F;
    const int R = C.M + 1;
    float *Gc = gr.G + b * R * N_out + i;  // G[b][m][i] at Gc[m * N_out]
    int K = 0;
    while (K < F && gr.q[so + K] >= 0) ++K;
    if (K <= kMsGReg) {
        // gamma_k and the spike constants in registers (backward over k), then
        // each G[m] summed over the spikes (same order, k descending) and
        // written once
        float gam[kMsGReg], tkv[kMsGReg], kdv[kMsGReg];
        int qv[kMsGReg];
        float gnext = 0.f;
#pragma unroll
        for (int k = kMsGReg - 1; k >= 0; --k) {
            gam[k] = 0.f;
            tkv[k] = 0.f;
            kdv[k] = 0.f;
            qv[k] = -1;
            if (k < K) {
                const float tk = gr.t[so + k];
                const float gbar = gr.g[so + k] + gnext;
                gam[k] = -gbar / fmaxf(gr.slope[so + k], C.slope_floor);
                qv[k] = min(gr.q[so + k], C.M);
                tkv[k] = tk;
                if (k > 0) {
                    const double tp = gr.t[so + k - 1];
                    const double tkd = tk;
                    kdv[k] = kern<KS>(C, static_cast<float>(tkd - tp));
                    const float d = static_cast<float>(tkd - tp);
                    float Kv, Kp;
                    {
                        float f, fp;
                        const Seg sg{0.f, 1.f};  // v = K(u), v' = K'(u) for unit current, V = 0
                        seg_eval<KS>(C, sg, d, f, fp);
                        Kv = f + C.theta;
                        Kp = fp;
                    }
                    const float dprev = gr.cur[so + k - 1] * (Kv * C.inv_ti + Kp) /
                                        fmaxf(gr.slope[so + k], C.slope_floor);
                    gnext = gbar * dprev;
                }
            }
        }
        for (int m = 0; m < R; ++m) {
            const double Tm = fma(static_cast<double>(m), static_cast<double>(C.dt), static_cast<double>(C.t0));
            float a = 0.f;
#pragma unroll
            for (int k = kMsGReg - 1; k >= 0; --k) {
                const int qprev = (k > 0) ? qv[k > 0 ? k - 1 : 0] : -1;
                if (m <= qv[k]) {
                    const float c =
                        (m > qprev)
                            ? kern<KS>(C, static_cast<float>(static_cast<double>(tkv[k]) - Tm))
                            : expf(-static_cast<float>(static_cast<double>(tkv[k > 0 ? k - 1 : 0]) - Tm) *
                                   C.inv_ti) * kdv[k];
                    a += gam[k] * c;
                }
            }
            Gc[static_cast<int64_t>(m) * N_out] = a;
        }
        return;
    }
    for (int m = 0; m < R; ++m) Gc[static_cast<int64_t>(m) * N_out] = 0.f;
    float gnext = 0.f;  // gbar_{k+1} d t_{k+1} / d t_k
    for (int k = K - 1; k >= 0; --k) {
        const float tk = gr.t[so + k];
        const float gbar = gr.g[so + k] + gnext;
        const float gam = -gbar / fmaxf(gr.slope[so + k], C.slope_floor);
        const int qk = min(gr.q[so + k], C.M);  // in range even for inconsistent inputs
        const double tkd = tk;
        if (k == 0) {
            for (int m = 0; m <= qk; ++m) {
                const double Tm = fma(static_cast<double>(m), static_cast<double>(C.dt), static_cast<double>(C.t0));
                Gc[static_cast<int64_t>(m) * N_out] += gam * kern<KS>(C, static_cast<float>(tkd - Tm));
            }
        } else {
            const double tp = gr.t[so + k - 1];
            const int qp = min(gr.q[so + k - 1], C.M);
            const float Kd = kern<KS>(C, static_cast<float>(tkd - tp));
            for (int m = 0; m <= qk; ++m) {
                const double Tm = fma(static_cast<double>(m), static_cast<double>(C.dt), static_cast<double>(C.t0));
                const float c = (m > qp) ? kern<KS>(C, static_cast<float>(tkd - Tm))
                                         : expf(-static_cast<float>(tp - Tm) * C.inv_ti) * Kd;
                Gc[static_cast<int64_t>(m) * N_out] += gam * c;
            }
            // d t_k / d t_{k-1} = I(t_{k-1}) (K(d)/tau_I + K'(d)) / slope_k
            const float d = static_cast<float>(tkd - tp);
            float Kv, Kp;
            {
                float f, fp;
                const Seg s{0.f, 1.f};  // v = K(u), v' = K'(u) for unit current, V = 0
                seg_eval<KS>(C, s, d, f, fp);
                Kv = f + C.theta;
                Kp = fp;
            }
            const float dprev = gr.cur[so + k - 1] * (Kv * C.inv_ti + Kp) /
                                fmaxf(gr.slope[so + k], C.slope_floor);
            gnext = gbar * dprev;
        }
    }
}

// Interval scan with reset for one neuron; the grid points arrive in order
// through step() (the sorted-row walk of the TTFS forward). In an interval
// the current segment starts at offset u0 (0, or the last spike in it) with
// state (V, I); each crossing is solved at once (seg_test, seg_solve),
// recorded, and the segment restarts there with V = 0 and the current at the
// spike. Without a spike in the interval the state is carried by the fp64
// recurrence; after one, from the segment that ends it.
template <int KS>
struct MsScan {
    double Vd = 0.0, Id = 0.0;
    int nk = 0, F = 0;
    bool ok = false;  // this lane has a neuron (outputs are written)
    int64_t so = 0;   // its first output slot
    float *t_out, *slope, *cur;
    int *q_idx;

    __device__ __forceinline__ bool found() const { return nk >= F; }

    // the walk's entry point (the last interval is told apart inside step)
    template <bool kLast>
    __device__ __forceinline__ void step_k(const LifConst &C, int m, float w) { step(C, m, w); }

    __device__ void step(const LifConst &C, int m, float w) {
        if (nk >= F) return;
        Id += static_cast<double>(w);
        const bool last = (m == C.M);
        const float len = last ? C.last_len : C.dt;
        const double Tm = fma(static_cast<double>(m), static_cast<double>(C.dt), static_cast<double>(C.t0));
        double u0 = 0.0, Vs = Vd, Is = Id;
        bool reset = false;
        while (nk < F) {
            const float seglen = static_cast<float>(static_cast<double>(len) - u0);
            // end value of the segment (not used on the last interval) and its
            // filter constants; after a reset the segment is shorter than the
            // interval, whose max K still bounds it
            double vn;
            float r_lo;
            if (!reset) {
                vn = fma(Vd, C.alpha_d, Id * C.k_dt_d);
                r_lo = last ? C.r_lo_last : C.r_lo_dt;
            } else {
                vn = last ? 0.0 : Is * kern_d64(C, static_cast<double>(len) - u0);
                r_lo = (C.kind == kGeneral && isfinite(seglen)) ? expf(-C.kappa * seglen) : 0.f;
            }
            const double kmax = last ? C.kmax_last_d : C.kmax_dt_d;
            Seg sf;
            float hi = 0.f, fhi = 0.f;
            if (!(seglen > 0.f) ||
                !seg_test<KS>(C, Vs, Is, vn, last, seglen, kmax, r_lo, sf, hi, fhi))
                break;
            float u, sl;
            seg_solve<KS>(C, sf, hi, fhi, u, sl);
            const double Ik = Is * exp(-static_cast<double>(u) * static_cast<double>(C.inv_ti));
            if (ok) {
                t_out[so + nk] = static_cast<float>(Tm + u0 + static_cast<double>(u));
                slope[so + nk] = sl;
                q_idx[so + nk] = m;
                cur[so + nk] = static_cast<float>(Ik);
            }
            ++nk;
            u0 += static_cast<double>(u);
            Vs = 0.0;
            Is = Ik;
            reset = true;
        }
        if (!reset) {
            Vd = fma(Vd, C.alpha_d, Id * C.k_dt_d);
            Id *= C.beta_d;
        } else if (!last) {
            const double rest = static_cast<double>(C.dt) - u0;
            Vd = Is * kern_d64(C, rest);
            Id = Is * exp(-rest * static_cast<double>(C.inv_ti));
        }
    }

    // slots after the last spike
    __device__ void finish() {
        if (!ok) return;
        for (int k = nk; k < F; ++k) {
            t_out[so + k] = INFINITY;
            slope[so + k] = 0.f;
            q_idx[so + k] = -1;
            cur[so + k] = 0.f;
        }
    }
};

// Multi-spike outputs of the row-parallel forward: a record is an input
// spike j_in * F_in + f, whose weight row is its index divided by F_in
// (multiplication by magic = ceil(2^40 / F_in), exact for indices below
// 2^40 / F_in); the scan is the one with reset above, and runs until every
// neuron of the tile holds F spikes or the grid ends.
struct RowOutMs {
    float *t_out, *slope, *cur;
    int *q_idx;
    int F;
    uint64_t magic;

    __device__ __forceinline__ int wrow(int j) const {
        return j > 0 ? static_cast<int>((static_cast<uint64_t>(j) * magic) >> 40) : 0;
    }

    template <int KS>
    __device__ __forceinline__ void scan(const LifConst &C, int N_out, int b, int i, bool row_ok,
                                         const float *tp, int kPt, int /* m_end: resets need every point */) const {
        MsScan<KS> sc;
        sc.F = F;
        sc.ok = row_ok;
        sc.so = (static_cast<int64_t>(b) * N_out + (row_ok ? i : 0)) * F;
        sc.t_out = t_out;
        sc.slope = slope;
        sc.cur = cur;
        sc.q_idx = q_idx;
        float wn = tp[0];  // next grid point's sum, read ahead
        for (int m = 0; m <= C.M; ++m) {
            const float wc = wn;
            if (m < C.M) wn = tp[(m + 1) * kPt];
            sc.step(C, m, wc);
            if (__all(sc.found() || !row_ok)) break;
        }
        sc.finish();
    }
};

// One sample per wave, one neuron per lane: the sample's input spikes,
// sorted by event row, are walked as in the TTFS forward (records are input
// spikes, so a record's weight row is its index / F_in) into the scan with
// reset. The wave stops once every lane holds F_out spikes.
template <typename WT, int KS>
__global__ __launch_bounds__(256) void ms_fwd_kernel(LifConst C, int B, int N_in, int F_in,
                                                     int N_out, int F_out,
                                                     const WT *__restrict__ Wt, SortedEv srt,
                                                     const int *__restrict__ n_valid,
                                                     float *__restrict__ t_out,
                                                     float *__restrict__ slope,
                                                     int *__restrict__ q_idx,
                                                     float *__restrict__ cur) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int waves = blockDim.x >> 6;
    const int i = blockIdx.x * kWave + lane;
    const bool row_ok = i < N_out;
    const int b = uniform(blockIdx.y * waves + wave);
    if (b >= B) return;  // wave-uniform; the kernel has no block barrier
    const int n = *as_const(n_valid + b);
    MsScan<KS> sc;
    sc.F = F_out;
    sc.ok = row_ok;
    sc.so = (static_cast<int64_t>(b) * N_out + (row_ok ? i : 0)) * F_out;
    sc.t_out = t_out;
    sc.slope = slope;
    sc.cur = cur;
    sc.q_idx = q_idx;
    walk_sorted_rows<WT, true>(C, N_in, N_out, Wt, srt, b, n, i, row_ok, F_in, sc);
    sc.finish();
}

// grad_W[i][j] = sum_b sum_f (G[b][m][i] L + G[b][m+1][i] R) over the events
// (m = row - 1) of input spike (b, j, f): lanes over neurons i, one wave per
// input j; G rows [b][m][:] are coalesced, the events uniform.
__global__ __launch_bounds__(kMsWaves * kWave) void ms_dw_kernel(LifConst C, int B, int N_in,
                                                                 int F_in, int N_out, MsEvents ev,
                                                                 const float *__restrict__ G,
                                                                 float *__restrict__ grad_W) {
    const int lane = threadIdx.x & (kWave - 1);
    const int j = blockIdx.y * kMsWaves + uniform(threadIdx.x >> 6);
    const int i = blockIdx.x * kWave + lane;
    if (j >= N_in) return;  // wave-uniform; no block barrier in this kernel
    const int R = C.M + 1;
    const int ic = i < N_out ? i : 0;
    float a = 0.f;
    for (int b = 0; b < B; ++b) {
        const int64_t eo = (static_cast<int64_t>(b) * N_in + j) * F_in;
        const float *Gb = G + static_cast<int64_t>(b) * R * N_out + ic;
        for (int f = 0; f < F_in; ++f) {
            const int row = *as_const(ev.row + eo + f);
            if (row < 0) continue;
            const int m = row - 1;  // L at grid point m, R at m + 1
            if (m >= 0) a = fmaf(Gb[static_cast<int64_t>(m) * N_out], *as_const(ev.L + eo + f), a);
            if (m + 1 <= C.M) a = fmaf(Gb[static_cast<int64_t>(m + 1) * N_out], *as_const(ev.R + eo + f), a);
        }
    }
    if (i < N_out) grad_W[static_cast<int64_t>(i) * N_in + j] = a;
}

// grad_t_in[b][j][f] = sum_i w_ij (G[b][m][i] dL + G[b][m+1][i] dR): one wave
// per (b, j) summing over neurons (lanes) with row j of W^T, then across the
// wave.
// dW for M <= kMsDwMaxM. A block takes one 64-neuron tile (lane = neuron i)
// and 64 inputs (kMsDwIn per wave) over a contiguous share of the batch. Per
// sample the tile G[b][0..M][tile] is staged in LDS (the next sample's tile
// is loaded into registers meanwhile), and each wave adds, input by input,
// G[m][i] L + G[m+1][i] R for the events of its inputs' spikes, whose fields
// are uniform (scalar loads, a whole spike index f for all kMsDwIn inputs at
// once). G is read from memory once per (block, sample) instead of once per
// (input, sample). Output: out[split][i][j], summed over splits in order
// (or grad_W itself with one split).
constexpr int kMsDwIn = 16;
constexpr int kMsDwPre = ((kMsDwMaxM + 1) * kWave + kMsWaves * kWave - 1) / (kMsWaves * kWave);

__global__ __launch_bounds__(kMsWaves * kWave) void ms_dw_tiled_kernel(
    LifConst C, int B, int N_in, int F_in, int N_out, int b_per, MsEvents ev,
    const float *__restrict__ G, float *__restrict__ out) {
    extern __shared__ float gs[];  // [2][M + 1][64]
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int R = C.M + 1;
    const int n_el = R * kWave;
    const int i0 = blockIdx.x * kWave;
    const int j0 = (blockIdx.y * kMsWaves + wave) * kMsDwIn;
    const int b0 = blockIdx.z * b_per;
    const int b1 = min(B, b0 + b_per);
    float pre[kMsDwPre];
    // thread t holds elements e = t + 256 k of the tile: row e / 64, column e % 64
    auto fetch = [&](int b) {
        const float *Gb = G + static_cast<int64_t>(b) * R * N_out;
#pragma unroll
        for (int k = 0; k < kMsDwPre; ++k) {
            const int e = threadIdx.x + k * kMsWaves * kWave;
            const int ii = i0 + (e & (kWave - 1));
            pre[k] = (e < n_el && ii < N_out) ? Gb[static_cast<int64_t>(e >> 6) * N_out + ii] : 0.f;
        }
    };
    auto stage = [&](float *dst) {
#pragma unroll
        for (int k = 0; k < kMsDwPre; ++k) {
            const int e = threadIdx.x + k * kMsWaves * kWave;
            if (e < n_el) dst[e] = pre[k];
        }
    };
    float acc[kMsDwIn];
#pragma unroll
    for (int k = 0; k < kMsDwIn; ++k) acc[k] = 0.f;
    const int jl = N_in - 1;
    if (b0 < b1) {
        fetch(b0);
        stage(gs);
    }
    __syncthreads();
    for (int b = b0; b < b1; ++b) {
        const int cb = (b - b0) & 1;
        if (b + 1 < b1) fetch(b + 1);
        const float *gb = gs + cb * n_el + lane;
        for (int f = 0; f < F_in; ++f) {
            int rw[kMsDwIn];
            float lv[kMsDwIn], rv[kMsDwIn];
#pragma unroll
            for (int k = 0; k < kMsDwIn; ++k) {
                const int64_t eo = (static_cast<int64_t>(b) * N_in + min(j0 + k, jl)) * F_in + f;
                rw[k] = (j0 + k <= jl) ? *as_const(ev.row + eo) : -1;
                lv[k] = *as_const(ev.L + eo);
                rv[k] = *as_const(ev.R + eo);
            }
#pragma unroll
            for (int k = 0; k < kMsDwIn; ++k) {
                const int m = rw[k] - 1;  // L at grid point m, R at m + 1
                if (rw[k] >= 0) {
                    if (m >= 0 && m <= C.M) acc[k] = fmaf(gb[m * kWave], lv[k], acc[k]);
                    if (m + 1 <= C.M) acc[k] = fmaf(gb[(m + 1) * kWave], rv[k], acc[k]);
                }
            }
        }
        if (b + 1 < b1) stage(gs + (cb ^ 1) * n_el);
        __syncthreads();
    }
    const int i = i0 + lane;
    if (i < N_out) {
        float *o = out + (static_cast<int64_t>(blockIdx.z) * N_out + i) * N_in;
#pragma unroll
        for (int k = 0; k < kMsDwIn; ++k)
            if (j0 + k <= jl) o[j0 + k] = acc[k];
    }
}

// out[k] = sum over s of part[s][k], in split order
__global__ __launch_bounds__(256) void ms_dw_reduce_kernel(int64_t n, int S,
                                                           const float *__restrict__ part,
                                                           float *__restrict__ out) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (k >= n) return;
    float a = part[k];
    for (int s = 1; s < S; ++s) a += part[s * n + k];
    out[k] = a;
}

template <typename WT>
__global__ __launch_bounds__(kMsWaves * kWave) void ms_dtin_kernel(LifConst C, int B, int N_in,
                                                                   int F_in, int N_out, MsEvents ev,
                                                                   const WT *__restrict__ Wt,
                                                                   const float *__restrict__ G,
                                                                   float *__restrict__ grad_t_in) {
    const int lane = threadIdx.x & (kWave - 1);
    const int j = blockIdx.x * kMsWaves + uniform(threadIdx.x >> 6);
    const int b = blockIdx.y;
    if (j >= N_in) return;  // wave-uniform
    const int R = C.M + 1;
    const int64_t eo = (static_cast<int64_t>(b) * N_in + j) * F_in;
    const float *Gb = G + static_cast<int64_t>(b) * R * N_out;
    const WT *wr = Wt + static_cast<int64_t>(j) * N_out;
    for (int f = 0; f < F_in; ++f) {
        const int row = *as_const(ev.row + eo + f);
        float a = 0.f;
        if (row >= 0) {
            const int m = row - 1;
            const float dl = (m >= 0) ? *as_const(ev.dL + eo + f) : 0.f;
            const float dr = (m + 1 <= C.M) ? *as_const(ev.dR + eo + f) : 0.f;
            const int64_t ml = static_cast<int64_t>(m >= 0 ? m : 0) * N_out;
            const int64_t mr = static_cast<int64_t>(m + 1 <= C.M ? m + 1 : C.M) * N_out;
            for (int i = lane; i < N_out; i += kWave) {
                const float w = WLoad<WT>::get(wr, i);
                a = fmaf(w, fmaf(Gb[ml + i], dl, Gb[mr + i] * dr), a);
            }
        }
        for (int s = kWave / 2; s > 0; s >>= 1) a += __shfl_xor(a, s);
        if (lane == 0) grad_t_in[eo + f] = a;
    }
}

unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

template <int KS>
hipError_t prep(const LifConst &C, int64_t n_spk, int N_in, int N_out, const float *t_in,
                MsEvents ev, const void *W, bool bf16, void *Wt, bool transpose, MsGrad gr,
                hipStream_t st) {
    const int n_ev = static_cast<int>(cdiv(n_spk, kMsPrepThreads));
    const int n_tr = (transpose && static_cast<int64_t>(N_in) * N_out > 0)
                         ? static_cast<int>(cdiv(N_in, 32) * cdiv(N_out, 32)) : 0;
    const int n_g = static_cast<int>(cdiv(gr.n, kMsPrepThreads));
    const unsigned blocks = static_cast<unsigned>(n_ev + n_tr + n_g);
    if (blocks == 0) return hipSuccess;
    if (bf16)
        hipLaunchKernelGGL((ms_prep_kernel<uint16_t, KS>), dim3(blocks), dim3(kMsPrepThreads), 0, st,
                           C, n_spk, n_ev, n_tr, N_in, N_out, t_in, ev,
                           static_cast<const uint16_t *>(W), static_cast<uint16_t *>(Wt), gr);
    else
        hipLaunchKernelGGL((ms_prep_kernel<float, KS>), dim3(blocks), dim3(kMsPrepThreads), 0, st,
                           C, n_spk, n_ev, n_tr, N_in, N_out, t_in, ev,
                           static_cast<const float *>(W), static_cast<float *>(Wt), gr);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_ms_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t F_in,
                             int64_t N_out, int64_t F_out, const void *W, bool bf16, void *Wt,
                             SortedEv srt, int *n_valid, const float *t_in, float *t_out,
                             float *slope, int *q_idx, float *cur, hipStream_t st) {
    hipError_t e = launch_sort_records(C, B, N_in * F_in, t_in, srt, n_valid, "ms_sort", st);
    if (e != hipSuccess) return e;
    {
        ProfScope prof("ms_transpose", st);
        MsEvents none_ev{};
        e = prep<kAnyKind>(C, 0, static_cast<int>(N_in), static_cast<int>(N_out), t_in, none_ev,
                           W, bf16, Wt, true, MsGrad{}, st);
        if (e != hipSuccess) return e;
    }
    ProfScope prof("ms_fwd", st);
    if (B == 0 || N_out == 0) return hipSuccess;
    const bool gen = C.kind == kGeneral;
    if (C.M <= kRowsMaxM) {
        // row-parallel: four waves sum a sample's spikes, one scan per tile
        const int R = C.M + 3;
        const int nt = rows_nt(N_out, R);
        dim3 grid(cdiv(cdiv(N_out, kWave), nt), static_cast<unsigned>(B));
        const size_t lds = rows_lds(nt, R);
        const bool vec = (N_out % nt) == 0;
        const uint64_t magic = ((uint64_t{1} << 40) + static_cast<uint64_t>(F_in) - 1) /
                               static_cast<uint64_t>(F_in);
        const RowOutMs out{t_out, slope, cur, q_idx, static_cast<int>(F_out), magic};
#define MSR_KV(WTY, NTV, KSV, VECV)                                                              \
    hipLaunchKernelGGL((fwd_rows_kernel<WTY, NTV, KSV, VECV, RowOutMs>), grid,                   \
                       dim3(kRowWaves * kWave), lds, st, C, static_cast<int>(N_in),              \
                       static_cast<int>(N_out), static_cast<const WTY *>(Wt), srt, out)
#define MSR_K(WTY, NTV, KSV)                  \
    do {                                      \
        if (vec) MSR_KV(WTY, NTV, KSV, true); \
        else MSR_KV(WTY, NTV, KSV, false);    \
    } while (0)
#define MSR(WTY, NTV)                                        \
    do {                                                     \
        if (gen) MSR_K(WTY, NTV, kGeneral);                  \
        else MSR_K(WTY, NTV, kAnyKind);                      \
    } while (0)
        if (bf16) {
            if (nt == 4) MSR(uint16_t, 4);
            else if (nt == 2) MSR(uint16_t, 2);
            else MSR(uint16_t, 1);
        } else {
            if (nt == 4) MSR(float, 4);
            else if (nt == 2) MSR(float, 2);
            else MSR(float, 1);
        }
#undef MSR
#undef MSR_K
#undef MSR_KV
        return hipGetLastError();
    }
    constexpr int waves = 4;
    dim3 grid(cdiv(N_out, kWave), cdiv(B, waves));
#define MSF(WTY, KSV)                                                                          \
    hipLaunchKernelGGL((ms_fwd_kernel<WTY, KSV>), grid, dim3(waves * kWave), 0, st, C,          \
                       static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(F_in),    \
                       static_cast<int>(N_out), static_cast<int>(F_out),                       \
                       static_cast<const WTY *>(Wt), srt, n_valid, t_out, slope, q_idx, cur)
    if (bf16) {
        if (gen) MSF(uint16_t, kGeneral); else MSF(uint16_t, kAnyKind);
    } else {
        if (gen) MSF(float, kGeneral); else MSF(float, kAnyKind);
    }
#undef MSF
    return hipGetLastError();
}

hipError_t launch_ms_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t F_in,
                              int64_t N_out, int64_t F_out, const void *W, bool bf16, void *Wt,
                              MsEvents ev, const float *t_in, const float *t_out,
                              const float *slope, const int *q_idx, const float *cur,
                              const float *grad_t, float *G, float *dw_part, float *grad_W,
                              float *grad_t_in, hipStream_t st) {
    const int64_t n_spk = B * N_in * F_in;
    MsGrad gr{t_out, slope, q_idx, cur, grad_t, G, B * N_out, static_cast<int>(F_out)};
    {
        ProfScope prof("ms_bwd_prep", st);
        hipError_t e = (C.kind == kGeneral)
                           ? prep<kGeneral>(C, n_spk, static_cast<int>(N_in), static_cast<int>(N_out),
                                            t_in, ev, W, bf16, Wt, grad_t_in != nullptr, gr, st)
                           : prep<kAnyKind>(C, n_spk, static_cast<int>(N_in), static_cast<int>(N_out),
                                            t_in, ev, W, bf16, Wt, grad_t_in != nullptr, gr, st);
        if (e != hipSuccess) return e;
    }
    if (grad_W && N_in * N_out > 0) {
        ProfScope prof("ms_dw", st);
        const int S = ms_dw_splits(C.M, B, N_in, N_out);
        if (S > 0) {
            const int per = static_cast<int>(cdiv(B, S));
            float *dst = (S > 1) ? dw_part : grad_W;
            const size_t lds = 2 * static_cast<size_t>(C.M + 1) * kWave * sizeof(float);
            hipLaunchKernelGGL(ms_dw_tiled_kernel,
                               dim3(cdiv(N_out, kWave), cdiv(N_in, kMsWaves * kMsDwIn),
                                    static_cast<unsigned>(S)),
                               dim3(kMsWaves * kWave), lds, st, C, static_cast<int>(B),
                               static_cast<int>(N_in), static_cast<int>(F_in),
                               static_cast<int>(N_out), per, ev, G, dst);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            if (S > 1) {
                const int64_t n = N_in * N_out;
                hipLaunchKernelGGL(ms_dw_reduce_kernel, dim3(cdiv(n, 256)), dim3(256), 0, st, n, S,
                                   dw_part, grad_W);
                e = hipGetLastError();
                if (e != hipSuccess) return e;
            }
        } else {
            hipLaunchKernelGGL(ms_dw_kernel, dim3(cdiv(N_out, kWave), cdiv(N_in, kMsWaves)),
                               dim3(kMsWaves * kWave), 0, st, C, static_cast<int>(B),
                               static_cast<int>(N_in), static_cast<int>(F_in), static_cast<int>(N_out),
                               ev, G, grad_W);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    if (grad_t_in && B * N_in > 0) {
        ProfScope prof("ms_dtin", st);
        dim3 grid(cdiv(N_in, kMsWaves), static_cast<unsigned>(B));
        if (bf16)
            hipLaunchKernelGGL(ms_dtin_kernel<uint16_t>, grid, dim3(kMsWaves * kWave), 0, st, C,
                               static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(F_in),
                               static_cast<int>(N_out), ev, static_cast<const uint16_t *>(Wt), G,
                               grad_t_in);
        else
            hipLaunchKernelGGL(ms_dtin_kernel<float>, grid, dim3(kMsWaves * kWave), 0, st, C,
                               static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(F_in),
                               static_cast<int>(N_out), ev, static_cast<const float *>(Wt), G,
                               grad_t_in);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace dstd
