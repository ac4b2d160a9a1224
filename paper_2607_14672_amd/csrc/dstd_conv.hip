// dstd_conv.hip -- DSTD-LIF convolutional-layer kernels for gfx950.
//
// A conv layer is the dense layer of App. B.1 whose weight matrix is the
// convolution's shared, local connectivity: w^_{(c,p), m} sums w_ij s_jm over
// the receptive field of position p. Event pooling (2x2 or global) averages
// the input events before the convolution; being linear, it is folded into
// the weights (W / P) with every raw input of a pooled cell kept as its own
// event source.
//
// Input ordering used by every kernel here ("cell-major"): the (pooled) map
// has Hp x Wp cells, each with PC = P * C_in raw inputs j' = d * C_in + ci
// (d = raw pixel inside the cell). Index ((b * Hp + py) * Wp + px) * PC + j'.
//
// The inputs of one cell row (b, py) that have events are bucketed by (event
// row r, cell column px) -- a counting sort, stable in j' -- so the records
// of row r under the KW cells of an output position's kernel row form ONE
// contiguous segment. Both the forward and the dt_in backward walk, per
// output position, the event rows in grid order and read KH segments per row.
//  - forward: lanes = output channels; row sums feed the interval scan as
//    rows close (the weighted events never exist in memory);
//  - dt_in: lanes = output channels carry G[m] = dL/dw^_m computed in place
//    from (gamma = -g/slope, t - T_q, q); every record gets the channel sum of
//    W (dL G[r-1] + dR G[r]) for the tap that joins it to this position, as
//    one partial per (record, tap), gathered in tap order afterwards.
// dW reduces over (b, position) samples with lanes = (tap, input channel),
// G again computed in place.
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"

#include <algorithm>

namespace dstd {

// raw pixel (y, x) of input j' = d * C_in + ci in cell (py, px)
__device__ __forceinline__ void raw_pixel(const ConvGeom &g, int py, int px, int d, int &y,
                                          int &x) {
    if (g.pool == 2) {
        y = 2 * py + (d >> 1);
        x = 2 * px + (d & 1);
    } else if (g.pool == 0) {
        y = d / g.W;
        x = d % g.W;
    } else {
        y = py;
        x = px;
    }
}

__device__ __forceinline__ int64_t nchw_index(const ConvGeom &g, int b, int ci, int y, int x) {
    return ((static_cast<int64_t>(b) * g.C_in + ci) * g.H + y) * g.W + x;
}

// ------------------------------------------------------------ cell sort --
// One block per cell row (b, py); wave w handles cells px = w, w + 4, ...
// LDS: hist[r][px] (later the next free slot of bucket (r, px)), then the
// per-thread partial sums of the prefix scan.
__global__ __launch_bounds__(256) void conv_sort_kernel(LifConst C, ConvGeom g,
                                                        const float *__restrict__ t_in,
                                                        ConvSorted cs) {
    extern __shared__ int sh[];
    const int R = rows_of(C);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int nw = blockDim.x >> 6;
    const int cr = blockIdx.x;  // b * Hp + py
    const int b = cr / g.Hp, py = cr % g.Hp;
    const int nb = R * g.Wp;  // buckets, flat f = r * Wp + px
    const bool bwd = cs.P != nullptr;
    const int KT = g.KH * g.KW;
    int *hist = sh;
    int *part = sh + nb;
    for (int k = threadIdx.x; k < nb; k += blockDim.x) hist[k] = 0;
    __syncthreads();
    for (int px = wave; px < g.Wp; px += nw) {
        for (int j0 = 0; j0 < g.PC; j0 += kWave) {
            const int j = j0 + lane;
            if (j < g.PC) {
                int y, x;
                raw_pixel(g, py, px, j / g.C_in, y, x);
                const int r = bin_row(C, t_in[nchw_index(g, b, j % g.C_in, y, x)]);
                if (r >= 0) atomicAdd(&hist[r * g.Wp + px], 1);
            }
        }
    }
    __syncthreads();
    // exclusive prefix over the buckets in (r, px) order
    const int chunk = (nb + blockDim.x - 1) / blockDim.x;
    const int lo = min(nb, static_cast<int>(threadIdx.x) * chunk), hi = min(nb, lo + chunk);
    int s = 0;
    for (int f = lo; f < hi; ++f) s += hist[f];
    part[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int t = 0; t < static_cast<int>(blockDim.x); ++t) {
            const int v = part[t];
            part[t] = run;
            run += v;
        }
        cs.off[static_cast<int64_t>(cr) * (nb + 1) + nb] = run;
    }
    __syncthreads();
    int run = part[threadIdx.x];
    int *off = cs.off + static_cast<int64_t>(cr) * (nb + 1);
    for (int f = lo; f < hi; ++f) {
        const int v = hist[f];
        off[f] = run;
        hist[f] = run;
        run += v;
    }
    __syncthreads();
    // placement: lanes with the same row are ranked by lane (j' ascending)
    const int64_t rb = static_cast<int64_t>(cr) * g.Wp * g.PC;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int px = wave; px < g.Wp; px += nw) {
        for (int j0 = 0; j0 < g.PC; j0 += kWave) {
            const int j = j0 + lane;
            Event e{-1, 0.f, 0.f, 0.f, 0.f};
            if (j < g.PC) {
                int y, x;
                raw_pixel(g, py, px, j / g.C_in, y, x);
                e = bin_event(C, t_in[nchw_index(g, b, j % g.C_in, y, x)]);
            }
            const int r = e.row;
            int pos = 0;
            uint64_t todo = __ballot(r >= 0);
            while (todo) {
                const int lead = __ffsll(static_cast<unsigned long long>(todo)) - 1;
                const int rl = __builtin_amdgcn_readlane(r, lead);
                const uint64_t same = __ballot(r == rl);
                int *slot = &hist[rl * g.Wp + px];
                const int base = *slot;
                if (r == rl) pos = base + __popcll(same & below);
                __builtin_amdgcn_wave_barrier();
                if (lane == lead) *slot = base + __popcll(same);
                __builtin_amdgcn_wave_barrier();
                todo &= ~same;
            }
            if (r >= 0) {
                const int64_t o = rb + pos;
                cs.key[o] = px * g.C_in + (j % g.C_in);
                cs.L[o] = bwd ? e.dL : e.L;
                cs.R[o] = bwd ? e.dR : e.R;
                if (bwd) {
                    cs.px[o] = px;
                    cs.src[o] = px * g.PC + j;
                    for (int k = 0; k < KT; ++k) cs.P[o * KT + k] = 0.f;
                }
            }
        }
    }
}

// ------------------------------------------------------ weight layout ----
// WT[(k * C_in + ci) * C_out + co] = W[co, ci, k] / P (k = ky*KW + kx).
template <typename WT>
__global__ __launch_bounds__(256) void conv_weights_kernel(ConvGeom g, const WT *__restrict__ W,
                                                           float *__restrict__ out) {
    const int KT = g.KH * g.KW;
    const int64_t n = static_cast<int64_t>(KT) * g.C_in * g.C_out;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    const int co = static_cast<int>(t % g.C_out);
    const int64_t u = t / g.C_out;
    const int ci = static_cast<int>(u % g.C_in);
    const int k = static_cast<int>(u / g.C_in);
    const float w = WLoad<WT>::get(W, (static_cast<int64_t>(co) * g.C_in + ci) * KT + k);
    out[t] = w * g.inv_P;
}

// ------------------------------------------------------ position walk ----
// The records an output position (b, oy, ox) reads: for event row r and
// kernel row ky, the segment [off[r][xa], off[r][xb]) of cell row
// py = oy*stride - pad + ky; a record's key px*C_in + ci plus the segment
// constant (ky*KW - x0)*C_in is its row in WT. The bucket starts of the KH
// cell rows are held one event row per lane (64 rows at a time).
constexpr int kCBatch = 8;

template <int KHT>
struct PosWalk {
    int b, pos, x0, xa, xb, nb1, wlim;
    int64_t recb[KHT], offb[KHT];
    int wofs[KHT];
    bool vky[KHT];
    int oa[KHT], ob[KHT];

    // returns the number of records in the KH cell rows (0: nothing to read)
    __device__ __forceinline__ int init(const LifConst &C, const ConvGeom &g, const ConvSorted &cs,
                                        int64_t p) {
        const int HoWo = g.Ho * g.Wo;
        b = uniform(static_cast<int>(p / HoWo));
        pos = uniform(static_cast<int>(p % HoWo));
        const int oy = pos / g.Wo, ox = pos % g.Wo;
        x0 = ox * g.stride - g.pad;
        xa = max(0, x0);
        xb = max(xa, min(g.Wp, x0 + g.KW));
        nb1 = rows_of(C) * g.Wp + 1;
        wlim = g.KH * g.KW * g.C_in - 1;
        int any = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int py = oy * g.stride - g.pad + ky;
            vky[ky] = ky < g.KH && py >= 0 && py < g.Hp && xa < xb;
            const int64_t cr = static_cast<int64_t>(b) * g.Hp + (vky[ky] ? py : 0);
            recb[ky] = cr * g.Wp * g.PC;
            offb[ky] = cr * nb1;
            wofs[ky] = (ky * g.KW - x0) * g.C_in;
            if (vky[ky]) any += *as_const(cs.off + offb[ky] + nb1 - 1);
        }
        return any;
    }

    __device__ __forceinline__ void load_offs(const ConvGeom &g, const ConvSorted &cs, int R,
                                              int r0, int lane) {
        const int r = min(r0 + lane, R - 1);
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int *o = cs.off + offb[ky] + static_cast<int64_t>(r) * g.Wp;
            oa[ky] = vky[ky] ? o[xa] : 0;
            ob[ky] = vky[ky] ? o[xb] : 0;
        }
    }

    // segment starts and lengths of event row r (load_offs of its 64-row
    // chunk done); returns the total length
    __device__ __forceinline__ int segments(int r, int *s0, int *n0) const {
        const int l = r & (kWave - 1);
        int n = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            s0[ky] = __builtin_amdgcn_readlane(oa[ky], l);
            n0[ky] = __builtin_amdgcn_readlane(ob[ky], l) - s0[ky];
            n += n0[ky];
        }
        return n;
    }

    // byte offset of a record's weight row; stale keys read past a segment
    // end are clamped so the scalar offset always stays inside WT
    __device__ __forceinline__ int wrow(int key, int ky, int rstride) const {
        return min(max(key + wofs[ky], 0), wlim) * rstride;
    }
};

// -------------------------------------------------------------- forward --
// Wave = one output position, lane = output channel of a 64-wide tile.
template <int KHT>
__global__ __launch_bounds__(256) void conv_fwd_kernel(LifConst C, ConvGeom g, int64_t n_pos,
                                                       const float *__restrict__ Wt,
                                                       ConvSorted cs, float *__restrict__ t_out,
                                                       float *__restrict__ slope,
                                                       int *__restrict__ q_idx) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int64_t p = static_cast<int64_t>(blockIdx.x) * (blockDim.x >> 6) + wave;
    if (p >= n_pos) return;  // wave-uniform; no block barrier below
    const int co = blockIdx.y * kWave + lane;
    const bool row_ok = co < g.C_out;
    const int HoWo = g.Ho * g.Wo;
    const int R = rows_of(C);
    PosWalk<KHT> wk;
    const int any = wk.init(C, g, cs, p);
    const int64_t o_out = (static_cast<int64_t>(wk.b) * g.C_out + co) * HoWo + wk.pos;
    if (any == 0) {  // no events in the receptive field: silent
        if (row_ok) {
            t_out[o_out] = INFINITY;
            slope[o_out] = 0.f;
            q_idx[o_out] = -1;
        }
        return;
    }
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(
        Wt, static_cast<uint32_t>(static_cast<int64_t>(wk.wlim + 1) * g.C_out * sizeof(float)));
    const int voff = (row_ok ? co : 0) * static_cast<int>(sizeof(float));
    const int rstride = g.C_out * static_cast<int>(sizeof(float));
    Scan sc;
    float aL = 0.f, aR = 0.f, carry = 0.f;
    for (int r = 0; r <= R - 2; ++r) {
        if ((r & (kWave - 1)) == 0) wk.load_offs(g, cs, R, r, lane);
        int s0[KHT], n0[KHT];
        if (wk.segments(r, s0, n0) > 0) {
            // first batch of every kernel row issued together
            float w[KHT][kCBatch], lv[KHT][kCBatch], rv[KHT][kCBatch];
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                const int64_t o = wk.recb[ky] + s0[ky];
#pragma unroll
                for (int kk = 0; kk < kCBatch; ++kk) {
                    w[ky][kk] = BufLoad<float>::get(wr, voff,
                                                    wk.wrow(as_const(cs.key + o)[kk], ky, rstride));
                    lv[ky][kk] = as_const(cs.L + o)[kk];
                    rv[ky][kk] = as_const(cs.R + o)[kk];
                }
            }
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
#pragma unroll
                for (int kk = 0; kk < kCBatch; ++kk) {
                    if (kk < n0[ky]) {
                        aL = fmaf(w[ky][kk], lv[ky][kk], aL);
                        aR = fmaf(w[ky][kk], rv[ky][kk], aR);
                    }
                }
            }
            // long segments: further batches
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                for (int k0 = kCBatch; k0 < n0[ky]; k0 += kCBatch) {
                    const int64_t o = wk.recb[ky] + s0[ky] + k0;
                    const int nk = n0[ky] - k0;
                    float wb[kCBatch], lb[kCBatch], rb[kCBatch];
#pragma unroll
                    for (int kk = 0; kk < kCBatch; ++kk) {
                        wb[kk] = BufLoad<float>::get(wr, voff,
                                                     wk.wrow(as_const(cs.key + o)[kk], ky, rstride));
                        lb[kk] = as_const(cs.L + o)[kk];
                        rb[kk] = as_const(cs.R + o)[kk];
                    }
#pragma unroll
                    for (int kk = 0; kk < kCBatch; ++kk) {
                        if (kk < nk) {
                            aL = fmaf(wb[kk], lb[kk], aL);
                            aR = fmaf(wb[kk], rb[kk], aR);
                        }
                    }
                }
            }
        }
        // row r closes: grid point m = r - 1 gets its L sums plus the
        // previous row's R sums
        if (r >= 1) sc.step(C, r - 1, aL + carry);
        carry = aR;
        aL = 0.f;
        aR = 0.f;
        if (__all(sc.found() || !row_ok)) break;
    }
    if (!row_ok) return;
    float to, sl;
    int q;
    sc.finish(C, to, sl, q);
    t_out[o_out] = to;
    slope[o_out] = sl;
    q_idx[o_out] = q;
}

// --------------------------------------------------------- backward ------
// Events of every input in cell-major order (row -1 = no events) for the dW
// reduction; dt_in starts at zero (inputs with events are overwritten later).
__global__ __launch_bounds__(256) void conv_events_kernel(LifConst C, ConvGeom g, int64_t n,
                                                          const float *__restrict__ t_in,
                                                          int *__restrict__ ev_row,
                                                          float *__restrict__ ev_L,
                                                          float *__restrict__ ev_R,
                                                          float *__restrict__ dt_in) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const int j = static_cast<int>(k % g.PC);
    const int64_t cell = k / g.PC;
    const int px = static_cast<int>(cell % g.Wp);
    const int64_t u = cell / g.Wp;
    const int py = static_cast<int>(u % g.Hp);
    const int b = static_cast<int>(u / g.Hp);
    int y, x;
    raw_pixel(g, py, px, j / g.C_in, y, x);
    const int64_t src = nchw_index(g, b, j % g.C_in, y, x);
    const Event e = bin_event(C, t_in[src]);
    ev_row[k] = e.row;
    ev_L[k] = e.L;
    ev_R[k] = e.R;
    if (dt_in) dt_in[src] = 0.f;
}

// Per output neuron (b, co, p) -> position-major [b][p][co]: the gradient
// triple (gamma, t - T_q, q) of grad_prep.
__global__ __launch_bounds__(256) void conv_grad_prep_kernel(LifConst C, ConvGeom g, int64_t n,
                                                             const float *__restrict__ t_out,
                                                             const float *__restrict__ slope,
                                                             const int *__restrict__ q_idx,
                                                             const float *__restrict__ grad_t,
                                                             float *__restrict__ gam,
                                                             float *__restrict__ uq,
                                                             int *__restrict__ qv) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    const int HoWo = g.Ho * g.Wo;
    const int co = static_cast<int>(t % g.C_out);
    const int64_t u = t / g.C_out;
    const int p = static_cast<int>(u % HoWo);
    const int64_t b = u / HoWo;
    const int64_t o = (b * g.C_out + co) * HoWo + p;
    const int q = q_idx[o];
    GradPrep gp{0.f, 0.f, -1};
    if (q >= 0) {  // silent neurons: no further loads
        const float g = grad_t[o];
        if (g != 0.f) gp = grad_prep(C, t_out[o], slope[o], q, g);
    }
    gam[t] = gp.gam;
    uq[t] = gp.uq;
    qv[t] = gp.q;
}

// live[s] = 1 if any channel at sample s = (b, p) passes gradient.
__global__ __launch_bounds__(256) void conv_live_kernel(int64_t n_samp, int C_out,
                                                        const int *__restrict__ qv,
                                                        int *__restrict__ live) {
    const int64_t s = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n_samp) return;
    const int *q = qv + s * C_out;
    int f = 0;
    for (int c = 0; c < C_out; ++c) f |= (q[c] >= 0) ? 1 : 0;
    live[s] = f;
}

// dt_in partials. Wave = output position; lane = output channel, NT tiles of
// 64 per lane. Rows stop after the last grid point any channel's G reaches.
template <int KHT, int NT>
__global__ __launch_bounds__(256) void conv_dtp_kernel(LifConst C, ConvGeom g, int64_t n_pos,
                                                       const float *__restrict__ Wt,
                                                       ConvSorted cs,
                                                       const float *__restrict__ gam,
                                                       const float *__restrict__ uq,
                                                       const int *__restrict__ qv) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int64_t p = static_cast<int64_t>(blockIdx.x) * (blockDim.x >> 6) + wave;
    if (p >= n_pos) return;  // wave-uniform; no block barrier below
    const int R = rows_of(C);
    const int KT = g.KH * g.KW;
    PosWalk<KHT> wk;
    if (wk.init(C, g, cs, p) == 0) return;  // no records to receive gradient
    const int64_t nbase = (static_cast<int64_t>(wk.b) * g.Ho * g.Wo + wk.pos) * g.C_out;
    float gm[NT], ua[NT], gA[NT], gB[NT];
    int qa[NT], voff[NT];
    int qmax = -1;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int co = t * kWave + lane;
        const int cc = min(co, g.C_out - 1);
        const bool ok = co < g.C_out;
        gm[t] = ok ? gam[nbase + cc] : 0.f;
        ua[t] = ok ? uq[nbase + cc] : 0.f;
        qa[t] = ok ? qv[nbase + cc] : -1;
        qmax = max(qmax, qa[t]);
        voff[t] = cc * static_cast<int>(sizeof(float));
    }
#pragma unroll
    for (int m = kWave / 2; m >= 1; m >>= 1) qmax = max(qmax, __shfl_xor(qmax, m));
    qmax = uniform(qmax);
    if (qmax < 0) return;  // no gradient reaches this position
    const int r_end = min(R - 2, qmax + 1);  // row r needs G[r-1], G[r]
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        gA[t] = 0.f;
        gB[t] = g_at(C, gm[t], ua[t], qa[t], 0);
    }
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(
        Wt, static_cast<uint32_t>(static_cast<int64_t>(wk.wlim + 1) * g.C_out * sizeof(float)));
    const int rstride = g.C_out * static_cast<int>(sizeof(float));
    for (int r = 0; r <= r_end; ++r) {
        if ((r & (kWave - 1)) == 0) wk.load_offs(g, cs, R, r, lane);
        int s0[KHT], n0[KHT];
        if (wk.segments(r, s0, n0) > 0) {
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                for (int k0 = 0; k0 < n0[ky]; k0 += kCBatch) {
                    const int64_t o = wk.recb[ky] + s0[ky] + k0;
                    const int nk = n0[ky] - k0;
                    float v[kCBatch];
#pragma unroll
                    for (int kk = 0; kk < kCBatch; ++kk) {
                        const int wo = wk.wrow(as_const(cs.key + o)[kk], ky, rstride);
                        const float dl = as_const(cs.L + o)[kk], dr = as_const(cs.R + o)[kk];
                        float acc = 0.f;
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const float w = BufLoad<float>::get(wr, voff[t], wo);
                            acc = fmaf(w, fmaf(dl, gA[t], dr * gB[t]), acc);
                        }
                        v[kk] = acc;
                    }
                    // channel sums (butterfly; every lane ends with the total)
#pragma unroll
                    for (int m = kWave / 2; m >= 1; m >>= 1) {
#pragma unroll
                        for (int kk = 0; kk < kCBatch; ++kk) v[kk] += __shfl_xor(v[kk], m);
                    }
                    // lane kk stores record kk's partial for its tap
                    float mine = 0.f;
                    int pxl = 0;
#pragma unroll
                    for (int kk = 0; kk < kCBatch; ++kk) {
                        const int pk = as_const(cs.px + o)[kk];
                        if (lane == kk) {
                            mine = v[kk];
                            pxl = pk;
                        }
                    }
                    if (lane < nk && lane < kCBatch)
                        cs.P[(o + lane) * KT + ky * g.KW + (pxl - wk.x0)] = mine;
                }
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            gA[t] = gB[t];
            gB[t] = g_at(C, gm[t], ua[t], qa[t], r + 1);
        }
    }
}

// dt_in of every input with events: the sum of its per-tap partials (taps
// that reach no output position stay 0), written to its NCHW slot.
__global__ __launch_bounds__(256) void conv_dt_gather_kernel(ConvGeom g, int R, int64_t n,
                                                             ConvSorted cs,
                                                             float *__restrict__ dt_in) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    const int64_t per = static_cast<int64_t>(g.Wp) * g.PC;
    const int64_t cr = t / per;
    const int slot = static_cast<int>(t % per);
    const int nb1 = R * g.Wp + 1;
    if (slot >= cs.off[cr * nb1 + nb1 - 1]) return;
    const int KT = g.KH * g.KW;
    float s = 0.f;
    for (int k = 0; k < KT; ++k) s += cs.P[t * KT + k];
    const int src = cs.src[t];
    const int px = src / g.PC, j = src % g.PC;
    const int py = static_cast<int>(cr % g.Hp), b = static_cast<int>(cr / g.Hp);
    int y, x;
    raw_pixel(g, py, px, j / g.C_in, y, x);
    dt_in[nchw_index(g, b, j % g.C_in, y, x)] = s;
}

// dW[co, ci, k] = (1/P) sum_{b, p} sum_d (G[b, r, p, co] L + G[b, r+1, p, co] R)
// over the raw inputs d of the cell that tap k of position p reads.
// Lane = (k, ci); a block covers 256 of them and a tile of TI channels whose
// sums stay in registers over its share of the (b, p) samples. G[b, :, p,
// tile] is computed in place from (gamma, t - T_q, q) -- each thread owns one
// channel and a fixed set of rows; channels without gradient cost no
// exponential -- and staged in LDS as (G[r], G[r+1]) pairs, double buffered,
// the next sample's values in registers (NPER per thread) during this one's
// sums. A sample whose tile is all zero is skipped.
template <int TI, int NPER>
__global__ __launch_bounds__(256) void conv_dw_kernel(LifConst C, ConvGeom g, int64_t n_samp,
                                                      int s_per_split, int pstride,
                                                      const float *__restrict__ gam,
                                                      const float *__restrict__ uq,
                                                      const int *__restrict__ qv,
                                                      const int *__restrict__ live_in,
                                                      const int *__restrict__ ev_row,
                                                      const float *__restrict__ ev_L,
                                                      const float *__restrict__ ev_R,
                                                      float *__restrict__ part) {
    extern __shared__ float2 ps[];  // [2][TI][pstride], then the live sample list
    __shared__ int n_live_w[4];
    const int R = rows_of(C);
    const int NJ = g.KH * g.KW * g.C_in;
    const int jj = blockIdx.x * blockDim.x + threadIdx.x;
    const int co0 = blockIdx.y * TI;
    const int ni = min(TI, g.C_out - co0);
    const int64_t s_lo = static_cast<int64_t>(blockIdx.z) * s_per_split;
    const int64_t s_hi = min(n_samp, s_lo + s_per_split);
    const bool j_ok = jj < NJ;
    const int k = (j_ok ? jj : 0) / g.C_in, ci = (j_ok ? jj : 0) % g.C_in;
    const int ky = k / g.KW, kx = k % g.KW;
    const int HoWo = g.Ho * g.Wo;
    float acc[TI];
#pragma unroll
    for (int ii = 0; ii < TI; ++ii) acc[ii] = 0.f;
    const int total = R * TI;
    // element c of this thread: row r = r_first + c * (256 / TI), channel l
    const int l_own = threadIdx.x % TI, r_first = threadIdx.x / TI;
    constexpr int kRowStep = 256 / TI;
    const GStep gst = g_step(C, kRowStep);
    float pre[NPER];
    // G[b, :, p, tile] of sample s; returns whether any value is nonzero
    auto fetch = [&](int64_t s) {
        const int64_t nb = s * g.C_out + co0 + min(l_own, ni - 1);
        const bool own = l_own < ni;
        const float gm = own ? gam[nb] : 0.f;
        const float u = own ? uq[nb] : 0.f;
        const int q = own ? qv[nb] : -1;
        g_strided<NPER>(C, gst, gm, u, q, r_first - 1, kRowStep, pre);
        bool nz = false;
#pragma unroll
        for (int c = 0; c < NPER; ++c) nz = nz || pre[c] != 0.f;
        return nz;
    };
    auto store = [&](float2 *buf) {
#pragma unroll
        for (int c = 0; c < NPER; ++c) {
            const int kk = threadIdx.x + c * 256;
            if (kk < total) {
                const int r = kk / TI, l = kk % TI;
                float2 *row = buf + l * pstride;
                if (r < R - 1) row[r].x = pre[c];
                if (r > 0) row[r - 1].y = pre[c];
            }
        }
        for (int l = threadIdx.x; l < TI; l += blockDim.x)
            buf[l * pstride + R - 1] = make_float2(0.f, 0.f);
    };
    // the split's samples through which any gradient flows, in order
    int *list = reinterpret_cast<int *>(ps + 2 * TI * pstride);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int n_live = 0;
    for (int64_t c0 = s_lo; c0 < s_hi; c0 += 256) {
        const int64_t sc = c0 + threadIdx.x;
        const bool f = sc < s_hi && live_in[sc] != 0;
        const uint64_t m = __ballot(f);
        if (lane == 0) n_live_w[wave] = __popcll(m);
        __syncthreads();
        int base = n_live;
        for (int w = 0; w < wave; ++w) base += n_live_w[w];
        if (f) list[base + __popcll(m & below)] = static_cast<int>(sc - s_lo);
        for (int w = 0; w < 4; ++w) n_live += n_live_w[w];
        __syncthreads();
    }
    bool live = false;  // the staged sample's tile has a nonzero value
    if (n_live > 0) {
        live = fetch(s_lo + list[0]);
        store(ps);
    }
    live = __syncthreads_or(live);
    for (int i = 0; i < n_live; ++i) {
        const int64_t s = s_lo + list[i];
        float2 *cur = ps + (i & 1) * TI * pstride;
        const bool more = i + 1 < n_live;
        bool live_next = false;
        if (more) live_next = fetch(s_lo + list[i + 1]);
        if (live) {
            const int b = static_cast<int>(s / HoWo), p = static_cast<int>(s % HoWo);
            const int py = (p / g.Wo) * g.stride - g.pad + ky;
            const int px = (p % g.Wo) * g.stride - g.pad + kx;
            if (j_ok && py >= 0 && py < g.Hp && px >= 0 && px < g.Wp) {
                const int64_t e0 = ((static_cast<int64_t>(b) * g.Hp + py) * g.Wp + px) * g.PC + ci;
                for (int d = 0; d < g.P; ++d) {
                    const int64_t e = e0 + static_cast<int64_t>(d) * g.C_in;
                    const int r = ev_row[e];
                    if (r >= 0) {
                        const float L = ev_L[e], Rv = ev_R[e];
                        const float2 *q = cur + r;
#pragma unroll
                        for (int ii = 0; ii < TI; ++ii) {
                            const float2 gg = q[ii * pstride];
                            acc[ii] = fmaf(gg.x, L, fmaf(gg.y, Rv, acc[ii]));
                        }
                    }
                }
            }
        }
        if (more) store(ps + ((i + 1) & 1) * TI * pstride);
        live = __syncthreads_or(live_next);
    }
    if (!j_ok) return;
    float *out = part + (static_cast<int64_t>(blockIdx.z) * g.C_out + co0) * NJ + jj;
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
        if (ii < ni) out[static_cast<int64_t>(ii) * NJ] = acc[ii];
}

// dW[co, ci, ky, kx] = (1/P) sum_z part[z][co][k * C_in + ci]. Threads follow
// the partial-sum layout (coalesced reads); a block holds 32 consecutive
// entries x 8 split groups: group h sums z = h, h + 8, ...; the 8 group sums
// are added in group order (fixed order: deterministic) and written to the
// [co][ci][ky][kx] slot.
constexpr int kRedOut = 32, kRedGrp = 8;

__global__ __launch_bounds__(256) void conv_dw_reduce_kernel(ConvGeom g, int nsplit,
                                                             const float *__restrict__ part,
                                                             float *__restrict__ dW) {
    __shared__ float red[kRedGrp][kRedOut];
    const int KT = g.KH * g.KW;
    const int NJ = KT * g.C_in;
    const int64_t n = static_cast<int64_t>(g.C_out) * NJ;
    const int lo = threadIdx.x % kRedOut, h = threadIdx.x / kRedOut;
    const int64_t src = static_cast<int64_t>(blockIdx.x) * kRedOut + lo;  // [co][k][ci]
    float s = 0.f;
    if (src < n) {
#pragma unroll 8
        for (int z = h; z < nsplit; z += kRedGrp) s += part[static_cast<int64_t>(z) * n + src];
    }
    red[h][lo] = s;
    __syncthreads();
    if (h == 0 && src < n) {
        float tot = 0.f;
        for (int q = 0; q < kRedGrp; ++q) tot += red[q][lo];
        const int co = static_cast<int>(src / NJ);
        const int rem = static_cast<int>(src % NJ);
        const int k = rem / g.C_in, ci = rem % g.C_in;
        dW[(static_cast<int64_t>(co) * g.C_in + ci) * KT + k] = tot * g.inv_P;
    }
}

// ------------------------------------------------------------ launchers --
int conv_sort_lds_bytes(int M, const ConvGeom &g) {
    return ((M + 3) * g.Wp + 256) * static_cast<int>(sizeof(int));
}

static hipError_t launch_conv_weights(const ConvGeom &g, const void *W, bool bf16, float *Wt,
                                      hipStream_t st) {
    const int64_t nw = static_cast<int64_t>(g.KH) * g.KW * g.C_in * g.C_out;
    ProfScope prof("conv_weights", st);
    const unsigned blocks = static_cast<unsigned>((nw + 255) / 256);
    if (bf16)
        hipLaunchKernelGGL(conv_weights_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, g,
                           static_cast<const uint16_t *>(W), Wt);
    else
        hipLaunchKernelGGL(conv_weights_kernel<float>, dim3(blocks), dim3(256), 0, st, g,
                           static_cast<const float *>(W), Wt);
    return hipGetLastError();
}

static hipError_t launch_conv_sort(const LifConst &C, const ConvGeom &g, int64_t B,
                                   const float *t_in, ConvSorted cs, hipStream_t st) {
    ProfScope prof("conv_sort", st);
    hipLaunchKernelGGL(conv_sort_kernel, dim3(static_cast<unsigned>(B * g.Hp)), dim3(256),
                       conv_sort_lds_bytes(C.M, g), st, C, g, t_in, cs);
    return hipGetLastError();
}

hipError_t launch_conv_forward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                               bool bf16, float *Wt, ConvSorted cs, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st) {
    hipError_t e = launch_conv_weights(g, W, bf16, Wt, st);
    if (e != hipSuccess) return e;
    if ((e = launch_conv_sort(C, g, B, t_in, cs, st)) != hipSuccess) return e;
    const int64_t n_pos = B * g.Ho * g.Wo;
    constexpr int waves = 4;
    dim3 grid(static_cast<unsigned>((n_pos + waves - 1) / waves),
              static_cast<unsigned>((g.C_out + kWave - 1) / kWave));
    ProfScope prof("conv_fwd", st);
    if (g.KH == 1)
        hipLaunchKernelGGL(conv_fwd_kernel<1>, grid, dim3(waves * kWave), 0, st, C, g, n_pos, Wt,
                           cs, t_out, slope, q_idx);
    else if (g.KH <= 3)
        hipLaunchKernelGGL(conv_fwd_kernel<3>, grid, dim3(waves * kWave), 0, st, C, g, n_pos, Wt,
                           cs, t_out, slope, q_idx);
    else
        hipLaunchKernelGGL(conv_fwd_kernel<kConvMaxK>, grid, dim3(waves * kWave), 0, st, C, g,
                           n_pos, Wt, cs, t_out, slope, q_idx);
    return hipGetLastError();
}

static int conv_dw_ti(const ConvGeom &g, int M) {
    const int ps = (M + 3) | 1;
    const int ti_max = (ps * 63 * 8 < 65536) ? 64 : 32;  // LDS immediate offsets
    return (g.C_out <= 32) ? 32 : ti_max;
}

static int conv_dw_nper(int M, int ti) {
    const int need = ((M + 3) * ti + 255) / 256;
    for (int n : {5, 9, 17, 33}) if (need <= n) return n;
    return -1;
}

ConvDwPlan plan_conv_dw(const ConvGeom &g, int64_t B, int M) {
    ConvDwPlan p;
    p.ti = conv_dw_ti(g, M);
    const int64_t nj = static_cast<int64_t>(g.KH) * g.KW * g.C_in;
    const int64_t n_samp = B * g.Ho * g.Wo;
    const int64_t tiles = ((nj + 255) / 256) * ((g.C_out + p.ti - 1) / p.ti);
    const int64_t nw = nj * g.C_out;
    int64_t ns = 1;
    // >= 4 blocks per CU, >= 16 samples per split and <= 64 MiB of partial
    // sums; in any case at most kConvMaxSplitSamples samples per split (the
    // block's live list)
    while ((tiles * ns < 1024 && n_samp / (ns * 2) >= 16 && ns * 2 * nw * 4 <= (64 << 20)) ||
           (n_samp + ns - 1) / ns > kConvMaxSplitSamples)
        ns *= 2;
    p.s_per_split = static_cast<int>(std::max<int64_t>(1, (n_samp + ns - 1) / ns));
    p.nsplit = static_cast<int>(std::max<int64_t>(1, (n_samp + p.s_per_split - 1) / p.s_per_split));
    return p;
}

hipError_t launch_conv_backward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                                bool bf16, const float *t_in, const float *t_out,
                                const float *slope, const int *q_idx, const float *grad_t,
                                ConvBwdWs ws, float *grad_W, float *grad_t_in, hipStream_t st) {
    const int R = C.M + 3;
    const int64_t n_in = B * g.Hp * g.Wp * g.PC;
    const int64_t n_pos = B * g.Ho * g.Wo;
    hipError_t e;
    if (n_in > 0) {
        ProfScope prof("conv_events", st);
        hipLaunchKernelGGL(conv_events_kernel, dim3(static_cast<unsigned>((n_in + 255) / 256)),
                           dim3(256), 0, st, C, g, n_in, t_in, ws.row, ws.L, ws.R, grad_t_in);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    {
        // per neuron (gamma, t - T_q, q), position-major: G of both gradients
        const int64_t n = n_pos * g.C_out;
        ProfScope prof("conv_grad_prep", st);
        if (n > 0)
            hipLaunchKernelGGL(conv_grad_prep_kernel, dim3(static_cast<unsigned>((n + 255) / 256)),
                               dim3(256), 0, st, C, g, n, t_out, slope, q_idx, grad_t, ws.gam,
                               ws.uq, ws.q);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (grad_W) {
        ConvDwPlan p = plan_conv_dw(g, B, C.M);
        const int64_t nj = static_cast<int64_t>(g.KH) * g.KW * g.C_in;
        const int pstride = (C.M + 3) | 1;
        dim3 grid(static_cast<unsigned>((nj + 255) / 256),
                  static_cast<unsigned>((g.C_out + p.ti - 1) / p.ti),
                  static_cast<unsigned>(p.nsplit));
        const size_t lds = 2 * static_cast<size_t>(p.ti) * pstride * sizeof(float2) +
                           static_cast<size_t>(p.s_per_split) * sizeof(int);
        const int nper = conv_dw_nper(C.M, p.ti);
        if (n_pos > 0) {
            ProfScope prof("conv_live", st);
            hipLaunchKernelGGL(conv_live_kernel, dim3(static_cast<unsigned>((n_pos + 255) / 256)),
                               dim3(256), 0, st, n_pos, g.C_out, ws.q, ws.live);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        {
            ProfScope prof("conv_dw", st);
#define CDW_LAUNCH(TIV, NP)                                                                   \
    hipLaunchKernelGGL((conv_dw_kernel<TIV, NP>), grid, dim3(256), lds, st, C, g, n_pos,       \
                       p.s_per_split, pstride, ws.gam, ws.uq, ws.q, ws.live, ws.row, ws.L, ws.R, \
                       ws.part)
            if (p.ti == 64) {
                if (nper == 5) CDW_LAUNCH(64, 5);
                else if (nper == 9) CDW_LAUNCH(64, 9);
                else if (nper == 17) CDW_LAUNCH(64, 17);
                else CDW_LAUNCH(64, 33);
            } else {
                if (nper == 5) CDW_LAUNCH(32, 5);
                else if (nper == 9) CDW_LAUNCH(32, 9);
                else if (nper == 17) CDW_LAUNCH(32, 17);
                else CDW_LAUNCH(32, 33);
            }
#undef CDW_LAUNCH
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        const int64_t n = static_cast<int64_t>(g.C_out) * nj;
        ProfScope prof("conv_dw_reduce", st);
        hipLaunchKernelGGL(conv_dw_reduce_kernel,
                           dim3(static_cast<unsigned>((n + kRedOut - 1) / kRedOut)),
                           dim3(kRedOut * kRedGrp), 0, st, g, p.nsplit, ws.part, grad_W);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (grad_t_in && n_in > 0) {
        if ((e = launch_conv_weights(g, W, bf16, ws.wt, st)) != hipSuccess) return e;
        if ((e = launch_conv_sort(C, g, B, t_in, ws.srt, st)) != hipSuccess) return e;
        if (n_pos > 0) {
            constexpr int waves = 4;
            dim3 grid(static_cast<unsigned>((n_pos + waves - 1) / waves));
            const int nt = (g.C_out + kWave - 1) / kWave;
            ProfScope prof("conv_dtp", st);
#define DTP_LAUNCH(KHV, NTV)                                                                  \
    hipLaunchKernelGGL((conv_dtp_kernel<KHV, NTV>), grid, dim3(waves * kWave), 0, st, C, g,    \
                       n_pos, ws.wt, ws.srt, ws.gam, ws.uq, ws.q)
#define DTP_NT(KHV)                               \
    do {                                          \
        if (nt == 1) DTP_LAUNCH(KHV, 1);          \
        else if (nt == 2) DTP_LAUNCH(KHV, 2);     \
        else if (nt <= 4) DTP_LAUNCH(KHV, 4);     \
        else DTP_LAUNCH(KHV, 8);                  \
    } while (0)
            if (g.KH == 1) DTP_NT(1);
            else if (g.KH <= 3) DTP_NT(3);
            else DTP_NT(kConvMaxK);
#undef DTP_NT
#undef DTP_LAUNCH
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        ProfScope prof("conv_dt_gather", st);
        hipLaunchKernelGGL(conv_dt_gather_kernel, dim3(static_cast<unsigned>((n_in + 255) / 256)),
                           dim3(256), 0, st, g, R, n_in, ws.srt, grad_t_in);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace dstd
