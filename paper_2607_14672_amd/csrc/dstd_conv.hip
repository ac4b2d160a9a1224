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
// Forward: the inputs of one cell row (b, py) are bucketed by (event row r,
// cell column px) -- counting sort, stable in j' -- so the records of row r
// for the KW cells under an output position's kernel row form ONE contiguous
// segment. An output wavefront (lanes = output channels) walks the rows in
// grid order, sums the KH segments of each row and runs the interval scan
// as rows close (the dense forward's scheme; the weighted events never
// exist in memory).
// Backward: dW and dt_in follow the dense kernels with the receptive-field
// index maps; G is position-major so channel tiles are contiguous.
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
// LDS: hist[px][r] (later the next free slot of bucket (r, px)), then the
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
                cs.L[o] = e.L;
                cs.R[o] = e.R;
            }
        }
    }
}

// ------------------------------------------------------ weight layouts ---
// Forward: WT[(k * C_in + ci) * C_out + co] = W[co, ci, k] / P (k = ky*KW+kx).
// Backward dt_in: WD[(k * C_out + co) * C_in + ci] = W[co, ci, k] / P.
template <typename WT>
__global__ __launch_bounds__(256) void conv_weights_kernel(ConvGeom g, const WT *__restrict__ W,
                                                           float *__restrict__ out, int to_wd) {
    const int KT = g.KH * g.KW;
    const int64_t n = static_cast<int64_t>(KT) * g.C_in * g.C_out;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    int co, ci, k;
    if (to_wd) {  // t = (k * C_out + co) * C_in + ci
        ci = static_cast<int>(t % g.C_in);
        const int64_t u = t / g.C_in;
        co = static_cast<int>(u % g.C_out);
        k = static_cast<int>(u / g.C_out);
    } else {      // t = (k * C_in + ci) * C_out + co
        co = static_cast<int>(t % g.C_out);
        const int64_t u = t / g.C_out;
        ci = static_cast<int>(u % g.C_in);
        k = static_cast<int>(u / g.C_in);
    }
    const float w = WLoad<WT>::get(W, (static_cast<int64_t>(co) * g.C_in + ci) * KT + k);
    out[t] = w * g.inv_P;
}

// -------------------------------------------------------------- forward --
// Wave = one output position (b, oy, ox), lane = output channel of a 64-wide
// tile. Per event row r and kernel row ky the records form the segment
// [off[r][xa], off[r][xb]) of cell row py = oy*stride - pad + ky; a record's
// key px*C_in + ci plus the per-segment constant (ky*KW - x0)*C_in is its
// weight row. The bucket starts of the KH cell rows are held one event row
// per lane (64 rows at a time) and read with readlane.
constexpr int kCBatch = 8;

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
    const int b = uniform(static_cast<int>(p / HoWo));
    const int pos = uniform(static_cast<int>(p % HoWo));
    const int oy = pos / g.Wo, ox = pos % g.Wo;
    const int R = rows_of(C);
    const int x0 = ox * g.stride - g.pad;
    const int xa = max(0, x0), xb = max(xa, min(g.Wp, x0 + g.KW));
    const int nb1 = R * g.Wp + 1;
    const int wlim = g.KH * g.KW * g.C_in - 1;
    int64_t recb[KHT], offb[KHT];
    int wofs[KHT];
    bool vky[KHT];
#pragma unroll
    for (int ky = 0; ky < KHT; ++ky) {
        const int py = oy * g.stride - g.pad + ky;
        vky[ky] = ky < g.KH && py >= 0 && py < g.Hp && xa < xb;
        const int64_t cr = static_cast<int64_t>(b) * g.Hp + (vky[ky] ? py : 0);
        recb[ky] = cr * g.Wp * g.PC;
        offb[ky] = cr * nb1;
        wofs[ky] = (ky * g.KW - x0) * g.C_in;
    }
    int oa[KHT], ob[KHT];
    auto load_offs = [&](int r0) {
        const int r = min(r0 + lane, R - 1);
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int *o = cs.off + offb[ky] + static_cast<int64_t>(r) * g.Wp;
            oa[ky] = vky[ky] ? o[xa] : 0;
            ob[ky] = vky[ky] ? o[xb] : 0;
        }
    };
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(
        Wt, static_cast<uint32_t>(static_cast<int64_t>(wlim + 1) * g.C_out * sizeof(float)));
    const int voff = (row_ok ? co : 0) * static_cast<int>(sizeof(float));
    const int rstride = g.C_out * static_cast<int>(sizeof(float));
    // weight row of a record; stale keys read past a segment end are clamped
    // so the scalar offset always stays inside WT
    auto wrow = [&](int key, int wo) { return min(max(key + wo, 0), wlim) * rstride; };
    Scan sc;
    float aL = 0.f, aR = 0.f, carry = 0.f;
    for (int r = 0; r <= R - 2; ++r) {
        if ((r & (kWave - 1)) == 0) load_offs(r);
        const int l = r & (kWave - 1);
        int s0[KHT], n0[KHT];
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            s0[ky] = __builtin_amdgcn_readlane(oa[ky], l);
            n0[ky] = __builtin_amdgcn_readlane(ob[ky], l) - s0[ky];
        }
        // first batch of every kernel row issued together
        float w[KHT][kCBatch], lv[KHT][kCBatch], rv[KHT][kCBatch];
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int64_t o = recb[ky] + s0[ky];
#pragma unroll
            for (int kk = 0; kk < kCBatch; ++kk) {
                w[ky][kk] = BufLoad<float>::get(wr, voff, wrow(as_const(cs.key + o)[kk], wofs[ky]));
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
                const int64_t o = recb[ky] + s0[ky] + k0;
                const int nk = n0[ky] - k0;
                float wb[kCBatch], lb[kCBatch], rb[kCBatch];
#pragma unroll
                for (int kk = 0; kk < kCBatch; ++kk) {
                    wb[kk] = BufLoad<float>::get(wr, voff, wrow(as_const(cs.key + o)[kk], wofs[ky]));
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
    const int64_t o = (static_cast<int64_t>(b) * g.C_out + co) * HoWo + pos;
    t_out[o] = to;
    slope[o] = sl;
    q_idx[o] = q;
}

// --------------------------------------------------------- backward ------
// Events of every input in cell-major order (row -1 = no events).
__global__ __launch_bounds__(256) void conv_events_kernel(LifConst C, ConvGeom g, int64_t n,
                                                          const float *__restrict__ t_in,
                                                          int *__restrict__ ev_row,
                                                          float *__restrict__ ev_L,
                                                          float *__restrict__ ev_R,
                                                          float *__restrict__ ev_dL,
                                                          float *__restrict__ ev_dR) {
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
    const Event e = bin_event(C, t_in[nchw_index(g, b, j % g.C_in, y, x)]);
    ev_row[k] = e.row;
    ev_L[k] = e.L;
    ev_R[k] = e.R;
    ev_dL[k] = e.dL;
    ev_dR[k] = e.dR;
}

// dW[co, ci, k] = (1/P) sum_{b, p} sum_d (G[b, r, p, co] L + G[b, r+1, p, co] R)
// over the raw inputs d of the cell that tap k of position p reads.
// Lane = (k, ci); a block covers 256 of them and a tile of TI channels whose
// sums stay in registers over its share of the (b, p) samples. G[b, :, p,
// tile] is staged in LDS as (G[r], G[r+1]) pairs, double buffered, with the
// next sample's loads in registers (NPER per thread) during this one's sums.
template <int TI, int NPER>
__global__ __launch_bounds__(256) void conv_dw_kernel(LifConst C, ConvGeom g, int64_t n_samp,
                                                      int s_per_split, int pstride,
                                                      const float *__restrict__ G,
                                                      const int *__restrict__ ev_row,
                                                      const float *__restrict__ ev_L,
                                                      const float *__restrict__ ev_R,
                                                      float *__restrict__ part) {
    extern __shared__ float2 ps[];  // [2][TI][pstride]
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
    const int64_t gstride = static_cast<int64_t>(HoWo) * g.C_out;  // one G row
    float acc[TI];
#pragma unroll
    for (int ii = 0; ii < TI; ++ii) acc[ii] = 0.f;
    const int total = R * TI;
    float pre[NPER];
    auto fetch = [&](int64_t s) {
        const int b = static_cast<int>(s / HoWo), p = static_cast<int>(s % HoWo);
        const float *gb = G + (static_cast<int64_t>(b) * R * HoWo + p) * g.C_out + co0;
#pragma unroll
        for (int c = 0; c < NPER; ++c) {
            const int kk = threadIdx.x + c * 256;
            const int r = min(kk / TI, R - 1), l = min(kk % TI, ni - 1);
            pre[c] = gb[r * gstride + l];
        }
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
    if (s_lo < s_hi) {
        fetch(s_lo);
        store(ps);
    }
    __syncthreads();
    for (int64_t s = s_lo; s < s_hi; ++s) {
        float2 *cur = ps + ((s - s_lo) & 1) * TI * pstride;
        const bool more = s + 1 < s_hi;
        if (more) fetch(s + 1);
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
        if (more) store(ps + ((s + 1 - s_lo) & 1) * TI * pstride);
        __syncthreads();
    }
    if (!j_ok) return;
    float *out = part + (static_cast<int64_t>(blockIdx.z) * g.C_out + co0) * NJ + jj;
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
        if (ii < ni) out[static_cast<int64_t>(ii) * NJ] = acc[ii];
}

// dW[co, ci, ky, kx] = (1/P) sum_z part[z][co][k * C_in + ci], fixed order.
__global__ __launch_bounds__(256) void conv_dw_reduce_kernel(ConvGeom g, int nsplit,
                                                             const float *__restrict__ part,
                                                             float *__restrict__ dW) {
    const int KT = g.KH * g.KW;
    const int NJ = KT * g.C_in;
    const int64_t n = static_cast<int64_t>(g.C_out) * NJ;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    const int k = static_cast<int>(t % KT);
    const int64_t u = t / KT;
    const int ci = static_cast<int>(u % g.C_in);
    const int co = static_cast<int>(u / g.C_in);
    const int64_t src = static_cast<int64_t>(co) * NJ + static_cast<int64_t>(k) * g.C_in + ci;
    float s = 0.f;
    for (int z = 0; z < nsplit; ++z) s += part[static_cast<int64_t>(z) * n + src];
    dW[t] = s * g.inv_P;
}

// dt_in of raw input (cell, j'): dL A_r + dR A_{r+1}, A_m = sum over taps k
// and channels co of WD[k, co, ci] G[b, m, p(cell, k), co]. Lane = j' of a
// cell (blockIdx.y selects the 256-wide chunk of j'); a block (blockIdx.x)
// holds SB consecutive cells of one cell row and, per tap and
// 64-channel chunk, their G tiles in LDS (row stride 65 words: the
// lane-dependent rows r, r+1 come from one conflict-free ds_read2). Taps
// that reach no output position for a cell stage zeros; a tap that misses
// every cell of the block is skipped.
template <int SB>
__global__ __launch_bounds__(256) void conv_dtin_kernel(LifConst C, ConvGeom g, int B,
                                                        const float *__restrict__ G,
                                                        const float *__restrict__ Wd,
                                                        const int *__restrict__ ev_row,
                                                        const float *__restrict__ ev_dL,
                                                        const float *__restrict__ ev_dR,
                                                        float *__restrict__ dt_in) {
    extern __shared__ float gs[];  // [SB][R + 1][kDtStride]
    const int R = rows_of(C);
    const int RT = R + 1;
    const int jd = blockIdx.y * blockDim.x + threadIdx.x;
    const bool j_ok = jd < g.PC;
    const int ci = (j_ok ? jd : 0) % g.C_in;
    const int nxc = (g.Wp + SB - 1) / SB;
    const int cy = blockIdx.x;
    const int b = cy / (g.Hp * nxc);
    const int py = (cy / nxc) % g.Hp;
    const int px0 = (cy % nxc) * SB;
    const int HoWo = g.Ho * g.Wo;
    const int64_t cellrow = (static_cast<int64_t>(b) * g.Hp + py) * g.Wp;
    int base[SB];
    float aL[SB], aR[SB];
#pragma unroll
    for (int s = 0; s < SB; ++s) {
        aL[s] = 0.f;
        aR[s] = 0.f;
        const int px = px0 + s;
        int r = (j_ok && px < g.Wp) ? ev_row[(cellrow + px) * g.PC + jd] : -1;
        if (r < 0) r = R - 1;  // rows R-1 and R are zero
        base[s] = (s * RT + r) * kDtStride;
    }
    for (int k = threadIdx.x; k < SB * kDtStride; k += blockDim.x)
        gs[((k / kDtStride) * RT + R) * kDtStride + (k % kDtStride)] = 0.f;
    for (int ky = 0; ky < g.KH; ++ky) {
        const int oyn = py + g.pad - ky;
        if (oyn < 0 || oyn % g.stride != 0 || oyn / g.stride >= g.Ho) continue;  // uniform
        const int oy = oyn / g.stride;
        for (int kx = 0; kx < g.KW; ++kx) {
            int pos[SB];
            bool any = false;
#pragma unroll
            for (int s = 0; s < SB; ++s) {
                const int oxn = px0 + s + g.pad - kx;
                const bool v = px0 + s < g.Wp && oxn >= 0 && oxn % g.stride == 0 &&
                               oxn / g.stride < g.Wo;
                pos[s] = v ? oy * g.Wo + oxn / g.stride : -1;
                any = any || v;
            }
            if (!any) continue;  // uniform
            const int k = ky * g.KW + kx;
            for (int c0 = 0; c0 < g.C_out; c0 += kWave) {
                const int nco = min(kWave, g.C_out - c0);
                // weights of this chunk for the lane's channel; indices are
                // clamped into range (columns past the chunk meet zero G)
                float w[kWave];
                const float *wk = Wd + static_cast<int64_t>(k) * g.C_out * g.C_in + ci;
#pragma unroll
                for (int ii = 0; ii < kWave; ++ii)
                    w[ii] = wk[static_cast<int64_t>(min(c0 + ii, g.C_out - 1)) * g.C_in];
                __syncthreads();
                for (int t = threadIdx.x; t < SB * R * kWave; t += blockDim.x) {
                    const int s = t / (R * kWave);
                    const int r = (t / kWave) % R;
                    const int l = t % kWave;
                    int ps = -1;
#pragma unroll
                    for (int u = 0; u < SB; ++u)
                        if (u == s) ps = pos[u];
                    gs[(s * RT + r) * kDtStride + l] =
                        (ps >= 0 && l < nco)
                            ? G[((static_cast<int64_t>(b) * R + r) * HoWo + ps) * g.C_out + c0 + l]
                            : 0.f;
                }
                __syncthreads();
#pragma unroll
                for (int ii = 0; ii < kWave; ++ii) {
#pragma unroll
                    for (int s = 0; s < SB; ++s) {
                        const float g0 = gs[base[s] + ii];
                        const float g1 = gs[base[s] + kDtStride + ii];
                        aL[s] = fmaf(w[ii], g0, aL[s]);
                        aR[s] = fmaf(w[ii], g1, aR[s]);
                    }
                }
            }
        }
    }
    if (!j_ok) return;
    const int d = jd / g.C_in;
#pragma unroll
    for (int s = 0; s < SB; ++s) {
        const int px = px0 + s;
        if (px >= g.Wp) continue;
        const int64_t e = (cellrow + px) * g.PC + jd;
        const bool has = base[s] != (s * RT + R - 1) * kDtStride;
        int y, x;
        raw_pixel(g, py, px, d, y, x);
        dt_in[nchw_index(g, b, ci, y, x)] = has ? fmaf(aL[s], ev_dL[e], aR[s] * ev_dR[e]) : 0.f;
    }
}

// ------------------------------------------------------------ launchers --
int conv_sort_lds_bytes(int M, const ConvGeom &g) {
    return ((M + 3) * g.Wp + 256) * static_cast<int>(sizeof(int));
}

hipError_t launch_conv_forward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                               bool bf16, float *Wt, ConvSorted cs, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st) {
    const int64_t nw = static_cast<int64_t>(g.KH) * g.KW * g.C_in * g.C_out;
    {
        ProfScope prof("conv_weights", st);
        const unsigned blocks = static_cast<unsigned>((nw + 255) / 256);
        if (bf16)
            hipLaunchKernelGGL(conv_weights_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, g,
                               static_cast<const uint16_t *>(W), Wt, 0);
        else
            hipLaunchKernelGGL(conv_weights_kernel<float>, dim3(blocks), dim3(256), 0, st, g,
                               static_cast<const float *>(W), Wt, 0);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        ProfScope prof("conv_sort", st);
        hipLaunchKernelGGL(conv_sort_kernel, dim3(static_cast<unsigned>(B * g.Hp)), dim3(256),
                           conv_sort_lds_bytes(C.M, g), st, C, g, t_in, cs);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
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
    int64_t ns = 1;
    // >= 4 blocks per CU; >= 16 samples per split
    while (tiles * ns < 1024 && n_samp / (ns * 2) >= 16) ns *= 2;
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
    hipError_t e;
    if (n_in > 0) {
        ProfScope prof("conv_events", st);
        hipLaunchKernelGGL(conv_events_kernel, dim3(static_cast<unsigned>((n_in + 255) / 256)),
                           dim3(256), 0, st, C, g, n_in, t_in, ws.row, ws.L, ws.R, ws.dL, ws.dR);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    e = launch_grad_g(C, B, static_cast<int64_t>(g.Ho) * g.Wo, g.C_out, t_out, slope, q_idx,
                      grad_t, ws.G, st);
    if (e != hipSuccess) return e;
    if (grad_W) {
        ConvDwPlan p = plan_conv_dw(g, B, C.M);
        const int64_t nj = static_cast<int64_t>(g.KH) * g.KW * g.C_in;
        const int pstride = (C.M + 3) | 1;
        dim3 grid(static_cast<unsigned>((nj + 255) / 256),
                  static_cast<unsigned>((g.C_out + p.ti - 1) / p.ti),
                  static_cast<unsigned>(p.nsplit));
        const size_t lds = 2 * static_cast<size_t>(p.ti) * pstride * sizeof(float2);
        const int64_t n_samp = B * g.Ho * g.Wo;
        const int nper = conv_dw_nper(C.M, p.ti);
        {
            ProfScope prof("conv_dw", st);
#define CDW_LAUNCH(TIV, NP)                                                                   \
    hipLaunchKernelGGL((conv_dw_kernel<TIV, NP>), grid, dim3(256), lds, st, C, g, n_samp,      \
                       p.s_per_split, pstride, ws.G, ws.row, ws.L, ws.R, ws.part)
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
        hipLaunchKernelGGL(conv_dw_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)),
                           dim3(256), 0, st, g, p.nsplit, ws.part, grad_W);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (grad_t_in && n_in > 0) {
        const int64_t nw = static_cast<int64_t>(g.KH) * g.KW * g.C_in * g.C_out;
        {
            ProfScope prof("conv_weights", st);
            const unsigned blocks = static_cast<unsigned>((nw + 255) / 256);
            if (bf16)
                hipLaunchKernelGGL(conv_weights_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, g,
                                   static_cast<const uint16_t *>(W), ws.wd, 1);
            else
                hipLaunchKernelGGL(conv_weights_kernel<float>, dim3(blocks), dim3(256), 0, st, g,
                                   static_cast<const float *>(W), ws.wd, 1);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        const int sb = conv_dtin_sb(C.M, g);
        const int threads = static_cast<int>(std::min<int64_t>(256, (g.PC + kWave - 1) / kWave * kWave));
        const int nxc = (g.Wp + sb - 1) / sb;
        dim3 grid(static_cast<unsigned>(B * g.Hp * nxc),
                  static_cast<unsigned>((g.PC + threads - 1) / threads));
        const size_t lds = static_cast<size_t>(sb) * (R + 1) * kDtStride * sizeof(float);
        ProfScope prof("conv_dtin", st);
        if (sb == 4)
            hipLaunchKernelGGL(conv_dtin_kernel<4>, grid, dim3(threads), lds, st, C, g,
                               static_cast<int>(B), ws.G, ws.wd, ws.row, ws.dL, ws.dR, grad_t_in);
        else if (sb == 2)
            hipLaunchKernelGGL(conv_dtin_kernel<2>, grid, dim3(threads), lds, st, C, g,
                               static_cast<int>(B), ws.G, ws.wd, ws.row, ws.dL, ws.dR, grad_t_in);
        else
            hipLaunchKernelGGL(conv_dtin_kernel<1>, grid, dim3(threads), lds, st, C, g,
                               static_cast<int>(B), ws.G, ws.wd, ws.row, ws.dL, ws.dR, grad_t_in);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

int conv_dtin_sb(int M, const ConvGeom &g) {
    int sb = 4;
    while (sb > 1 && (sb > g.Wp || static_cast<size_t>(sb) * (M + 4) * kDtStride * sizeof(float) >
                                        80 * 1024))
        sb >>= 1;
    return sb;
}

}  // namespace dstd
