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

// Raw input v = ((ky * KW + kx) * P + d) * C_in + ci (v < 64) of the
// receptive field of an output position of image b whose window starts at
// cell row py0 = oy * stride - pad and cell column x0: its NCHW index, or -1
// where the cell lies in the padding; wrow = its weight row k * C_in + ci.
__device__ __forceinline__ int64_t rf_input(const ConvGeom &g, int b, int py0, int x0, int v,
                                            int &wrow) {
    const int t1 = fdiv(v, g.dv_cin), ci = v - t1 * g.C_in;
    const int k = fdiv(t1, g.dv_p), d = t1 - k * g.P;
    const int ky = fdiv(k, g.dv_kw), kx = k - ky * g.KW;
    const int py = py0 + ky, px = x0 + kx;
    wrow = k * g.C_in + ci;
    if (py < 0 || py >= g.Hp || px < 0 || px >= g.Wp) return -1;
    int y, x;
    raw_pixel(g, py, px, d, y, x);
    return nchw_index(g, b, ci, y, x);
}

// Events of the raw inputs [1024 blk, 1024 blk + 1024) in NCHW order (layers
// whose forward bins its receptive fields directly, plain input): key = event
// row (-1: none), L, R where the row is >= 0. Every position that reads an
// input then loads its event instead of binning it again.
constexpr int kBinPerBlock = 1024;
__device__ void bin_block(const LifConst &C, int64_t n_in, const float *__restrict__ t_in,
                          const ConvSorted &cs, int blk) {
    const int64_t i0 = static_cast<int64_t>(blk) * kBinPerBlock + threadIdx.x;
    float v[kBinPerBlock / 256];
#pragma unroll
    for (int u = 0; u < kBinPerBlock / 256; ++u) {
        const int64_t i = i0 + u * 256;
        v[u] = (i < n_in) ? t_in[i] : INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kBinPerBlock / 256; ++u) {
        const int64_t i = i0 + u * 256;
        if (i < n_in) {
            const Event e = bin_event(C, v[u]);
            cs.key[i] = e.row;
            if (e.row >= 0) {
                cs.L[i] = e.L;
                cs.R[i] = e.R;
            }
        }
    }
}

// The t-th raw input of cell row (b, py) in NCHW order (channel-major, so
// consecutive t are mostly consecutive addresses): its NCHW index, and its
// cell-major slot px * PC + j' in `slot`.
__device__ __forceinline__ int64_t cell_row_input(const ConvGeom &g, int b, int py, int t,
                                                  int &slot) {
    const int per_ch = g.Wp * g.P;
    const int ci = fdiv(t, g.dv_pch), rem = t - ci * per_ch;  // t < 2^30
    int y, x, px, d;
    if (g.pool == 2) {
        const int dy = fdiv(rem, g.dv_w);
        x = rem - dy * g.W;
        y = 2 * py + dy;
        px = x >> 1;
        d = dy * 2 + (x & 1);
    } else if (g.pool == 0) {
        d = rem;
        y = fdiv(d, g.dv_w);
        x = d - y * g.W;
        px = 0;
    } else {
        x = rem;
        y = py;
        px = rem;
        d = 0;
    }
    slot = px * g.PC + d * g.C_in + ci;
    return nchw_index(g, b, ci, y, x);
}

// ------------------------------------------------------------ cell sort --
// One block of 256 threads per cell row (b, py).
// LDS: hist[r][px] (later the next free slot of bucket (r, px)), the 256
// per-thread partial sums of the prefix scan, then (when they fit) the cell
// row's input spike times in cell-major order, read once in NCHW order, and
// (when they fit too) the four waves' lists of inputs with events.
// Wave w owns cells px = w, w + 4, ... (each bucket is ranked by one wave
// only); where a cell has fewer than 64 inputs a wave takes several of its
// cells per pass. Records of a bucket keep the input order (j' ascending).
// The cell row's events (ev) are written too: every input's row, and L, R
// where the row is >= 0.
__host__ __device__ __forceinline__ int sort_stage_floats(int M, const ConvGeom &g) {
    const int per = g.Wp * g.PC;
    return ((M + 3) * g.Wp + 256 + per) * 4 <= 64 * 1024 ? per : 0;
}

// With the row staged: ints of the four waves' lists of event inputs (each
// wave owns the cell columns px = wave mod 4, at most ceil(Wp / 4) * PC
// inputs), or 0 where they do not fit beside the staging in 64 KB.
constexpr int kSortWaves = 4;  // the sort runs in blocks of 256 threads
__host__ __device__ __forceinline__ int sort_list_ints(int M, const ConvGeom &g) {
    const int stage = sort_stage_floats(M, g);
    const int cap = (g.Wp + kSortWaves - 1) / kSortWaves * g.PC * kSortWaves;
    return (stage > 0 && ((M + 3) * g.Wp + 256 + stage + cap) * 4 <= 64 * 1024) ? cap : 0;
}

__device__ void sort_cell_row(const LifConst &C, const ConvGeom &g, const float *__restrict__ t_in,
                              const ConvSorted &cs, const CellEv &ev, int cr, int *sh) {
    const int R = rows_of(C);
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int nw = blockDim.x >> 6;
    const int b = cr / g.Hp, py = cr % g.Hp;
    const int nb = R * g.Wp;  // buckets, flat f = r * Wp + px
    const int noff = conv_off_stride(R, g);
    const bool fwd = cs.L != nullptr, bwd = cs.dL != nullptr;
    int *hist = sh;
    int *part = sh + nb;
    float *tl = sort_stage_floats(C.M, g) > 0 ? reinterpret_cast<float *>(part + 256) : nullptr;
    for (int k = threadIdx.x; k < nb; k += blockDim.x) hist[k] = 0;
    if (tl) {
        // staged rows are checked for events as they are read: a row without
        // any (the deep layers at random initialisation) skips the
        // histogram pass. The test is a window 0.001 dt wider at both ends
        // than the one bin_row keeps, [T_0 - dt, T_M + dt) (a superset:
        // bin_row's rounding moves its bounds far less), so it costs two
        // compares; NaN and +-inf fail it.
        const int per = g.Wp * g.PC;
        const float w_lo = C.t0 - 1.001f * C.dt;
        const float w_hi = fmaf(static_cast<float>(C.M) + 1.001f, C.dt, C.t0);
        bool any = false;
        // four inputs per pass, their loads issued together
        for (int t4 = threadIdx.x; t4 < per; t4 += 4 * blockDim.x) {
            int slot[4];
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int t = t4 + u * static_cast<int>(blockDim.x);
                const int64_t src = cell_row_input(g, b, py, min(t, per - 1), slot[u]);
                v[u] = (t < per) ? t_in[src] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (t4 + u * static_cast<int>(blockDim.x) < per) {
                    tl[slot[u]] = v[u];
                    any = any || (v[u] >= w_lo && v[u] < w_hi);
                }
            }
        }
        if (!__syncthreads_or(any)) {
            if (ev.row && threadIdx.x == 0) ev.live[cr] = 0;
            int *off0 = cs.off + static_cast<int64_t>(cr) * noff;
            for (int f = threadIdx.x; f < noff; f += blockDim.x) off0[f] = 0;
            return;
        }
    } else {
        __syncthreads();
    }
    auto t_at = [&](int px, int j) {
        if (tl) return tl[px * g.PC + j];
        int y, x;
        const int d = fdiv(j, g.dv_cin);
        raw_pixel(g, py, px, d, y, x);
        return t_in[nchw_index(g, b, j - d * g.C_in, y, x)];
    };
    const int cpi = (g.PC < kWave) ? kWave / g.PC : 1;  // cells per pass
    const int lsub = (g.PC < kWave) ? lane / g.PC : 0;
    const int lj = (g.PC < kWave) ? lane % g.PC : lane;
    const int64_t rb = static_cast<int64_t>(cr) * g.Wp * g.PC;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    // List form (the row staged and the lists fitting): the histogram pass
    // also appends each event input (slot px * PC + j, row r) to its wave's
    // list in pass order and writes every input's event row; the placement
    // then visits only the listed inputs. A wave's buckets (r, px) hold only
    // its own cell columns, so list order is the pass order within each.
    const int lcap = (tl && nw == kSortWaves) ? sort_list_ints(C.M, g) / kSortWaves : 0;
    int *lst = lcap > 0 ? reinterpret_cast<int *>(tl + sort_stage_floats(C.M, g)) + wave * lcap
                        : nullptr;
    int nq = 0;
    bool has = false;
    for (int i0 = 0; wave + nw * i0 < g.Wp; i0 += cpi) {
        const int px = wave + nw * (i0 + lsub);
        const bool cell_ok = lsub < cpi && px < g.Wp;
        for (int j0 = 0; j0 < g.PC; j0 += kWave) {
            const int j = j0 + lj;
            int r = -1;
            if (cell_ok && j < g.PC) {
                r = bin_row(C, t_at(px, j));
                if (lst && ev.row) ev.row[rb + px * g.PC + j] = r;
                if (r >= 0) {
                    atomicAdd(&hist[r * g.Wp + px], 1);
                    has = true;
                }
            }
            if (lst) {
                const uint64_t m = __ballot(r >= 0);
                if (r >= 0) lst[nq + __popcll(m & below)] = ((px * g.PC + j) << 9) | r;
                nq += __popcll(m);
            }
        }
    }
    has = __syncthreads_or(has);
    if (ev.row && threadIdx.x == 0) ev.live[cr] = has;
    if (!has) {
        // no input of this cell row has events: empty buckets
        int *off0 = cs.off + static_cast<int64_t>(cr) * noff;
        for (int f = threadIdx.x; f < noff; f += blockDim.x) off0[f] = 0;
        return;
    }
    // exclusive prefix over the buckets in (r, px) order: per-thread chunk
    // sums, scanned by wave 0 (four per lane), then each chunk in order
    const int chunk = (nb + blockDim.x - 1) / blockDim.x;
    const int lo = min(nb, static_cast<int>(threadIdx.x) * chunk), hi = min(nb, lo + chunk);
    int s = 0;
    for (int f = lo; f < hi; ++f) s += hist[f];
    part[threadIdx.x] = s;
    __syncthreads();
    if (wave == 0) {
        const int v0 = part[4 * lane], v1 = part[4 * lane + 1], v2 = part[4 * lane + 2],
                  v3 = part[4 * lane + 3];
        const int tot = v0 + v1 + v2 + v3;
        int inc = tot;
#pragma unroll
        for (int m = 1; m < kWave; m <<= 1) {
            const int o = __shfl_up(inc, m);
            if (lane >= m) inc += o;
        }
        const int ex = inc - tot;
        part[4 * lane] = ex;
        part[4 * lane + 1] = ex + v0;
        part[4 * lane + 2] = ex + v0 + v1;
        part[4 * lane + 3] = ex + v0 + v1 + v2;
        if (lane == kWave - 1) {
            // the last row's end and the record count
            int *off = cs.off + static_cast<int64_t>(cr) * noff;
            off[g.Wp * R + R - 1] = inc;
            off[noff - 1] = inc;
        }
    }
    __syncthreads();
    int run = part[threadIdx.x];
    int *off = cs.off + static_cast<int64_t>(cr) * noff;
    int r = lo / g.Wp, px = lo - r * g.Wp;  // bucket f = r * Wp + px, advanced with f
    for (int f = lo; f < hi; ++f) {
        const int v = hist[f];
        off[px * R + r] = run;
        if (px == 0 && r > 0) off[g.Wp * R + r - 1] = run;  // the end of row r - 1
        hist[f] = run;
        run += v;
        if (++px == g.Wp) {
            px = 0;
            ++r;
        }
    }
    __syncthreads();
    // placement: lanes of one bucket are ranked by lane (j' ascending). The
    // lanes of one pass that share a bucket are found by matching the bits of
    // a per-pass bucket key k = row * cpi + lsub (one ballot per bit, a cost
    // independent of how many buckets the pass touches); the highest lane of
    // each group then moves the bucket's next free slot.
    if (lst) {
        // list form: 64 listed inputs per pass, key row * ncw + px / 4
        // (ncw = the wave's cell columns); entries are in pass order, so each
        // bucket's records keep the input order
        const int ncw = (g.Wp + kSortWaves - 1) / kSortWaves;
        const int kb2 = uniform(R * ncw > 1 ? 32 - __clz(R * ncw - 1) : 0);
        for (int c0 = 0; c0 < nq; c0 += kWave) {
            const bool ok = c0 + lane < nq;
            const int en = ok ? lst[c0 + lane] : 0;
            const int slot = en >> 9, r = en & 511;
            const int px = fdiv(slot, g.dv_pc), j = slot - px * g.PC;
            Event e{-1, 0.f, 0.f, 0.f, 0.f};
            if (ok) e = bin_event(C, tl[slot]);  // its row is r
            const int kb = ok ? r * ncw + px / kSortWaves : 0;
            uint64_t same = __ballot(ok);
            for (int bit = 0; bit < kb2; ++bit) {
                const bool on = (kb >> bit) & 1;
                const uint64_t bal = __ballot(on);
                same &= on ? bal : ~bal;
            }
            const int f = r * g.Wp + px;
            int pos = 0;
            if (ok) {
                const int base = hist[f];
                pos = base + __popcll(same & below);
                if ((same >> lane) == 1ull) hist[f] = base + __popcll(same);
            }
            __builtin_amdgcn_wave_barrier();
            if (ok) {
                if (ev.row) {
                    ev.L[rb + slot] = e.L;
                    ev.R[rb + slot] = e.R;
                }
                const int64_t o = rb + pos;
                cs.key[o] = px * g.C_in + (j - fdiv(j, g.dv_cin) * g.C_in);
                if (fwd) {
                    cs.L[o] = e.L;
                    cs.R[o] = e.R;
                }
                if (bwd) {
                    cs.dL[o] = e.dL;
                    cs.dR[o] = e.dR;
                    cs.px[o] = (r << 16) | px;
                    cs.src[o] = slot;
                }
            }
        }
        return;
    }
    const int kbits = uniform(R * cpi > 1 ? 32 - __clz(R * cpi - 1) : 0);
    for (int i0 = 0; wave + nw * i0 < g.Wp; i0 += cpi) {
        const int px = wave + nw * (i0 + lsub);
        const bool cell_ok = lsub < cpi && px < g.Wp;
        for (int j0 = 0; j0 < g.PC; j0 += kWave) {
            const int j = j0 + lj;
            Event e{-1, 0.f, 0.f, 0.f, 0.f};
            int f = -1;
            if (cell_ok && j < g.PC) {
                e = bin_event(C, t_at(px, j));
                const int64_t k = rb + static_cast<int64_t>(px) * g.PC + j;
                if (ev.row) {
                    // (L, R) are read only where the row is >= 0
                    ev.row[k] = e.row;
                    if (e.row >= 0) {
                        ev.L[k] = e.L;
                        ev.R[k] = e.R;
                    }
                }
                if (e.row >= 0) f = e.row * g.Wp + px;
            }
            const int kb = (f >= 0) ? e.row * cpi + lsub : 0;
            uint64_t same = __ballot(f >= 0);
            for (int bit = 0; bit < kbits; ++bit) {
                const bool on = (kb >> bit) & 1;
                const uint64_t bal = __ballot(on);
                same &= on ? bal : ~bal;
            }
            int pos = 0;
            if (f >= 0) {
                const int base = hist[f];
                pos = base + __popcll(same & below);
                if ((same >> lane) == 1ull) hist[f] = base + __popcll(same);
            }
            __builtin_amdgcn_wave_barrier();
            if (f >= 0) {
                const int64_t o = rb + pos;
                cs.key[o] = px * g.C_in + (j - fdiv(j, g.dv_cin) * g.C_in);
                if (fwd) {
                    cs.L[o] = e.L;
                    cs.R[o] = e.R;
                }
                if (bwd) {
                    cs.dL[o] = e.dL;
                    cs.dR[o] = e.dR;
                    cs.px[o] = (e.row << 16) | px;
                    cs.src[o] = px * g.PC + j;
                }
            }
        }
    }
}

// The events of one cell row without the sort (dW wanted, dt_in not), read
// in NCHW order.
__device__ void events_cell_row(const LifConst &C, const ConvGeom &g,
                                const float *__restrict__ t_in, const CellEv &ev, int cr) {
    const int b = cr / g.Hp, py = cr % g.Hp;
    const int per = g.Wp * g.PC;
    const int64_t rb = static_cast<int64_t>(cr) * per;
    bool has = false;
    for (int t = threadIdx.x; t < per; t += blockDim.x) {
        int slot;
        const int64_t src = cell_row_input(g, b, py, t, slot);
        const Event e = bin_event(C, t_in[src]);
        ev.row[rb + slot] = e.row;
        if (e.row >= 0) {  // (L, R) are read only where the row is >= 0
            ev.L[rb + slot] = e.L;
            ev.R[rb + slot] = e.R;
        }
        has = has || e.row >= 0;
    }
    has = __syncthreads_or(has);
    if (threadIdx.x == 0) ev.live[cr] = has;
}

// ------------------------------------------------------ weight layout ----
// WT[(k * C_in + ci) * C_out + co] = W[co, ci, k] / P (k = ky*KW + kx): W seen
// as [C_out][C_in * KT] (u = ci * KT + k) is transposed in 32 x 32 tiles
// through LDS (reads along u and writes along co coalesced); block blk takes
// tile (co0, u0) = ((blk / ntu) * 32, (blk % ntu) * 32).
constexpr int kWtLdsBytes = 32 * 33 * static_cast<int>(sizeof(float));

__host__ __device__ __forceinline__ int64_t weight_tiles(const ConvGeom &g) {
    const int64_t nu = static_cast<int64_t>(g.C_in) * g.KH * g.KW;
    return ((nu + 31) / 32) * ((g.C_out + 31) / 32);
}

template <typename WT>
__device__ void weights_block(const ConvGeom &g, const WT *__restrict__ W, float *__restrict__ out,
                              int64_t blk, float (*buf)[33]) {
    const int KT = g.KH * g.KW;
    const int NU = g.C_in * KT;
    const int ntu = (NU + 31) / 32;
    const int u0 = static_cast<int>(blk % ntu) * 32, c0 = static_cast<int>(blk / ntu) * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int r = ty; r < 32; r += blockDim.x >> 5) {
        const int co = c0 + r, u = u0 + tx;
        if (co < g.C_out && u < NU) buf[r][tx] = WLoad<WT>::get(W, static_cast<int64_t>(co) * NU + u);
    }
    __syncthreads();
    for (int r = ty; r < 32; r += blockDim.x >> 5) {
        const int u = u0 + r, co = c0 + tx;
        if (u < NU && co < g.C_out) {
            const int ci = u / KT, k = u % KT;
            out[(static_cast<int64_t>(k) * g.C_in + ci) * g.C_out + co] = buf[tx][r] * g.inv_P;
        }
    }
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

    // geometry of position p (no memory reads)
    __device__ __forceinline__ void init(const LifConst &C, const ConvGeom &g, int64_t p) {
        const int HoWo = g.Ho * g.Wo;
        const int pi = static_cast<int>(p);  // B * Ho * Wo < 2^31 (checked at the boundary)
        b = uniform(pi / HoWo);
        pos = uniform(pi % HoWo);
        const int oy = pos / g.Wo, ox = pos % g.Wo;
        x0 = ox * g.stride - g.pad;
        xa = max(0, x0);
        xb = max(xa, min(g.Wp, x0 + g.KW));
        nb1 = conv_off_stride(rows_of(C), g);
        wlim = g.KH * g.KW * g.C_in - 1;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int py = oy * g.stride - g.pad + ky;
            vky[ky] = ky < g.KH && py >= 0 && py < g.Hp && xa < xb;
            const int64_t cr = static_cast<int64_t>(b) * g.Hp + (vky[ky] ? py : 0);
            recb[ky] = cr * g.Wp * g.PC;
            offb[ky] = cr * nb1;
            wofs[ky] = (ky * g.KW - x0) * g.C_in;
        }
    }

    // the number of records in the KH cell rows (0: nothing to read)
    __device__ __forceinline__ int cell_records(const ConvSorted &cs) const {
        int any = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky)
            if (vky[ky]) any += *as_const(cs.off + offb[ky] + nb1 - 1);
        return any;
    }

    __device__ __forceinline__ void load_offs(const ConvGeom &g, const ConvSorted &cs, int R,
                                              int r0, int lane) {
        const int r = min(r0 + lane, R - 1);
        // bucket starts are clamped to the cell row's slots (a backward that
        // reuses a kept forward sort trusts workspace contents); lanes read
        // one column of the table each, contiguously
        const int per = g.Wp * g.PC;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int *o = cs.off + offb[ky] + r;
            oa[ky] = vky[ky] ? min(max(o[xa * R], 0), per) : 0;
            ob[ky] = vky[ky] ? min(max(o[xb * R], oa[ky]), per) : 0;
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
// The position's records, in the order the sums need them (event row, then
// kernel row, then bucket order), form a virtual list: lanes = event rows
// hold the KH segment bounds of their row and an exclusive prefix of the
// row counts; for 64 list entries at a time each lane finds its entry's row
// (binary search over the prefix with lane shuffles), its segment and its
// record, and loads the record's fields with one vector load each; the
// decoded entries (weight-row offset, row, L, R) go to a small LDS area of
// the wave. The entries are then summed in batches of up to 8 entries of one
// event row (each entry read back as one 16-byte LDS broadcast, the batch's
// weight rows loaded together), and rows close into the interval scan as the
// row changes. Sums and their order are those of a row-by-row walk.
struct FwdEntry { int wb, row; float L, R; };
// kDirect (receptive fields of at most 64 raw inputs, at most 64 event rows,
// pooled or plain input): no cell-row sort; lane v takes raw input
// v = ((ky * KW + kx) * P + d) * C_in + ci of the receptive field, bins its
// spike time itself, and the lanes are ranked by event row (stable in v, so
// within a row the order is kernel row, cell column, input slot: the sorted
// walk's order) from ballots of the row's bits; the ranked entries go to the
// same LDS list as one chunk of the walk.
// A block takes kFwdWaves consecutive output positions of one 64-channel
// tile, one per wave. Before its own position, every wave of the sorted walk
// makes the same block-level test from scalar loads (no barrier): where the
// block's positions lie in one image and the cell rows their receptive
// fields span hold no records at all, the waves write the block's silent
// outputs together, as runs of kFwdWaves consecutive positions per channel,
// instead of 64 single floats 4 * Ho * Wo bytes apart per position (such
// scattered stores bound the forward of layers without input events).
// (At most 72 VGPRs, seven waves per SIMD, where that needs no spill: conv9
// 0.819 -> 0.795 ms against six; else at most 80. Eight would spill.)
constexpr int kFwdWaves = 4;
template <int KHT, int KS, bool kDirect>
constexpr int fwd_min_waves() {
    return (KHT <= 3 && (kDirect || KS != kAnyKind)) ? 7 : 6;
}
template <int KHT, int KS, bool kDirect>
__global__ __launch_bounds__(kFwdWaves * kWave) __attribute__((amdgpu_waves_per_eu(fwd_min_waves<KHT, KS, kDirect>(), 8))) void conv_fwd_kernel(LifConst C, ConvGeom g, int64_t n_pos,
                                                       const float *__restrict__ Wt,
                                                       ConvSorted cs, const float *__restrict__ t_in,
                                                       float *__restrict__ t_out,
                                                       float *__restrict__ slope,
                                                       int *__restrict__ q_idx, int pre) {
    // a wave's list, padded so that a batch starting at any entry stays inside
    __shared__ FwdEntry ent[kFwdWaves][kWave + kCBatch];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int64_t p0 = static_cast<int64_t>(xcd_block(blockIdx.x, gridDim.x)) * kFwdWaves;
    const int64_t p = p0 + wave;
    const int HoWo = g.Ho * g.Wo;
    if constexpr (!kDirect) {
        // positions p0 .. pl (p0 < n_pos: the grid holds no empty block);
        // B * Ho * Wo < 2^31 (checked at the boundary)
        const int q0 = static_cast<int>(p0), ql = static_cast<int>(min(p0 + kFwdWaves, n_pos) - 1);
        const int b0 = q0 / HoWo;
        if (b0 == ql / HoWo) {
            const int y_lo = max(0, (q0 - b0 * HoWo) / g.Wo * g.stride - g.pad);
            const int y_hi = min(g.Hp - 1, (ql - b0 * HoWo) / g.Wo * g.stride - g.pad + g.KH - 1);
            const int nb1 = conv_off_stride(rows_of(C), g);
            int recs = 0;
            for (int y = y_lo; y <= y_hi; ++y)
                recs |= *as_const(cs.off + (static_cast<int64_t>(b0) * g.Hp + y) * nb1 + nb1 - 1);
            if (recs == 0) {
                // element e = wave * 64 + lane: channel e / kFwdWaves,
                // position e % kFwdWaves
                const int e = wave * kWave + lane;
                const int64_t ps = p0 + e % kFwdWaves;
                const int o = blockIdx.y * kWave + e / kFwdWaves;
                if (ps < n_pos && o < g.C_out) {
                    const int pi = static_cast<int>(ps);
                    const int bb = pi / HoWo;
                    const int64_t idx = (static_cast<int64_t>(bb) * g.C_out + o) * HoWo + (pi - bb * HoWo);
                    t_out[idx] = INFINITY;
                    slope[idx] = 0.f;
                    q_idx[idx] = -1;
                }
                return;
            }
        }
    }
    if (p >= n_pos) return;  // wave-uniform; no block barrier below
    FwdEntry *my = ent[wave];
    if (lane < kCBatch) my[kWave + lane] = FwdEntry{0, 0, 0.f, 0.f};
    const int co = blockIdx.y * kWave + lane;
    const bool row_ok = co < g.C_out;
    const int R = rows_of(C);
    PosWalk<KHT> wk;
    wk.init(C, g, p);
    const int64_t o_out = (static_cast<int64_t>(wk.b) * g.C_out + co) * HoWo + wk.pos;
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(
        Wt, static_cast<uint32_t>(static_cast<int64_t>(wk.wlim + 1) * g.C_out * sizeof(float)));
    const int voff = (row_ok ? co : 0) * static_cast<int>(sizeof(float));
    const int rstride = g.C_out * static_cast<int>(sizeof(float));
    Scan<KS> sc;
    float aL = 0.f, aR = 0.f, carry = 0.f;
    int cur = 0;  // row being summed
    // close rows cur .. target-1: point r-1 gets row r's L sums plus row
    // r-1's R sums. A record's row is at most R-2, so closing up to it never
    // reaches grid point M (the last interval, tested only at the end).
    auto close_to_mid = [&](int target) {
        while (cur < target) {
            if (cur >= 1) sc.template step_k<false>(C, cur - 1, aL + carry);
            carry = aR;
            aL = 0.f;
            aR = 0.f;
            ++cur;
        }
    };
    auto close_to_end = [&](int target) {
        while (cur < target) {
            if (cur >= 1) sc.step(C, cur - 1, aL + carry);
            carry = aR;
            aL = 0.f;
            aR = 0.f;
            ++cur;
        }
    };
    // (direct path) the sums of a batch of nk <= kCBatch list entries in
    // order; true once every lane has found its interval. A full batch inside
    // one event row (rows never decrease along the list) is summed without
    // per-entry tests.
    auto sum_batch = [&](const FwdEntry (&e)[kCBatch], const float (&w)[kCBatch], int nk) {
        const int ra = uniform(e[0].row);
        if (nk == kCBatch && ra == uniform(e[kCBatch - 1].row)) {
            if (ra != cur) {
                close_to_mid(ra);
                if (__all(sc.found() || !row_ok)) return true;
            }
#pragma unroll
            for (int q = 0; q < kCBatch; ++q) {
                aL = fmaf(w[q], e[q].L, aL);
                aR = fmaf(w[q], e[q].R, aR);
            }
            return false;
        }
#pragma unroll
        for (int q = 0; q < kCBatch; ++q) {
            if (q < nk) {
                const int row = uniform(e[q].row);
                if (row != cur) {
                    close_to_mid(row);
                    if (__all(sc.found() || !row_ok)) return true;
                }
                aL = fmaf(w[q], e[q].L, aL);
                aR = fmaf(w[q], e[q].R, aR);
            }
        }
        return false;
    };
    bool done = false, started = false;
    if constexpr (kDirect) {
        const int F = g.KH * g.KW * g.PC;
        bool has = false;
        FwdEntry me{0, -1, 0.f, 0.f};
        if (lane < F) {
            int wrow;
            const int64_t src = rf_input(g, wk.b, (wk.pos / g.Wo) * g.stride - g.pad, wk.x0,
                                         lane, wrow);
            if (src >= 0) {
                if (pre) {  // binned once per input by the set-up launch
                    const int r = cs.key[src];
                    const float Lv = cs.L[src], Rv = cs.R[src];
                    if (r >= 0) {
                        has = true;
                        me = FwdEntry{wrow * rstride, r, Lv, Rv};
                    }
                } else {
                    const Event e = bin_event<KS>(C, t_in[src]);
                    if (e.row >= 0) {
                        has = true;
                        me = FwdEntry{wrow * rstride, e.row, e.L, e.R};
                    }
                }
            }
        }
        const uint64_t hm = __ballot(has);
        const int total = __popcll(hm);
        if (total == 0) {  // no events in the receptive field: silent
            if (row_ok) {
                t_out[o_out] = INFINITY;
                slope[o_out] = 0.f;
                q_idx[o_out] = -1;
            }
            return;
        }
        // stable rank by event row: lanes with a smaller row, then lanes
        // with the same row and a lower index
        uint64_t lt = 0, eq = hm;
        const int kbits = uniform(32 - __clz(max(R - 2, 1)));
        for (int bit = kbits - 1; bit >= 0; --bit) {
            const bool on = has && ((me.row >> bit) & 1);
            const uint64_t bal = __ballot(on);
            if (on) lt |= eq & ~bal;
            eq &= on ? bal : (hm & ~bal);
        }
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        if (has) my[__popcll(lt) + __popcll(eq & below)] = me;
        __builtin_amdgcn_wave_barrier();
        cur = uniform(my[0].row);  // the scan starts at the first row with records
        started = true;
        for (int s0 = 0; s0 < total; s0 += kCBatch) {
            FwdEntry e[kCBatch];
            float w[kCBatch];
#pragma unroll
            for (int q = 0; q < kCBatch; ++q) e[q] = my[s0 + q];  // LDS broadcasts
#pragma unroll
            for (int q = 0; q < kCBatch; ++q) w[q] = BufLoad<float>::get(wr, voff + e[q].wb, 0);
            if (sum_batch(e, w, min(kCBatch, total - s0))) {
                done = true;
                break;
            }
        }
    } else {
    // the KH cell rows' record counts (scalar loads) rule out most positions
    // without events in their receptive field before any vector load
    if (wk.cell_records(cs) == 0) {
        if (row_ok) {
            t_out[o_out] = INFINITY;
            slope[o_out] = 0.f;
            q_idx[o_out] = -1;
        }
        return;
    }
    for (int r0 = 0; r0 <= R - 2 && !done; r0 += kWave) {
        wk.load_offs(g, cs, R, r0, lane);
        const bool rvalid = r0 + lane <= R - 2;
        int n0[KHT];
        int nr = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            n0[ky] = rvalid ? wk.ob[ky] - wk.oa[ky] : 0;
            nr += n0[ky];
        }
        int inc = nr;
#pragma unroll
        for (int m = 1; m < kWave; m <<= 1) {
            const int o = __shfl_up(inc, m);
            if (lane >= m) inc += o;
        }
        const int start = inc - nr;
        const int start_eff = rvalid ? start : 0x7fffffff;
        const int total = uniform(__builtin_amdgcn_readlane(inc, kWave - 1));
        if (!started && total > 0) {
            // rows before the first one with records add nothing to a zero
            // state: the scan starts there
            cur = r0 + __ffsll(static_cast<unsigned long long>(__ballot(nr > 0))) - 1;
            started = true;
        }
        for (int c0 = 0; c0 < total && !done; c0 += kWave) {
            const int v = c0 + lane;
            const bool rec_ok = v < total;
            // row lane lo: the last row whose prefix start is <= v
            int lo = 0;
#pragma unroll
            for (int step = kWave / 2; step >= 1; step >>= 1) {
                const int cand = lo + step;
                const int sv = __shfl(start_eff, cand & (kWave - 1));
                if (cand < kWave && sv <= v) lo = cand;
            }
            int kk = v - __shfl(start, lo);
            int sel = -1, ridx = 0;
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                const int a = __shfl(wk.oa[ky], lo), nn = __shfl(n0[ky], lo);
                if (sel < 0) {
                    if (kk < nn) {
                        sel = ky;
                        ridx = a + kk;
                    } else {
                        kk -= nn;
                    }
                }
            }
            int64_t gi = 0;
            int wof = 0;
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                if (sel == ky) {
                    gi = wk.recb[ky] + ridx;
                    wof = wk.wofs[ky];
                }
            }
            const bool ok = rec_ok && sel >= 0;
            const int key = ok ? cs.key[gi] : 0;
            const float Lv = ok ? cs.L[gi] : 0.f;
            const float Rv = ok ? cs.R[gi] : 0.f;
            const int wb = min(max(key + wof, 0), wk.wlim) * rstride;
            // the entry's row, and how many entries of that row the list holds
            // from this one on (itself included): row | nrem << 16 (rows < 2^16)
            const int nrem = min(__shfl(inc, lo) - v, kWave);
            my[lane] = FwdEntry{wb, (r0 + lo) | (nrem << 16), Lv, Rv};
            __builtin_amdgcn_wave_barrier();
            const int nc = min(kWave, total - c0);
            // batches never cross a row: up to kCBatch entries of the head
            // entry's row, summed without per-entry row tests; a batch's
            // entries past its row are read (and their weights loaded) but
            // not summed
            for (int s0 = 0; s0 < nc;) {
                FwdEntry e[kCBatch];
                float w[kCBatch];
#pragma unroll
                for (int q = 0; q < kCBatch; ++q) e[q] = my[s0 + q];  // LDS broadcasts
#pragma unroll
                for (int q = 0; q < kCBatch; ++q) w[q] = BufLoad<float>::get(wr, voff + e[q].wb, 0);
                const int hd = uniform(e[0].row);
                const int ra = hd & 0xffff;
                const int nk = max(1, min(min(kCBatch, hd >> 16), nc - s0));  // always advances
                if (ra != cur) {
                    close_to_mid(ra);
                    if (__all(sc.found() || !row_ok)) {
                        done = true;
                        break;
                    }
                }
                if (nk == kCBatch) {
#pragma unroll
                    for (int q = 0; q < kCBatch; ++q) {
                        aL = fmaf(w[q], e[q].L, aL);
                        aR = fmaf(w[q], e[q].R, aR);
                    }
                } else {
#pragma unroll
                    for (int q = 0; q < kCBatch - 1; ++q) {
                        if (q < nk) {
                            aL = fmaf(w[q], e[q].L, aL);
                            aR = fmaf(w[q], e[q].R, aR);
                        }
                    }
                }
                s0 += nk;
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
    }  // kDirect
    if (!started) {  // no events in the receptive field: silent
        if (row_ok) {
            t_out[o_out] = INFINITY;
            slope[o_out] = 0.f;
            q_idx[o_out] = -1;
        }
        return;
    }
    if (!done) {
        // the last row's sums reach grid points cur-1 and cur; after them no
        // input arrives: the rest of the window is one free-decay segment
        close_to_end(min(cur + 2, R - 1));
        if (cur < R - 1) sc.tail(C, cur - 1);
    }
    if (!row_ok) return;
    float to, sl;
    int q;
    sc.finish(C, to, sl, q);
    t_out[o_out] = to;
    slope[o_out] = sl;
    q_idx[o_out] = q;
}

// NP output positions per wave, LP = 64 / NP lanes each (one channel per
// lane; with NP = 1 a grid row per 64-channel tile). Needs at most LP event
// rows (R - 1 <= LP) and at most kListMaxRec raw inputs per receptive field
// (E = KH * KW * PC). Each position's lanes decode its records -- in the
// order of the chunked walk: event row, kernel row, bucket order -- into the
// wave's LDS list; then the positions sum the event rows in lockstep, one row
// at a time (a position with fewer records in the row adds zero-weight
// entries, which leave its sums unchanged), and close each row into the
// interval scan together, so the scan runs on all 64 lanes and the row
// structure needs no per-record test. Every neuron's sums and their order
// are those of the chunked walk.
constexpr int kListMaxRec = 640;

// LDS ints of one wave's list of ne records: the weight rows as 16-bit
// indices (a list layer's receptive field has at most kListMaxRec / 2 raw
// inputs, so its weight rows fit), then the (L, R) pairs, 8-byte aligned
__host__ __device__ __forceinline__ int list_wave_ints(int ne) {
    const int ne4 = (ne + 3) & ~3;
    return ne4 / 2 + 2 * ne4;
}

// K consecutive records of a row from the LDS list at idx, of which the lane's
// position has `left` (entries past them add zero weight): weights loaded as
// one batch, then summed in order. kFull: every position of the wave has all
// K (no masking).
template <int K, bool kFull = false>
__device__ __forceinline__ void list_batch(const uint16_t *erow, const float2 *eLR, int idx,
                                           int left, __amdgpu_buffer_rsrc_t wr, int voff,
                                           int rstride, float &aL, float &aR) {
    int wb[K];
    float Lq[K], Rq[K], w[K];
#pragma unroll
    for (int q = 0; q < K; ++q) {
        const bool ok = kFull || q < left;
        wb[q] = ok ? static_cast<int>(__umul24(erow[idx + q], rstride)) : 0;  // both < 2^24
        const float2 lr = ok ? eLR[idx + q] : make_float2(0.f, 0.f);
        Lq[q] = lr.x;
        Rq[q] = lr.y;
    }
#pragma unroll
    for (int q = 0; q < K; ++q) w[q] = BufLoad<float>::get(wr, voff + wb[q], 0);
#pragma unroll
    for (int q = 0; q < K; ++q) {
        aL = fmaf(w[q], Lq[q], aL);
        aR = fmaf(w[q], Rq[q], aR);
    }
}

// kDirect (E <= LP): as in the chunked walk, no cell-row sort: lane li of a
// position takes raw input li of its receptive field and bins it; the row
// counts come from LDS integer atomics, and each record's place in its row
// from ballots of the row bits (stable in li: the sorted walk's order).
template <int KHT, int KS, int NP, bool kDirect>
__global__ __launch_bounds__(256) void conv_fwd_list_kernel(LifConst C, ConvGeom g, int64_t n_pos,
                                                            const float *__restrict__ Wt,
                                                            ConvSorted cs,
                                                            const float *__restrict__ t_in,
                                                            float *__restrict__ t_out,
                                                            float *__restrict__ slope,
                                                            int *__restrict__ q_idx, int pre) {
    constexpr int LP = kWave / NP;
    extern __shared__ int list_lds[];  // per wave: weight rows [NP][E] (16-bit), then (L, R)[NP][E]
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int half = lane / LP, li = lane % LP, hb = half * LP;  // hb: the position's first lane
    const int nwb = blockDim.x >> 6;
    const int64_t pb = static_cast<int64_t>(xcd_block(blockIdx.x, gridDim.x)) * nwb * NP;
    const int64_t p0 = pb + wave * NP;
    if constexpr (!kDirect) {
        // the block's positions pb .. (nwb * NP of them; pb < n_pos): where
        // they lie in one image and the cell rows their receptive fields span
        // hold no records, the waves write the block's silent outputs
        // together, as runs of nwb * NP positions per channel (the same test
        // in every wave, from scalar loads: no barrier)
        const int HoWo = g.Ho * g.Wo, npb = nwb * NP;
        const int q0 = static_cast<int>(pb), ql = static_cast<int>(min(pb + npb, n_pos) - 1);
        const int b0 = q0 / HoWo;
        if (b0 == ql / HoWo) {
            const int y_lo = max(0, (q0 - b0 * HoWo) / g.Wo * g.stride - g.pad);
            const int y_hi = min(g.Hp - 1, (ql - b0 * HoWo) / g.Wo * g.stride - g.pad + g.KH - 1);
            const int nb1 = conv_off_stride(rows_of(C), g);
            int recs = 0;
            for (int y = y_lo; y <= y_hi; ++y)
                recs |= *as_const(cs.off + (static_cast<int64_t>(b0) * g.Hp + y) * nb1 + nb1 - 1);
            if (recs == 0) {
                // element e = wave * 64 + lane: channel e / npb, position e % npb
                for (int e = wave * kWave + lane; e < npb * LP; e += static_cast<int>(blockDim.x)) {
                    const int64_t ps = pb + e % npb;
                    const int o = blockIdx.y * LP + e / npb;
                    if (ps < n_pos && o < g.C_out) {
                        const int pi = static_cast<int>(ps);
                        const int bb = pi / HoWo;
                        const int64_t idx = (static_cast<int64_t>(bb) * g.C_out + o) * HoWo + (pi - bb * HoWo);
                        t_out[idx] = INFINITY;
                        slope[idx] = 0.f;
                        q_idx[idx] = -1;
                    }
                }
                return;
            }
        }
    }
    if (p0 >= n_pos) return;  // wave-uniform; no block barrier below
    const int64_t p = p0 + half;
    const bool pos_ok = p < n_pos;
    const int E = g.KH * g.KW * g.PC;
    const int ebase = half * E;  // the position's part of the wave's list
    const int WI = list_wave_ints(NP * E);
    uint16_t *erow = reinterpret_cast<uint16_t *>(list_lds + wave * WI);
    // (L, R) of a record: one 8-byte read
    float2 *eLR = reinterpret_cast<float2 *>(list_lds + wave * WI + ((NP * E + 3) & ~3) / 2);
    const int co = blockIdx.y * LP + li;
    const bool row_ok = pos_ok && co < g.C_out;
    const int HoWo = g.Ho * g.Wo;
    const int R = rows_of(C);
    const int64_t pp = pos_ok ? p : p0;
    const int b = static_cast<int>(pp) / HoWo, pos = static_cast<int>(pp) % HoWo;
    const int oy = pos / g.Wo, ox = pos % g.Wo;
    const int x0 = ox * g.stride - g.pad;
    const int xa = max(0, x0), xb = max(xa, min(g.Wp, x0 + g.KW));
    const int nb1 = conv_off_stride(R, g);
    const int wlim = g.KH * g.KW * g.C_in - 1;
    int64_t recb[KHT], offb[KHT];
    int wofs[KHT];
    bool vky[KHT];
    const int64_t o_out = (static_cast<int64_t>(b) * g.C_out + co) * HoWo + pos;
    auto write_silent = [&]() {
        if (row_ok) {
            t_out[o_out] = INFINITY;
            slope[o_out] = 0.f;
            q_idx[o_out] = -1;
        }
    };
    // lane li of a position = its event row li: the row's record count (and
    // on the sorted path its segment bounds), then an exclusive prefix of
    // the counts within the position's lanes
    const bool rvalid = li <= R - 2;
    int oa[KHT], n0[KHT];
    int nr = 0;
    // direct path: this lane's own record
    bool dhas = false;
    int drow = 0, dwb = 0;
    float2 dlr = make_float2(0.f, 0.f);
    if constexpr (kDirect) {
        int *hist = list_lds + (blockDim.x >> 6) * WI + wave * kWave;  // [NP][LP] row counts
        hist[lane] = 0;
        __builtin_amdgcn_wave_barrier();
        if (pos_ok && li < E) {
            int wrow;
            const int64_t src = rf_input(g, b, oy * g.stride - g.pad, x0, li, wrow);
            if (src >= 0) {
                int r;
                float Lv, Rv;
                if (pre) {  // binned once per input by the set-up launch
                    r = cs.key[src];
                    Lv = cs.L[src];
                    Rv = cs.R[src];
                } else {
                    const Event e = bin_event<KS>(C, t_in[src]);
                    r = e.row;
                    Lv = e.L;
                    Rv = e.R;
                }
                if (r >= 0) {
                    dhas = true;
                    drow = r;
                    dwb = wrow;  // weight row
                    dlr = make_float2(Lv, Rv);
                    atomicAdd(&hist[hb + r], 1);
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (!__any(dhas)) {  // no events in any receptive field
            write_silent();
            return;
        }
        nr = rvalid ? hist[lane] : 0;
    } else {
        int any = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int py = oy * g.stride - g.pad + ky;
            vky[ky] = pos_ok && ky < g.KH && py >= 0 && py < g.Hp && xa < xb;
            const int64_t cr = static_cast<int64_t>(b) * g.Hp + (vky[ky] ? py : 0);
            recb[ky] = cr * g.Wp * g.PC;
            offb[ky] = cr * nb1;
            wofs[ky] = (ky * g.KW - x0) * g.C_in;
            if (vky[ky]) any += cs.off[offb[ky] + nb1 - 1];
        }
        if (!__any(any > 0)) {  // no receptive field's cell rows hold records
            write_silent();
            return;
        }
        const int rr = min(li, R - 2);
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int *o = cs.off + offb[ky] + rr;
            const int a = vky[ky] ? o[xa * R] : 0, e = vky[ky] ? o[xb * R] : 0;
            oa[ky] = a;
            n0[ky] = rvalid ? e - a : 0;
            nr += n0[ky];
        }
    }
    int inc = nr;
#pragma unroll
    for (int m = 1; m < LP; m <<= 1) {
        const int o = __shfl_up(inc, m, LP);
        if (li >= m) inc += o;
    }
    const int start = inc - nr;
    const int start_eff = rvalid ? start : 0x7fffffff;
    int tot = 0, tmax = 0;
#pragma unroll
    for (int h = 0; h < NP; ++h) {
        const int th = uniform(__builtin_amdgcn_readlane(inc, h * LP + LP - 1));
        if (h == half) tot = th;
        tmax = max(tmax, th);
    }
    const int rstride = g.C_out * static_cast<int>(sizeof(float));
    if constexpr (kDirect) {
        // place = the row's start + the records of the same row in lower lanes
        const uint64_t half_mask = (((1ull << (LP - 1)) << 1) - 1) << hb;
        const uint64_t hm = __ballot(dhas) & half_mask;
        uint64_t eq = hm;
        const int kbits = uniform(32 - __clz(max(R - 2, 1)));
        for (int bit = 0; bit < kbits; ++bit) {
            const bool on = dhas && ((drow >> bit) & 1);
            const uint64_t bal = __ballot(on);
            eq &= on ? bal : (hm & ~bal);
        }
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        const int rs = __shfl(start, hb + (dhas ? drow : 0));
        if (dhas) {
            const int at = ebase + rs + __popcll(eq & below);
            erow[at] = static_cast<uint16_t>(dwb);
            eLR[at] = dlr;
        }
    } else
    // decode LP records per position at a time into the LDS list
    for (int c0 = 0; c0 < tmax; c0 += LP) {
        const int v = c0 + li;
        int lo = 0;  // the position's last row whose start is <= v
#pragma unroll
        for (int step = LP / 2; step >= 1; step >>= 1) {
            const int cand = lo + step;
            const int sv = __shfl(start_eff, hb + (cand & (LP - 1)));
            if (cand < LP && sv <= v) lo = cand;
        }
        int kk = v - __shfl(start, hb + lo);
        int sel = -1, ridx = 0;
#pragma unroll
        for (int ky = 0; ky < KHT; ++ky) {
            const int a = __shfl(oa[ky], hb + lo), nn = __shfl(n0[ky], hb + lo);
            if (sel < 0) {
                if (kk < nn) {
                    sel = ky;
                    ridx = a + kk;
                } else {
                    kk -= nn;
                }
            }
        }
        if (v < tot && sel >= 0) {
            int64_t gi = 0;
            int wof = 0;
#pragma unroll
            for (int ky = 0; ky < KHT; ++ky) {
                if (sel == ky) {
                    gi = recb[ky] + ridx;
                    wof = wofs[ky];
                }
            }
            erow[ebase + v] = static_cast<uint16_t>(min(max(cs.key[gi] + wof, 0), wlim));
            eLR[ebase + v] = make_float2(cs.L[gi], cs.R[gi]);
        }
    }
    __builtin_amdgcn_wave_barrier();
    uint64_t rows_any = __ballot(nr > 0);
#pragma unroll
    for (int h = 1; h < NP; ++h) rows_any |= rows_any >> (h * LP);
    if (NP > 1) rows_any &= (1ull << LP) - 1;
    if (rows_any == 0) {  // no records in any receptive field
        write_silent();
        return;
    }
    // rows before the first one with records add nothing to a zero state
    const int r_first = __ffsll(static_cast<unsigned long long>(rows_any)) - 1;
    const int r_last = 63 - __clzll(static_cast<long long>(rows_any));
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(
        Wt, static_cast<uint32_t>(static_cast<int64_t>(wlim + 1) * g.C_out * sizeof(float)));
    const int voff = (row_ok ? co : 0) * static_cast<int>(sizeof(float));
    Scan<KS> sc;
    float aL = 0.f, aR = 0.f, carry = 0.f;
    for (int r = r_first; r <= R - 2; ++r) {
        if (r <= r_last) {
            int n = 0, nmin = 0x7fffffff, my_n = 0, my_s = ebase;
#pragma unroll
            for (int h = 0; h < NP; ++h) {
                const int nh = uniform(__builtin_amdgcn_readlane(nr, h * LP + r));
                const int sh = uniform(__builtin_amdgcn_readlane(start, h * LP + r));
                n = max(n, nh);
                nmin = min(nmin, nh);
                if (h == half) {
                    my_n = nh;
                    my_s += sh;
                }
            }
            // batches of 8 (unmasked while every position has them), then
            // 4, then single records: no load or sum past the row's largest
            // count
            int i0 = 0;
            for (; i0 + 8 <= nmin; i0 += 8)
                list_batch<8, true>(erow, eLR, my_s + i0, my_n - i0, wr, voff, rstride, aL, aR);
            for (; i0 + 8 <= n; i0 += 8)
                list_batch<8>(erow, eLR, my_s + i0, my_n - i0, wr, voff, rstride, aL, aR);
            if (i0 + 4 <= n) {
                list_batch<4>(erow, eLR, my_s + i0, my_n - i0, wr, voff, rstride, aL, aR);
                i0 += 4;
            }
            for (; i0 < n; ++i0) list_batch<1>(erow, eLR, my_s + i0, my_n - i0, wr, voff, rstride, aL, aR);
        } else if (r == r_last + 2) {
            // every record is in: grid points r-1 .. M see no input, the rest
            // of the window is one free-decay segment
            sc.tail(C, r - 1);
            break;
        }
        // grid point r-1: this row's L sums plus the previous row's R sums
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
// Gradient triples (gamma, t - T_q, q) of grad_prep for kGradPos output
// positions s = b * Ho*Wo + p and one tile of kGradCh channels (block blk =
// position group * tiles + tile): read from the NCHW outputs with positions
// along the lanes, staged in LDS and written position-major [s][co] (each
// position's channels contiguous).
// rend[s] = min(R-2, max q + 1) over the channels of s that pass gradient
// (G[m] vanishes for m > q, and a record of event row r reads G[r-1] and
// G[r]), -1 if none does.
constexpr int kGradPos = 16, kGradCh = 64;
constexpr int kGradLdsBytes = (3 * kGradCh * (kGradPos + 1) + kGradPos) * 4;

__device__ void grad_block(const LifConst &C, const ConvGeom &g, int64_t n_pos, int64_t blk,
                           const float *__restrict__ t_out, const float *__restrict__ slope,
                           const int *__restrict__ q_idx, const float *__restrict__ grad_t,
                           const Synfire &sf, float *__restrict__ gam, float *__restrict__ uq,
                           int *__restrict__ qv, int *__restrict__ rend, int *sh) {
    constexpr int kS = kGradPos + 1;
    float *sg = reinterpret_cast<float *>(sh);
    float *su = sg + kGradCh * kS;
    int *sq = reinterpret_cast<int *>(su + kGradCh * kS);
    int *sl = sq + kGradCh * kS;
    const int HoWo = g.Ho * g.Wo;
    const int ntile = (g.C_out + kGradCh - 1) / kGradCh;
    const int tile = static_cast<int>(blk % ntile);
    const int64_t s0 = (blk / ntile) * kGradPos;
    if (threadIdx.x < kGradPos) sl[threadIdx.x] = -1;
    __syncthreads();
    // Only positions through which gradient passes are written (the dW and
    // dt_in kernels read no others); with more than one channel tile their
    // largest q over all channels is found first (by every tile's block).
    const bool tiles = ntile > 1;
    // each thread keeps one position (blockDim is a multiple of kGradPos):
    // its NCHW offset at channel 0, decoded once
    const int pl = static_cast<int>(threadIdx.x) % kGradPos;
    const int cstep = static_cast<int>(blockDim.x) / kGradPos;
    const bool pos_ok = s0 + pl < n_pos;
    int64_t obase = 0;
    if (pos_ok) {
        const int si = static_cast<int>(s0 + pl);  // B * Ho * Wo < 2^31 (checked at the boundary)
        const int b = si / HoWo;
        obase = static_cast<int64_t>(b) * g.C_out * HoWo + (si - b * HoWo);
    }
    if (tiles) {
        if (pos_ok) {
            // four channels per pass, their loads issued together
            for (int c4 = static_cast<int>(threadIdx.x) / kGradPos; c4 < g.C_out; c4 += 4 * cstep) {
                int q[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int co = c4 + u * cstep;
                    q[u] = (co < g.C_out) ? q_idx[obase + static_cast<int64_t>(co) * HoWo] : -1;
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (q[u] >= 0) {
                        const int64_t o = obase + static_cast<int64_t>(c4 + u * cstep) * HoWo;
                        float gt = grad_t[o];
                        if (sf.on) gt += synfire_dt(sf, t_out[o]);
                        if (gt != 0.f) atomicMax(&sl[pl], q[u]);
                    }
                }
            }
        }
        __syncthreads();
    }
    {
        // a thread's kCh channels of its position (256 threads: 16 positions
        // x 4 channel rows): each load stage is issued for all of them before
        // the next, so the dependent loads (q, then the upstream gradient,
        // then the spike time and slope) overlap across channels
        constexpr int kCh = kGradCh * kGradPos / 256;
        const int c0 = tile * kGradCh;
        const int cl0 = static_cast<int>(threadIdx.x) / kGradPos;
        int64_t o[kCh];
        int q[kCh];
        float gt[kCh];
        // with channel tiles the pass above found whether any channel of the
        // position passes gradient; a position without writes nothing
        const bool live = pos_ok && (!tiles || sl[pl] >= 0);
#pragma unroll
        for (int u = 0; u < kCh; ++u) {
            const int co = c0 + cl0 + u * cstep;
            o[u] = obase + static_cast<int64_t>(co) * HoWo;
            q[u] = (co < g.C_out && live) ? q_idx[o[u]] : -1;
        }
#pragma unroll
        for (int u = 0; u < kCh; ++u) gt[u] = (q[u] >= 0) ? grad_t[o[u]] : 0.f;  // silent: no load
#pragma unroll
        for (int u = 0; u < kCh; ++u) {
            GradPrep gp{0.f, 0.f, -1};
            if (q[u] >= 0) {
                // the spike time only where it is used (no gradient: no load)
                const float t = (sf.on || gt[u] != 0.f) ? t_out[o[u]] : 0.f;
                float gu = gt[u];
                if (sf.on) gu += synfire_dt(sf, t);
                if (gu != 0.f) gp = grad_prep(C, t, slope[o[u]], q[u], gu);
            }
            const int cl = cl0 + u * cstep;
            sg[cl * kS + pl] = gp.gam;
            su[cl * kS + pl] = gp.uq;
            sq[cl * kS + pl] = gp.q;
            if (!tiles && gp.q >= 0) atomicMax(&sl[pl], gp.q);
        }
        __syncthreads();
        for (int e = threadIdx.x; e < kGradPos * kGradCh; e += blockDim.x) {
            const int pw = e / kGradCh, cl = e % kGradCh;
            const int co = c0 + cl;
            const int64_t sp = s0 + pw;
            if (co < g.C_out && sp < n_pos && sl[pw] >= 0) {
                const int64_t d = sp * g.C_out + co;
                gam[d] = sg[cl * kS + pw];
                uq[d] = su[cl * kS + pw];
                qv[d] = sq[cl * kS + pw];
            }
        }
        __syncthreads();
    }
    if (rend && tile == 0 && threadIdx.x < kGradPos && s0 + threadIdx.x < n_pos) {
        const int qm = sl[threadIdx.x];
        rend[s0 + threadIdx.x] = qm < 0 ? -1 : min(rows_of(C) - 2, qm + 1);
    }
}

// Dead-neuron term of output channel co: dq[co] = -gamma_q * scale * (number
// of silent (b, position) outputs of the channel); integer counts, so the
// block sum is exact.
__device__ void dead_channel_block(const ConvGeom &g, int64_t B, const int *__restrict__ q_idx,
                                   const Synfire &sf, int co, int *sh) {
    const int HoWo = g.Ho * g.Wo;
    const int64_t n = B * HoWo;
    int cnt = 0;
    for (int64_t e = threadIdx.x; e < n; e += blockDim.x) {
        const int64_t b = e / HoWo;
        const int p = static_cast<int>(e % HoWo);
        cnt += (q_idx[(b * g.C_out + co) * HoWo + p] < 0) ? 1 : 0;
    }
    sh[threadIdx.x] = cnt;
    __syncthreads();
    for (int h = blockDim.x / 2; h > 0; h >>= 1) {
        if (static_cast<int>(threadIdx.x) < h) sh[threadIdx.x] += sh[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) sf.dq[co] = -(sf.gq * sf.scale * static_cast<float>(sh[0]));
}

// dt_in partials. Wave = output position; lane = output channel, NT tiles of
// 64 per lane. Rows stop after the last grid point any channel's G reaches.
// A block of 256 threads takes positions 4 * bx .. 4 * bx + 3.
template <int KHT, int NT, int KS>
__device__ __forceinline__ void dtp_block(const LifConst &C, const ConvGeom &g, int64_t n_pos,
                                          const float *__restrict__ Wt, const ConvSorted &cs,
                                          const float *__restrict__ gam,
                                          const float *__restrict__ uq,
                                          const int *__restrict__ qv,
                                          const int *__restrict__ rend, int64_t bx) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int64_t p = bx * 4 + wave;
    if (p >= n_pos) return;  // wave-uniform; no block barrier below
    const int r_end = *as_const(rend + p);  // rows r <= r_end need G[r-1], G[r]
    if (r_end < 0) return;                  // no channel here passes gradient
    const int R = rows_of(C);
    const int KT = g.KH * g.KW;
    PosWalk<KHT> wk;
    wk.init(C, g, p);
    if (wk.cell_records(cs) == 0) return;  // no records to receive gradient
    const int64_t nbase = (static_cast<int64_t>(wk.b) * g.Ho * g.Wo + wk.pos) * g.C_out;
    float gm[NT], ua[NT], gA[NT], gB[NT];
    int qa[NT], voff[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int co = t * kWave + lane;
        const int cc = min(co, g.C_out - 1);
        const bool ok = co < g.C_out;
        gm[t] = ok ? gam[nbase + cc] : 0.f;
        ua[t] = ok ? uq[nbase + cc] : 0.f;
        qa[t] = ok ? qv[nbase + cc] : -1;
        voff[t] = cc * static_cast<int>(sizeof(float));
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        gA[t] = 0.f;
        gB[t] = g_at<KS>(C, gm[t], ua[t], qa[t], 0);
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
                        const float dl = as_const(cs.dL + o)[kk], dr = as_const(cs.dR + o)[kk];
                        float acc = 0.f;
#pragma unroll
                        for (int t = 0; t < NT; ++t) {
                            const float w = BufLoad<float>::get(wr, voff[t], wo);
                            acc = fmaf(w, fmaf(dl, gA[t], dr * gB[t]), acc);
                        }
                        v[kk] = acc;
                    }
                    // channel sums: lane 8kk ends with record kk's total and
                    // stores it as the record's partial for its tap
                    static_assert(kCBatch == 8, "wave_sum8 reduces eight records");
                    const float tot = wave_sum8(v, lane);
                    const int kl = lane >> 3;
                    if ((lane & 7) == 0 && kl < nk) {
                        const int kx = min(max((cs.px[o + kl] & 0xffff) - wk.x0, 0), g.KW - 1);
                        cs.P[(o + kl) * KT + ky * g.KW + kx] = tot;
                    }
                }
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            gA[t] = gB[t];
            gB[t] = g_at<KS>(C, gm[t], ua[t], qa[t], r + 1);
        }
    }
}

template <int KHT, int NT, int KS>
__global__ __launch_bounds__(256) void conv_dtp_kernel(LifConst C, ConvGeom g, int64_t n_pos,
                                                       const float *__restrict__ Wt,
                                                       ConvSorted cs,
                                                       const float *__restrict__ gam,
                                                       const float *__restrict__ uq,
                                                       const int *__restrict__ qv,
                                                       const int *__restrict__ rend) {
    dtp_block<KHT, NT, KS>(C, g, n_pos, Wt, cs, gam, uq, qv, rend, blockIdx.x);
}

// dt_in of the raw inputs of cell row cr, slots [s0, s0 + ns) of its
// cell-major order (kGatherSlots at most; a block per slice). Each record
// sums its per-tap partials in tap order, taking only the taps through which
// an output position passed gradient to the record's event row (the entries
// the dt_in kernel wrote); the sums are staged in LDS at the record's slot,
// and the slice is written in NCHW order (inputs without events get 0), so
// consecutive threads write consecutive addresses.
constexpr int kGatherSlots = 4096;

__device__ void dt_gather_block(const ConvGeom &g, int R, const ConvSorted &cs,
                                const int *__restrict__ rend, float *__restrict__ dt_in, int cr,
                                int s0, float *buf) {
    const int per = g.Wp * g.PC;
    const int ns = min(kGatherSlots, per - s0);
    const int nb1 = conv_off_stride(R, g);
    const int nrec = uniform(min(max(cs.off[static_cast<int64_t>(cr) * nb1 + nb1 - 1], 0), per));
    const int b = cr / g.Hp, py = cr % g.Hp;
    const int64_t pos0 = static_cast<int64_t>(b) * g.Ho * g.Wo;
    // output rows oy whose kernel row ky = py + pad - oy * stride is in
    // range, walked with ky ascending (the tap order of the sum)
    const int ny0 = py + g.pad;
    const int oy_hi = min(g.Ho - 1, ny0 / g.stride);
    const int oy_lo = (max(0, ny0 - g.KH + 1) + g.stride - 1) / g.stride;
    // no record, or no output position of those rows passes gradient: the
    // cell row's dt_in is 0
    bool live = false;
    if (nrec > 0)
        for (int k = threadIdx.x; k < (oy_hi - oy_lo + 1) * g.Wo; k += blockDim.x)
            live = live || rend[pos0 + static_cast<int64_t>(oy_lo) * g.Wo + k] >= 0;
    if (!__syncthreads_or(live)) {
        for (int t = threadIdx.x; t < per; t += blockDim.x) {
            int slot;
            const int64_t dst = cell_row_input(g, b, py, t, slot);
            if (slot >= s0 && slot < s0 + ns) dt_in[dst] = 0.f;
        }
        return;
    }
    for (int t = threadIdx.x; t < ns; t += blockDim.x) buf[t] = 0.f;
    __syncthreads();
    const int64_t rb = static_cast<int64_t>(cr) * per;
    const int KT = g.KH * g.KW;
    for (int k = threadIdx.x; k < nrec; k += blockDim.x) {
        const int src = cs.src[rb + k];
        if (src < s0 || src >= s0 + ns) continue;
        const int pr = cs.px[rb + k];
        const int px = pr & 0xffff, row = pr >> 16;
        const int nx0 = px + g.pad;
        const int ox_hi = min(g.Wo - 1, nx0 / g.stride);
        const int ox_lo = (max(0, nx0 - g.KW + 1) + g.stride - 1) / g.stride;
        const float *P = cs.P + (rb + k) * KT;
        float acc = 0.f;
        for (int oy = oy_hi; oy >= oy_lo; --oy) {
            const int ky = ny0 - oy * g.stride;
            const int *rr = rend + pos0 + static_cast<int64_t>(oy) * g.Wo;
            for (int ox = ox_hi; ox >= ox_lo; --ox)
                if (row <= rr[ox]) acc += P[ky * g.KW + nx0 - ox * g.stride];
        }
        buf[src - s0] = acc;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < per; t += blockDim.x) {
        int slot;
        const int64_t dst = cell_row_input(g, b, py, t, slot);
        if (slot >= s0 && slot < s0 + ns) dt_in[dst] = buf[slot - s0];
    }
}

// dW[co, ci, k] = (1/P) sum_{b, p} sum_d (G[b, r, p, co] L + G[b, r+1, p, co] R)
// over the raw inputs d of the cell that tap k of position p reads.
// Lane = (k, ci); a block covers 256 of them and a tile of TI channels whose
// sums stay in registers over its share of the (b, p) samples. G[b, :, p,
// tile] is computed in place from (gamma, t - T_q, q) -- each thread owns one
// channel and a fixed set of rows; channels without gradient cost no
// exponential -- and staged in LDS as rows G[r][channel] of TI + 1 floats,
// double buffered (an event's two halves G[r][i], G[r+1][i] are TI + 1 dwords
// apart: one two-address LDS read; rows R-1 and R stay zero), the next
// sample's values in registers (NPER per thread) during this one's sums. A
// sample whose tile is all zero is skipped.
// Block (bx, by, bz): inputs 256 bx .., channel tile by, batch split bz.
// gs: the dynamic LDS ([2][R + 1][TI + 1], then the live sample list);
// n_live_w: four ints of LDS.
struct ConvDwArgs {
    int64_t n_samp;
    int s_per_split;
    const float *gam, *uq;
    const int *qv, *rend, *cr_live, *ev_row;
    const float *ev_L, *ev_R;
    float *part;
    int *zlive;
};
template <int TI, int NPER, int KS>
__device__ __forceinline__ void dw_block(const LifConst &C, const ConvGeom &g,
                                         const ConvDwArgs &a, int bx, int by, int bz,
                                         float *gs, int *n_live_w) {
    const int64_t n_samp = a.n_samp;
    const int s_per_split = a.s_per_split;
    const float *__restrict__ gam = a.gam;
    const float *__restrict__ uq = a.uq;
    const int *__restrict__ qv = a.qv;
    const int *__restrict__ rend = a.rend;
    const int *__restrict__ cr_live = a.cr_live;
    const int *__restrict__ ev_row = a.ev_row;
    const float *__restrict__ ev_L = a.ev_L;
    const float *__restrict__ ev_R = a.ev_R;
    constexpr int kStr = TI + 1;
    const int R = rows_of(C);
    const int gbuf = (R + 1) * kStr;
    const int NJ = g.KH * g.KW * g.C_in;
    const int jj = bx * 256 + threadIdx.x;
    const int co0 = by * TI;
    const int ni = min(TI, g.C_out - co0);
    const int64_t s_lo = static_cast<int64_t>(bz) * s_per_split;
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
    const GStep gst = g_step<KS>(C, kRowStep);
    float pre[NPER];
    // G[b, :, p, tile] of sample s; returns whether any value is nonzero
    auto fetch = [&](int64_t s) {
        const int64_t nb = s * g.C_out + co0 + min(l_own, ni - 1);
        const bool own = l_own < ni;
        const float gm = own ? gam[nb] : 0.f;
        const float u = own ? uq[nb] : 0.f;
        const int q = own ? qv[nb] : -1;
        g_strided<NPER, KS>(C, gst, gm, u, q, r_first - 1, kRowStep, pre);
        bool nz = false;
#pragma unroll
        for (int c = 0; c < NPER; ++c) nz = nz || pre[c] != 0.f;
        return nz;
    };
    auto store = [&](float *buf) {
#pragma unroll
        for (int c = 0; c < NPER; ++c) {
            const int kk = threadIdx.x + c * 256;
            if (kk < total) {
                const int r = kk / TI, l = kk % TI;
                if (r < R - 1) buf[r * kStr + l] = pre[c];
            }
        }
    };
    for (int t = threadIdx.x; t < 2 * 2 * kStr; t += 256)
        gs[(t / (2 * kStr)) * gbuf + (R - 1) * kStr + t % (2 * kStr)] = 0.f;
    // the split's samples through which any gradient flows, in order
    int *list = reinterpret_cast<int *>(gs + 2 * gbuf);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int n_live = 0;
    for (int64_t c0 = s_lo; c0 < s_hi; c0 += 256) {
        const int64_t sc = c0 + threadIdx.x;
        const bool f = sc < s_hi && rend[sc] >= 0;
        const uint64_t m = __ballot(f);
        if (lane == 0) n_live_w[wave] = __popcll(m);
        __syncthreads();
        int base = n_live;
        for (int w = 0; w < wave; ++w) base += n_live_w[w];
        if (f) list[base + __popcll(m & below)] = static_cast<int>(sc - s_lo);
        for (int w = 0; w < 4; ++w) n_live += n_live_w[w];
        __syncthreads();
    }
    // a split without such samples writes no partials (the reduction skips it)
    if (threadIdx.x == 0 && bx == 0 && by == 0) a.zlive[bz] = n_live > 0;
    if (n_live == 0) return;
    bool live = false;  // the staged sample's tile has a nonzero value
    {
        live = fetch(s_lo + list[0]);
        store(gs);
    }
    live = __syncthreads_or(live);
    for (int i = 0; i < n_live; ++i) {
        const int64_t s = s_lo + list[i];
        const float *cur = gs + (i & 1) * gbuf;
        const bool more = i + 1 < n_live;
        bool live_next = false;
        if (more) live_next = fetch(s_lo + list[i + 1]);
        if (live) {
            const int b = static_cast<int>(s) / HoWo, p = static_cast<int>(s) % HoWo;
            const int py = (p / g.Wo) * g.stride - g.pad + ky;
            const int px = (p % g.Wo) * g.stride - g.pad + kx;
            if (j_ok && py >= 0 && py < g.Hp && px >= 0 && px < g.Wp &&
                cr_live[static_cast<int64_t>(b) * g.Hp + py]) {
                const int64_t e0 = ((static_cast<int64_t>(b) * g.Hp + py) * g.Wp + px) * g.PC + ci;
                for (int d = 0; d < g.P; ++d) {
                    const int64_t e = e0 + static_cast<int64_t>(d) * g.C_in;
                    const int r = min(ev_row[e], R - 2);
                    if (r >= 0) {
                        const float L = ev_L[e], Rv = ev_R[e];
                        const float *q = cur + r * kStr;
#pragma unroll
                        for (int ii = 0; ii < TI; ++ii)
                            acc[ii] = fmaf(q[ii], L, fmaf(q[ii + kStr], Rv, acc[ii]));
                    }
                }
            }
        }
        if (more) store(gs + ((i + 1) & 1) * gbuf);
        live = __syncthreads_or(live_next);
    }
    if (!j_ok) return;
    float *out = a.part + (static_cast<int64_t>(bz) * g.C_out + co0) * NJ + jj;
#pragma unroll
    for (int ii = 0; ii < TI; ++ii)
        if (ii < ni) out[static_cast<int64_t>(ii) * NJ] = acc[ii];
}

template <int TI, int NPER, int KS>
__global__ __launch_bounds__(256) void conv_dw_kernel(LifConst C, ConvGeom g, ConvDwArgs a) {
    extern __shared__ float gs[];
    __shared__ int n_live_w[4];
    dw_block<TI, NPER, KS>(C, g, a, blockIdx.x, blockIdx.y, blockIdx.z, gs, n_live_w);
}

// dW blocks (nbx * nby * nbz of them, x fastest) and then the dt_in partial
// blocks of the same layer in one launch: the two read the same gradient
// triples and write disjoint buffers, so they need no order between them.
template <int TI, int NPER, int KHT, int NT, int KS>
__global__ __launch_bounds__(256) void conv_dwdt_kernel(LifConst C, ConvGeom g, ConvDwArgs a,
                                                        int nbx, int nby, int n_dw,
                                                        int64_t n_pos,
                                                        const float *__restrict__ Wt,
                                                        ConvSorted cs) {
    extern __shared__ float gs[];
    __shared__ int n_live_w[4];
    const int id = blockIdx.x;
    if (id < n_dw) {
        const int bx = id % nbx, t = id / nbx;
        dw_block<TI, NPER, KS>(C, g, a, bx, t % nby, t / nby, gs, n_live_w);
    } else {
        dtp_block<KHT, NT, KS>(C, g, n_pos, Wt, cs, a.gam, a.uq, a.qv, a.rend, id - n_dw);
    }
}

// dW[co, ci, ky, kx] = (1/P) sum_z part[z][co][k * C_in + ci]. Threads follow
// the partial-sum layout (coalesced reads); a block takes groups of 256 / G
// consecutive entries x G split groups (G from red_groups: more groups where
// there are many splits; at most 512 blocks, each taking every nblk-th entry
// group): group h sums z = h, h + G, ...; the G group sums are added in
// group order (fixed order: deterministic) and written to the [co][ci][ky][kx]
// slot. Splits without gradient-carrying samples wrote no partials and are
// skipped (their sums would be +0, which leaves every partial sum unchanged);
// where no split has any, the block writes the dead-neuron term (or 0) at once.
__host__ __device__ __forceinline__ int red_groups(int nsplit) {
    int G = 8;
    while (G < 64 && G * 16 < nsplit) G *= 2;
    return G;
}

__device__ void dw_reduce_block(const ConvGeom &g, int nsplit, const float *__restrict__ part,
                                const int *__restrict__ zlive, const float *__restrict__ dq,
                                float *__restrict__ dW, int blk, int nblk, float *red) {
    const int KT = g.KH * g.KW;
    const int NJ = KT * g.C_in;
    const int64_t n = static_cast<int64_t>(g.C_out) * NJ;
    const int G = red_groups(nsplit), O = static_cast<int>(blockDim.x) / G;
    const int lo = threadIdx.x % O, h = threadIdx.x / O;
    bool any = false;
    for (int z = threadIdx.x; z < nsplit; z += blockDim.x) any = any || zlive[z] != 0;
    any = __syncthreads_or(any);
    if (!any) {
        // no split carries gradient (the same for every block of the layer):
        // dW is the dead-neuron term or 0, written in dW's own order
        // (coalesced)
        for (int64_t i = static_cast<int64_t>(blk) * blockDim.x + threadIdx.x; i < n;
             i += static_cast<int64_t>(nblk) * blockDim.x)
            dW[i] = dq ? 0.f + dq[i / NJ] : 0.f;
        return;
    }
    // groups of O outputs, nblk blocks apart (block-uniform trip count)
    const int64_t ngrp = (n + O - 1) / O;
    for (int64_t grp = blk; grp < ngrp; grp += nblk) {
        const int64_t src = grp * O + lo;  // [co][k][ci]
        float s = 0.f;
        if (src < n) {
#pragma unroll 8
            for (int z = h; z < nsplit; z += G)
                if (zlive[z]) s += part[static_cast<int64_t>(z) * n + src];
        }
        red[h * O + lo] = s;
        __syncthreads();
        float tot = 0.f;
        if (h == 0)
            for (int q = 0; q < G; ++q) tot += red[q * O + lo];
        __syncthreads();  // red is rewritten by the next group
        if (h == 0 && src < n) {
            const int co = static_cast<int>(src / NJ);
            const int rem = static_cast<int>(src % NJ);
            const int k = rem / g.C_in, ci = rem % g.C_in;
            const float v = tot * g.inv_P;
            dW[(static_cast<int64_t>(co) * g.C_in + ci) * KT + k] = dq ? v + dq[co] : v;
        }
    }
}

// --------------------------------------------------------- fused launches --
// Independent per-call work shares one launch by block role (a launch costs
// several microseconds even when its work is tiny).
// Forward set-up: blocks [0, n_sort) sort cell rows (with ev set, keeping
// the cell-major events for the backward too), the next n_bin bin the raw
// inputs of a direct layer once (bin_block), the rest lay out WT.
template <typename WT>
__global__ __launch_bounds__(256) void conv_fprep_kernel(LifConst C, ConvGeom g, int n_sort,
                                                         int n_bin, int64_t n_in,
                                                         const float *__restrict__ t_in,
                                                         ConvSorted cs, CellEv ev,
                                                         const WT *__restrict__ W,
                                                         float *__restrict__ Wt) {
    extern __shared__ int sh[];
    const int blk = static_cast<int>(blockIdx.x);
    if (blk < n_sort)
        sort_cell_row(C, g, t_in, cs, ev, blk, sh);
    else if (blk < n_sort + n_bin)
        bin_block(C, n_in, t_in, cs, blk - n_sort);
    else
        weights_block<WT>(g, W, Wt, blk - n_sort - n_bin, reinterpret_cast<float (*)[33]>(sh));
}

// Backward set-up: [0, n_cr) cell rows (events for dW; with cs.key set also
// the sort with derivatives), then n_gr blocks of gradient triples and
// per-position gradient rows (rend), n_dq blocks of dead-neuron terms (one
// per channel, synfire terms on) and the WT layout.
template <typename WT>
__global__ __launch_bounds__(256) void conv_bprep_kernel(
    LifConst C, ConvGeom g, int n_cr, int n_gr, int n_dq, const float *__restrict__ t_in,
    ConvSorted cs, CellEv ev, int64_t n_pos, const float *__restrict__ t_out,
    const float *__restrict__ slope, const int *__restrict__ q_idx,
    const float *__restrict__ grad_t, Synfire sf, float *__restrict__ gam,
    float *__restrict__ uq, int *__restrict__ qv, int *__restrict__ rend,
    const WT *__restrict__ W, float *__restrict__ Wt) {
    extern __shared__ int sh[];
    // XCD-aware order: neighbouring gradient blocks read the two halves of
    // the same cache lines of the NCHW outputs
    int blk = xcd_block(blockIdx.x, gridDim.x);
    if (blk < n_cr) {
        if (cs.key)
            sort_cell_row(C, g, t_in, cs, ev, blk, sh);
        else
            events_cell_row(C, g, t_in, ev, blk);
        return;
    }
    blk -= n_cr;
    if (blk < n_gr) {
        grad_block(C, g, n_pos, blk, t_out, slope, q_idx, grad_t, sf, gam, uq, qv, rend, sh);
        return;
    }
    blk -= n_gr;
    if (blk < n_dq) {
        dead_channel_block(g, n_pos / (g.Ho * g.Wo), q_idx, sf, blk, sh);
        return;
    }
    weights_block<WT>(g, W, Wt, blk - n_dq, reinterpret_cast<float (*)[33]>(sh));
}

// Backward finish: [0, n_red) dW split reduction, the rest gathers dt_in
// (nsl blocks per cell row, one per slice of kGatherSlots slots).
__global__ __launch_bounds__(256) void conv_bfin_kernel(ConvGeom g, int R, int n_red, int nsplit,
                                                        const float *__restrict__ part,
                                                        const int *__restrict__ zlive,
                                                        const float *__restrict__ dq,
                                                        float *__restrict__ dW, int nsl,
                                                        ConvSorted cs, const int *__restrict__ rend,
                                                        float *__restrict__ dt_in) {
    static_assert(kGatherSlots >= 256, "the reduction shares the gather's LDS");
    __shared__ float lds[kGatherSlots];
    const int blk = static_cast<int>(blockIdx.x);
    if (blk < n_red) {
        dw_reduce_block(g, nsplit, part, zlive, dq, dW, blk, n_red, lds);
    } else {
        const int t = blk - n_red;
        dt_gather_block(g, R, cs, rend, dt_in, t / nsl, (t % nsl) * kGatherSlots, lds);
    }
}

// ------------------------------------------------------------ launchers --
// positions per wave of the list forward (its LDS list stays within 30 KB
// per block): 2 for at most 32 channels, 32 event rows and kListMaxRec / 2
// raw inputs per receptive field, else 0 (the chunked walk). One position
// per wave (64-channel tiles) was measured slower than the chunked walk
// (conv9's forward 0.81 against 0.68 ms): with few records per event row
// the row-by-row batches stay short, where the chunked walk's batches run
// across rows.
// the forward bins its inputs itself (no sort) where a receptive field holds
// at most as many raw inputs as a position has lanes (64; 32 with two
// positions per wave)
bool conv_fwd_direct(const ConvGeom &g, int np) {
    return g.KH * g.KW * g.PC <= (np == 2 ? kWave / 2 : kWave);
}

int conv_fwd_list_np(int M, const ConvGeom &g) {
    const int E = g.KH * g.KW * g.PC;
    return (g.C_out <= 32 && M + 2 <= 32 && 2 * E <= kListMaxRec) ? 2 : 0;
}

int conv_sort_lds_bytes(int M, const ConvGeom &g) {
    return ((M + 3) * g.Wp + 256 + sort_stage_floats(M, g) + sort_list_ints(M, g)) *
           static_cast<int>(sizeof(int));
}

hipError_t launch_conv_forward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                               bool bf16, float *Wt, ConvSorted cs, CellEv ev, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st) {
    const int np = conv_fwd_list_np(C.M, g);
    const bool direct = conv_fwd_direct(g, np);
    const bool keep = cs.dL != nullptr;
    // the direct walk bins its inputs itself: no cell-row sort, unless the
    // sort is kept for the backward
    const int n_sort = (direct && !keep) ? 0 : static_cast<int>(B * g.Hp);
    // without the sort, a direct layer on plain input has its raw inputs
    // binned once here, in NCHW order, in the sort's key/L/R arrays (as many
    // slots as raw inputs), and its positions load those events
    const int64_t n_in = B * g.C_in * g.H * g.W;
    const int pre = (direct && !keep && g.pool == 1) ? 1 : 0;
    const int n_bin = pre ? static_cast<int>((n_in + kBinPerBlock - 1) / kBinPerBlock) : 0;
    {
        ProfScope prof("conv_fprep", st);
        const unsigned blocks = static_cast<unsigned>(n_sort + n_bin + weight_tiles(g));
        const int lds = std::max(n_sort > 0 ? conv_sort_lds_bytes(C.M, g) : 0, kWtLdsBytes);
        if (bf16)
            hipLaunchKernelGGL(conv_fprep_kernel<uint16_t>, dim3(blocks), dim3(256), lds, st, C, g,
                               n_sort, n_bin, n_in, t_in, cs, ev, static_cast<const uint16_t *>(W), Wt);
        else
            hipLaunchKernelGGL(conv_fprep_kernel<float>, dim3(blocks), dim3(256), lds, st, C, g,
                               n_sort, n_bin, n_in, t_in, cs, ev, static_cast<const float *>(W), Wt);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t n_pos = B * g.Ho * g.Wo;
    constexpr int waves = 4;
    ProfScope prof("conv_fwd", st);
    if (np > 0) {
        const size_t lds =
            static_cast<size_t>(waves) * (list_wave_ints(np * g.KH * g.KW * g.PC) + (direct ? kWave : 0)) *
            sizeof(int);
        dim3 lgrid(static_cast<unsigned>((n_pos + np * waves - 1) / (np * waves)));
#define CFL(KHV, KSV, DV)                                                                         \
    hipLaunchKernelGGL((conv_fwd_list_kernel<KHV, KSV, 2, DV>), lgrid, dim3(waves * kWave), lds,  \
                       st, C, g, n_pos, Wt, cs, t_in, t_out, slope, q_idx, pre)
#define CFL_D(KHV, KSV)                                                   \
    do {                                                                  \
        if (direct) CFL(KHV, KSV, true);                                  \
        else CFL(KHV, KSV, false);                                        \
    } while (0)
#define CFL_K(KHV)                                                        \
    do {                                                                  \
        if (C.kind == kGeneral) CFL_D(KHV, kGeneral);                     \
        else CFL_D(KHV, kAnyKind);                                        \
    } while (0)
        if (g.KH == 1) CFL_K(1);
        else if (g.KH <= 3) CFL_K(3);
        else CFL_K(kConvMaxK);
#undef CFL_K
#undef CFL_D
#undef CFL
        return hipGetLastError();
    }
    dim3 grid(static_cast<unsigned>((n_pos + kFwdWaves - 1) / kFwdWaves),
              static_cast<unsigned>((g.C_out + kWave - 1) / kWave));
#define CFW(KHV, KSV, DV)                                                                        \
    hipLaunchKernelGGL((conv_fwd_kernel<KHV, KSV, DV>), grid, dim3(kFwdWaves * kWave), 0, st, C, \
                       g, n_pos, Wt, cs, t_in, t_out, slope, q_idx, pre)
#define CFW_D(KHV, KSV)                                                   \
    do {                                                                  \
        if (direct) CFW(KHV, KSV, true);                                  \
        else CFW(KHV, KSV, false);                                        \
    } while (0)
#define CFW_K(KHV)                                                        \
    do {                                                                  \
        if (C.kind == kGeneral) CFW_D(KHV, kGeneral);                     \
        else CFW_D(KHV, kAnyKind);                                        \
    } while (0)
    if (g.KH == 1) CFW_K(1);
    else if (g.KH <= 3) CFW_K(3);
    else CFW_K(kConvMaxK);
#undef CFW_K
#undef CFW_D
#undef CFW
    return hipGetLastError();
}

// channel tile: 32 for narrow layers or where two 64-wide G buffers would
// pass 48 KB of LDS
static int conv_dw_ti(const ConvGeom &g, int M) {
    if (g.C_out <= 32) return 32;
    return (2 * (M + 4) * 65 * 4 <= 48 * 1024) ? 64 : 32;
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
                                ConvBwdWs ws, float *grad_W, float *grad_t_in, const Synfire &sf,
                                bool reuse, hipStream_t st) {
    const int R = C.M + 3;
    const int64_t n_in = B * g.Hp * g.Wp * g.PC;
    const int64_t n_pos = B * g.Ho * g.Wo;
    const int64_t nj = static_cast<int64_t>(g.KH) * g.KW * g.C_in;
    const bool dt = grad_t_in && n_in > 0;
    hipError_t e;
    {
        // cell rows (events; with dt_in the sort), gradient triples +
        // gradient rows, and the WT layout for dt_in: one launch (with a
        // kept forward sort only the gradient roles)
        const int n_cr = (!reuse && n_in > 0 && (grad_W || dt)) ? static_cast<int>(B * g.Hp) : 0;
        const int n_gr = static_cast<int>((n_pos + kGradPos - 1) / kGradPos) *
                         ((g.C_out + kGradCh - 1) / kGradCh);
        const int n_wt = (dt && !reuse) ? static_cast<int>(weight_tiles(g)) : 0;
        // dead-neuron terms only where dW is written
        const bool dead = sf.on && sf.dq && grad_W;
        const int n_dq = dead ? g.C_out : 0;
        const CellEv ev{grad_W ? ws.row : nullptr, ws.L, ws.R, ws.crlive};
        ConvSorted cs = ws.srt;
        cs.L = cs.R = nullptr;  // the backward sort writes derivatives only
        if (!dt) cs.key = nullptr;
        int lds = std::max(kGradLdsBytes, 256 * static_cast<int>(sizeof(int)));
        if (dt) lds = std::max(lds, conv_sort_lds_bytes(C.M, g));
        const unsigned blocks = static_cast<unsigned>(n_cr + n_gr + n_dq + n_wt);
        ProfScope prof("conv_bprep", st);
        if (blocks > 0) {
            if (bf16)
                hipLaunchKernelGGL(conv_bprep_kernel<uint16_t>, dim3(blocks), dim3(256), lds, st, C,
                                   g, n_cr, n_gr, n_dq, t_in, cs, ev, n_pos, t_out, slope,
                                   q_idx, grad_t, sf, ws.gam, ws.uq, ws.q, ws.rend,
                                   static_cast<const uint16_t *>(W), ws.wt);
            else
                hipLaunchKernelGGL(conv_bprep_kernel<float>, dim3(blocks), dim3(256), lds, st, C,
                                   g, n_cr, n_gr, n_dq, t_in, cs, ev, n_pos, t_out, slope,
                                   q_idx, grad_t, sf, ws.gam, ws.uq, ws.q, ws.rend,
                                   static_cast<const float *>(W), ws.wt);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    ConvDwPlan p{};
    ConvDwArgs da{n_pos, 0, ws.gam, ws.uq, ws.q, ws.rend, ws.crlive, ws.row, ws.L, ws.R,
                  ws.part, ws.zlive};
    dim3 dw_grid(1, 1, 1);
    size_t dw_lds = 0;
    int nper = 0;
    if (grad_W) {
        p = plan_conv_dw(g, B, C.M);
        da.s_per_split = p.s_per_split;
        dw_grid = dim3(static_cast<unsigned>((nj + 255) / 256),
                       static_cast<unsigned>((g.C_out + p.ti - 1) / p.ti),
                       static_cast<unsigned>(p.nsplit));
        dw_lds = 2 * static_cast<size_t>(R + 1) * (p.ti + 1) * sizeof(float) +
                 static_cast<size_t>(p.s_per_split) * sizeof(int);
        nper = conv_dw_nper(C.M, p.ti);
    }
    const bool dtl = dt && n_pos > 0;
    constexpr int kDtWaves = 4;  // dt_in partial blocks: four positions each
    const int64_t n_dtp = dtl ? (n_pos + kDtWaves - 1) / kDtWaves : 0;
    const int nt = (g.C_out + kWave - 1) / kWave;
    const int nt_k = nt == 1 ? 1 : nt == 2 ? 2 : nt <= 4 ? 4 : 8;
    const int kh_k = g.KH == 1 ? 1 : g.KH <= 3 ? 3 : kConvMaxK;
    // dW and the dt_in partials in one launch where both run (general
    // kernel row, the tile shapes instantiated below); else one launch each
    bool fused = false;
    if (grad_W && dtl && C.kind == kGeneral) {
        const int64_t n_dw = static_cast<int64_t>(dw_grid.x) * dw_grid.y * dw_grid.z;
        if (n_dw + n_dtp < (int64_t{1} << 31)) {
            const dim3 grid(static_cast<unsigned>(n_dw + n_dtp));
            const int nbx = static_cast<int>(dw_grid.x), nby = static_cast<int>(dw_grid.y);
            ProfScope prof("conv_dwdt", st);
#define DWDT(TIV, NPV, KHV, NTV)                                                                \
    if (!fused && p.ti == TIV && nper == NPV && kh_k == KHV && nt_k == NTV) {                   \
        hipLaunchKernelGGL((conv_dwdt_kernel<TIV, NPV, KHV, NTV, kGeneral>), grid, dim3(256),   \
                           dw_lds, st, C, g, da, nbx, nby, static_cast<int>(n_dw), n_pos, ws.wt, \
                           ws.srt);                                                             \
        fused = true;                                                                           \
    }
            DWDT(32, 5, 1, 1) DWDT(32, 5, 3, 1)
            DWDT(64, 5, 1, 1) DWDT(64, 5, 1, 2) DWDT(64, 5, 1, 4)
            DWDT(64, 5, 3, 1) DWDT(64, 5, 3, 2) DWDT(64, 5, 3, 4)
            DWDT(64, 9, 1, 1) DWDT(64, 9, 1, 2) DWDT(64, 9, 1, 4)
            DWDT(64, 9, 3, 1) DWDT(64, 9, 3, 2) DWDT(64, 9, 3, 4)
#undef DWDT
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    if (grad_W && !fused) {
        ProfScope prof("conv_dw", st);
#define CDW_LAUNCH_K(TIV, NP, KSV) \
    hipLaunchKernelGGL((conv_dw_kernel<TIV, NP, KSV>), dw_grid, dim3(256), dw_lds, st, C, g, da)
#define CDW_LAUNCH(TIV, NP)                                               \
    do {                                                                  \
        if (C.kind == kGeneral) CDW_LAUNCH_K(TIV, NP, kGeneral);          \
        else CDW_LAUNCH_K(TIV, NP, kAnyKind);                             \
    } while (0)
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
#undef CDW_LAUNCH_K
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (dtl && !fused) {
        dim3 grid(static_cast<unsigned>(n_dtp));
        ProfScope prof("conv_dtp", st);
#define DTP_LAUNCH_K(KHV, NTV, KSV)                                                           \
    hipLaunchKernelGGL((conv_dtp_kernel<KHV, NTV, KSV>), grid, dim3(kDtWaves * kWave), 0, st,  \
                       C, g, n_pos, ws.wt, ws.srt, ws.gam, ws.uq, ws.q, ws.rend)
#define DTP_LAUNCH(KHV, NTV)                                              \
    do {                                                                  \
        if (C.kind == kGeneral) DTP_LAUNCH_K(KHV, NTV, kGeneral);         \
        else DTP_LAUNCH_K(KHV, NTV, kAnyKind);                            \
    } while (0)
#define DTP_NT(KHV)                               \
    do {                                          \
        if (nt_k == 1) DTP_LAUNCH(KHV, 1);        \
        else if (nt_k == 2) DTP_LAUNCH(KHV, 2);   \
        else if (nt_k == 4) DTP_LAUNCH(KHV, 4);   \
        else DTP_LAUNCH(KHV, 8);                  \
    } while (0)
        if (kh_k == 1) DTP_NT(1);
        else if (kh_k == 3) DTP_NT(3);
        else DTP_NT(kConvMaxK);
#undef DTP_NT
#undef DTP_LAUNCH
#undef DTP_LAUNCH_K
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    {
        // dW split reduction and dt_in gather: one launch
        const int64_t n = static_cast<int64_t>(g.C_out) * nj;
        // reduction blocks: one per red_out outputs, at most 512 (each then
        // takes every 512th group; two blocks per CU)
        const int red_out = 256 / red_groups(p.nsplit);
        const int n_red = grad_W ? static_cast<int>(std::min<int64_t>((n + red_out - 1) / red_out, 512)) : 0;
        const int per = g.Wp * g.PC;
        const int nsl = (per + kGatherSlots - 1) / kGatherSlots;
        const int n_ga = dt ? static_cast<int>(B * g.Hp) * nsl : 0;
        ProfScope prof("conv_bfin", st);
        if (n_red + n_ga > 0)
            hipLaunchKernelGGL(conv_bfin_kernel, dim3(static_cast<unsigned>(n_red + n_ga)),
                               dim3(256), 0, st, g, R, n_red, p.nsplit, ws.part, ws.zlive,
                               (sf.on && sf.dq) ? sf.dq : nullptr, grad_W, nsl, ws.srt, ws.rend,
                               grad_t_in);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace dstd
