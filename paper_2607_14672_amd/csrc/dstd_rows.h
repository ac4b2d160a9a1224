// dstd_rows.h -- the row-parallel forward over one sample's row-sorted event
// records (device code shared by the dense TTFS forward and the multi-spike
// forward; the two differ in how a record names its weight row and in the
// interval scan that consumes the grid-point sums).
#pragma once

#include "dstd_internal.h"

namespace dstd {

// Event-row ranges of a sample's sorted list. With rs[r] the start of row r
// (rs[R - 1] = rs[R] = n: the last row holds no records), the row holding
// record t < n is the number of rows r < R - 1 with rs[r] <= t, minus one;
// t >= n maps to R - 1. All lanes load the row starts at once (one round
// trip instead of a chain of dependent scalar loads) and count with ballots;
// a range's first records come back with readlane. The result: rows
// [ra, rb) holding records [ka, kb).
struct RowRange { int ra, rb, ka, kb; };

__device__ __forceinline__ RowRange row_range(const int *rs, int R, int n, int ta, int tb,
                                              bool first, bool last, int lane) {
    int ca = 0, cb = 0, v0 = 0;
    for (int r0 = 0; r0 < R - 1; r0 += kWave) {
        const int r = r0 + lane;
        const int v = (r < R - 1) ? rs[r] : 0x7fffffff;
        if (r0 == 0) v0 = v;
        ca += __popcll(__ballot(v <= ta));
        cb += __popcll(__ballot(v <= tb));
    }
    RowRange g;
    g.ra = first ? 0 : ((ta >= n) ? R - 1 : ca - 1);
    g.rb = last ? R - 1 : ((tb >= n) ? R - 1 : cb - 1);
    g.ka = (g.ra == R - 1) ? n : ((g.ra < kWave) ? __builtin_amdgcn_readlane(v0, g.ra) : rs[g.ra]);
    g.kb = (g.rb == R - 1) ? n : ((g.rb < kWave) ? __builtin_amdgcn_readlane(v0, g.rb) : rs[g.rb]);
    return g;
}

// Row-parallel forward (M <= kRowsMaxM). A block of kRowWaves wavefronts
// serves one sample and NT (1, 2 or 4) 64-neuron tiles: wave w sums, for all
// NT tiles, the records of a contiguous range of whole event rows (ranges
// split the sample's records about evenly), in the same per-row order as the
// single-wave walk above; then wave t < NT runs the interval scan of tile t.
// Grid point m takes the L sums of row m+1 plus the R sums of row m. Where
// both rows lie in one wave's range, that wave adds them and stores the
// point's sum in LDS; at a boundary between two ranges the two halves are
// stored apart (first row's L sums, last row's R sums, per wave) and added
// by the scanning wave. The sums, and their order, are those of the
// single-wave walk; one value per point halves the LDS a tile needs.
// LDS is tile-minor (point, tile, lane): a row close writes its NT tiles
// from one address with immediate offsets.
constexpr int kRowWaves = 4;
constexpr int kRowLdsCap = 48 * 1024;  // LDS budget per block when choosing NT
constexpr int kRowsMaxM = 64;
constexpr int kRowSub = 8;  // records per scalar load group; their NT tile loads fly together

// VEC: lane l sums the NT consecutive neurons NT*l .. NT*l+NT-1 of the
// block's NT*64 (one NT-wide weight load per record instead of NT loads one
// tile apart; N_out % NT == 0 so the loads are aligned). The point sums then
// sit at the same LDS offsets as without VEC (tile t, lane l' is neuron
// 64 t + l' = NT l + c), so the scan reads them unchanged.
template <typename WT, int NT, int KS, bool VEC, typename Out>
__global__ __launch_bounds__(kRowWaves * 64) void fwd_rows_kernel(LifConst C, int N_in, int N_out,
                                                                  const WT *__restrict__ Wt,
                                                                  SortedEv srt, Out out) {
    // LDS: P[R][NT][64] point sums, BL[kRowWaves][NT][64] and
    // BR[kRowWaves][NT][64] range-boundary halves, span[2][kRowWaves] ranges
    extern __shared__ float rsum[];
    constexpr int kPt = NT * kWave;  // floats per point (all tiles)
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    // XCD-aware order: the hardware block maps to a logical (tile block bx,
    // sample b) with the samples fastest, so each XCD takes one contiguous
    // range and works through one weight tile, all samples, at a time: its
    // W^T columns stay in that XCD's L2 instead of several tiles competing
    const int nby = static_cast<int>(gridDim.y);
    const int lin = xcd_block(static_cast<int>(blockIdx.x + blockIdx.y * gridDim.x),
                              static_cast<int>(gridDim.x) * nby);
    const int bx = lin / nby;
    const int b = lin - bx * nby;
    const int R = rows_of(C);
    float *P = rsum;
    float *BL = rsum + R * kPt;
    float *BR = BL + kRowWaves * kPt;
    int *span = reinterpret_cast<int *>(BR + kRowWaves * kPt);
    const int *rs = srt.rs + static_cast<int64_t>(b) * (R + 1);
    const int n = *as_const(rs + R);
    // range w: the rows holding records [w*n/kRowWaves, (w+1)*n/kRowWaves)
    const RowRange rg = row_range(rs, R, n, static_cast<int>((static_cast<int64_t>(n) * wave) / kRowWaves),
                                  static_cast<int>((static_cast<int64_t>(n) * (wave + 1)) / kRowWaves),
                                  wave == 0, wave == kRowWaves - 1, lane);
    const int r_lo = uniform(rg.ra), r_hi = uniform(rg.rb);
    const int k_lo = uniform(rg.ka), k_hi = uniform(rg.kb);
    const int64_t eo = static_cast<int64_t>(b) * srt.stride;
    const int *ej = srt.j + eo;
    const int *er = srt.r + eo;
    const float *eL = srt.L + eo;
    const float *eR = srt.R + eo;
    int cur = r_lo;
    float aL[NT], aR[NT], cy[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        aL[t] = 0.f;
        aR[t] = 0.f;
        cy[t] = 0.f;
    }
    // close row cur (target > cur): point cur-1 gets this row's L sums plus
    // the previous row's R sums (cy); rows cur+1 .. target-1 have no records,
    // so point cur is row cur's R sums alone and the points after it are 0
    // LDS slot of this lane's value t within a point's kPt floats
    constexpr int kLs = VEC ? 1 : kWave;
    const int lofs = VEC ? NT * lane : lane;
    auto close_to = [&](int target) {
        float *d = ((cur == r_lo) ? BL + wave * kPt : P + (cur - 1) * kPt) + lofs;
#pragma unroll
        for (int t = 0; t < NT; ++t) d[t * kLs] = aL[t] + cy[t];
        if (target > cur + 1) {
            float *e = P + cur * kPt + lofs;
#pragma unroll
            for (int t = 0; t < NT; ++t) e[t * kLs] = aR[t];
            for (int r = cur + 2; r < target; ++r) {
                float *z = P + (r - 1) * kPt + lofs;
#pragma unroll
                for (int t = 0; t < NT; ++t) z[t * kLs] = 0.f;
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) cy[t] = 0.f;
        } else {
#pragma unroll
            for (int t = 0; t < NT; ++t) cy[t] = aR[t];
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            aL[t] = 0.f;
            aR[t] = 0.f;
        }
        cur = target;
    };
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(Wt, static_cast<uint32_t>(static_cast<int64_t>(N_in) * N_out * sizeof(WT)));
    int voff[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int i = (bx * NT + t) * kWave + lane;
        voff[t] = min(i, N_out - 1) * static_cast<int>(sizeof(WT));
    }
    // VEC: one load of NT neurons; past N_out it reads the next row's first
    // weights or, after the last row, zeros (buffer range check): those sums
    // belong to lanes without a neuron and are never scanned into outputs
    const int voffv = (bx * NT * kWave + NT * lane) * static_cast<int>(sizeof(WT));
    const int rstride = N_out * static_cast<int>(sizeof(WT));
    const int jmax = max(N_in - 1, 0);
    // Record fields come through the scalar cache, kRowSub records per load
    // (the next group's in flight while this one is summed; reads past the
    // range stay inside the sorted lists' padding and are not summed). The
    // group's weight rows, all NT tiles, are loaded together.
    int nj[kRowSub], nr[kRowSub];
    float nL[kRowSub], nR[kRowSub];
    auto fetch = [&](int k) {
#pragma unroll
        for (int kk = 0; kk < kRowSub; ++kk) {
            nj[kk] = as_const(ej + k)[kk];
            nr[kk] = as_const(er + k)[kk];
            nL[kk] = as_const(eL + k)[kk];
            nR[kk] = as_const(eR + k)[kk];
        }
    };
    fetch(k_lo);
    for (int k0 = k_lo; k0 < k_hi; k0 += kRowSub) {
        int cr[kRowSub];
        float cL[kRowSub], cR[kRowSub], w[kRowSub][NT];
#pragma unroll
        for (int kk = 0; kk < kRowSub; ++kk) {
            const int jo = min(max(out.wrow(nj[kk]), 0), jmax) * rstride;
            if constexpr (VEC) {
                BufLoadN<WT, NT>::get(wr, voffv, jo, w[kk]);
            } else {
#pragma unroll
                for (int t = 0; t < NT; ++t) w[kk][t] = BufLoad<WT>::get(wr, voff[t], jo);
            }
            cr[kk] = nr[kk];
            cL[kk] = nL[kk];
            cR[kk] = nR[kk];
        }
        fetch(k0 + kRowSub);
        const int nk = min(kRowSub, k_hi - k0);
        if (nk == kRowSub && cr[kRowSub - 1] == cur) {
            // common case: the whole group continues the current row
#pragma unroll
            for (int kk = 0; kk < kRowSub; ++kk)
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    aL[t] = fmaf(w[kk][t], cL[kk], aL[t]);
                    aR[t] = fmaf(w[kk][t], cR[kk], aR[t]);
                }
        } else {
#pragma unroll
            for (int kk = 0; kk < kRowSub; ++kk) {
                if (kk < nk) {
                    if (cr[kk] != cur) close_to(cr[kk]);
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        aL[t] = fmaf(w[kk][t], cL[kk], aL[t]);
                        aR[t] = fmaf(w[kk][t], cR[kk], aR[t]);
                    }
                }
            }
        }
    }
    if (r_hi > cur) close_to(r_hi);
    if (r_hi > r_lo) {
#pragma unroll
        for (int t = 0; t < NT; ++t) BR[wave * kPt + lofs + t * kLs] = cy[t];
    }
    if (lane == 0) {
        span[wave] = r_lo;
        span[kRowWaves + wave] = r_hi;
    }
    __syncthreads();
    // wave t scans tile t
    if (wave >= NT) return;
    const int tile = wave;
    const int i = (bx * NT + tile) * kWave + lane;
    const bool row_ok = i < N_out;
    if (uniform(static_cast<int>(__any(row_ok))) == 0) return;
    // range boundaries: point lo(w) - 1 of each nonempty range w >= 1 (wave
    // 0's range always holds row 0 and is never empty) is w's first-row L
    // sums plus the last-row R sums of the nonempty range before it; this
    // wave writes it into its own tile's slot (no other wave stores there)
    float *tp = P + tile * kWave + lane;
    const float *tbl = BL + tile * kWave + lane;
    const float *tbr = BR + tile * kWave + lane;
    int prev = 0;
#pragma unroll
    for (int w = 1; w < kRowWaves; ++w) {
        const int lo = uniform(span[w]), hi = uniform(span[kRowWaves + w]);
        if (hi > lo) {
            tp[(lo - 1) * kPt] = tbl[w * kPt] + tbr[prev * kPt];
            prev = w;
        }
    }
    // the last grid point that receives input: the last record's row r
    // feeds points r - 1 and r (at most M)
    const int m_end = (n > 0) ? min(uniform(*as_const(er + n - 1)), C.M) : -1;
    out.template scan<KS>(C, N_out, b, i, row_ok, tp, kPt, m_end);
}

// Grid point sums needed by one block of NT tiles: P[R][NT][64] plus the
// range-boundary halves and the span table.
inline size_t rows_lds(int nt, int R) {
    return static_cast<size_t>(nt) * (R + 2 * kRowWaves) * kWave * sizeof(float) +
           2 * kRowWaves * sizeof(int);
}

// Up to four tiles per block (one scan per wave) when there are enough
// neurons and their point sums fit the LDS budget.
inline int rows_nt(int64_t N_out, int R) {
    const int64_t tiles = (N_out + kWave - 1) / kWave;
    for (int t : {4, 2})
        if (tiles >= t && rows_lds(t, R) <= static_cast<size_t>(kRowLdsCap)) return t;
    return 1;
}

// TTFS outputs: a record's input index is its weight row; the scan stops at
// the first crossing and writes (t_out, slope, q) once per neuron.
struct RowOutTtfs {
    float *t_out, *slope;
    int *q_idx;

    __device__ __forceinline__ int wrow(int j) const { return j; }

    // m_end: the last grid point with input (-1: none). Points after it
    // add nothing: from there the rest of the window is one free-decay
    // segment (Scan::tail).
    template <int KS>
    __device__ __forceinline__ void scan(const LifConst &C, int N_out, int b, int i, bool row_ok,
                                         const float *tp, int kPt, int m_end) const {
        Scan<KS> sc;
        float wn = tp[0];  // next grid point's sum, read ahead
        bool done = false;
        const int m_stop = min(C.M, m_end + 1);
        for (int m = 0; m < m_stop && !done; ++m) {
            const float wc = wn;
            wn = tp[(m + 1) * kPt];
            sc.template step_k<false>(C, m, wc);
            done = __all(sc.found() || !row_ok);
        }
        if (!done) {
            if (m_stop < C.M) sc.tail(C, m_stop);
            else sc.template step_k<true>(C, C.M, wn);  // the last interval
        }
        if (!row_ok) return;
        float to, sl;
        int q;
        sc.finish(C, to, sl, q);
        const int64_t o = static_cast<int64_t>(b) * N_out + i;
        t_out[o] = to;
        slope[o] = sl;
        q_idx[o] = q;
    }
};

}  // namespace dstd
