// dstd_walk.h -- the walk over one sample's row-sorted event records (device
// code shared by the dense TTFS forward and the multi-spike forward).
#pragma once

#include "dstd_internal.h"

namespace dstd {

// records per batch of scalar record reads and weight loads
constexpr int kBatch = 8;

// Lane = neuron i of a 64-neuron tile, one sample per wavefront. The wave
// walks its sample's event records in grid order: each record adds W[i, j] L
// and W[i, j] R to the running sums of its row (WT row j is one coalesced
// load with a scalar base). When a row closes, grid point m = row - 1 is
// complete (its L parts come from this row, its R parts from the previous
// one) and goes straight into the interval scan: the weighted events never
// exist in memory.
// sc.step(C, m, w^_m) receives the grid points in order; the
// walk stops once sc.found() holds for every lane with a neuron. A record's
// input index is its weight row (kDiv false), or that index divided by rowdiv
// (kDiv true: F_in records per input, as for a multi-spike layer).
template <typename WT, bool kDiv, typename ScanT>
__device__ __forceinline__ void walk_sorted_rows(const LifConst &C, int N_in, int N_out,
                                                 const WT *__restrict__ Wt, SortedEv srt, int b,
                                                 int n, int i, bool row_ok, int rowdiv,
                                                 ScanT &sc) {
    const int64_t eo = static_cast<int64_t>(b) * srt.stride;
    const int *ej = srt.j + eo;
    const int *er = srt.r + eo;
    const float *eL = srt.L + eo;
    const float *eR = srt.R + eo;
    int cur = 0;  // row whose records are being summed
    float aL = 0.f, aR = 0.f, carry = 0.f;
    bool done = false;
    // close rows cur .. target-1: grid point cur-1 gets this row's L sums
    // plus the previous row's R sums. A record's row is at most M+1, so
    // closing up to it stops before grid point M (the last interval, tested
    // at the end only).
    auto close_to = [&](int target) {
        while (cur < target && !done) {
            if (cur >= 1) sc.template step_k<false>(C, cur - 1, aL + carry);
            carry = aR;
            aL = 0.f;
            aR = 0.f;
            ++cur;
            if (__all(sc.found() || !row_ok)) done = true;
        }
    };
    // Weight loads are raw buffer loads: per-lane column offset (constant)
    // plus a scalar row offset j*N_out, so they need no address arithmetic
    // in vector registers.
    // Record arrays are padded by two batches, so the batched scalar reads
    // are unconditional; only a partial last batch is masked. Lanes past
    // N_out read column 0 (their results are never stored).
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(Wt, static_cast<uint32_t>(static_cast<int64_t>(N_in) * N_out * sizeof(WT)));
    const int voff = (row_ok ? i : 0) * static_cast<int>(sizeof(WT));
    const int rstride = N_out * static_cast<int>(sizeof(WT));
    // Reads past the end of the list see stale workspace: their input index
    // is clamped into [0, N_in) so every scalar offset stays inside WT.
    const unsigned jmax = static_cast<unsigned>(max(N_in - 1, 0));
    auto wrow = [&](int j) {
        const unsigned row = kDiv ? static_cast<unsigned>(j) / static_cast<unsigned>(rowdiv)
                                  : static_cast<unsigned>(j);
        return static_cast<int>(min(row, jmax)) * rstride;
    };
    float w[kBatch], wn[kBatch];
#pragma unroll
    for (int kk = 0; kk < kBatch; ++kk) wn[kk] = BufLoad<WT>::get(wr, voff, wrow(as_const(ej)[kk]));
    for (int k0 = 0; k0 < n && !done; k0 += kBatch) {
        int rr[kBatch], jj1[kBatch];
        float ll[kBatch], rv[kBatch];
#pragma unroll
        for (int kk = 0; kk < kBatch; ++kk) {
            w[kk] = wn[kk];
            rr[kk] = as_const(er + k0)[kk];
            ll[kk] = as_const(eL + k0)[kk];
            rv[kk] = as_const(eR + k0)[kk];
            jj1[kk] = as_const(ej + k0 + kBatch)[kk];
        }
        // the next batch's weights are in flight while this one is consumed
#pragma unroll
        for (int kk = 0; kk < kBatch; ++kk) wn[kk] = BufLoad<WT>::get(wr, voff, wrow(jj1[kk]));
        const int nk = min(kBatch, n - k0);
        if (nk == kBatch && rr[kBatch - 1] == cur) {
            // common case: a full batch that continues the current row
#pragma unroll
            for (int kk = 0; kk < kBatch; ++kk) {
                aL = fmaf(w[kk], ll[kk], aL);
                aR = fmaf(w[kk], rv[kk], aR);
            }
            continue;
        }
        int kk_start = 0;
        while (!done) {
            int stop = kBatch, target = 0;
#pragma unroll
            for (int kk = 0; kk < kBatch; ++kk) {
                if (kk >= kk_start && kk < stop && kk < nk) {
                    if (rr[kk] == cur) {
                        aL = fmaf(w[kk], ll[kk], aL);
                        aR = fmaf(w[kk], rv[kk], aR);
                    } else {
                        stop = kk;
                        target = rr[kk];
                    }
                }
            }
            if (stop >= kBatch || stop >= nk) break;
            close_to(target);
            kk_start = stop;
        }
    }
    close_to(C.M + 1);
    if (!done) sc.template step_k<true>(C, C.M, aL + carry);  // row M+2 has no records
}

}  // namespace dstd
