// dstd_kernels.h -- host-side launchers of the DSTD-LIF kernels (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dstd_internal.h"

namespace dstd {

struct DwPlan { int waves, jw, nsplit, b_per_split, ipt; };
// dW of large layers with one sample group and M >= 64: inputs per thread
constexpr int kDwWideIPT = 2;

// records past the end of a sample's sorted list that the forward kernel may
// read (and mask): the list array is padded by this many records
constexpr int kSortPad = 128;

DwPlan plan_dw(int64_t B, int64_t N_in, int64_t N_out, int M);

// per sample, the records with events (one per entry of t_in [B][n_rec])
// sorted by event row, as the forward walks them
hipError_t launch_sort_records(const LifConst &C, int64_t B, int64_t n_rec, const float *t_in,
                               SortedEv srt, int *n_valid, const char *name, hipStream_t st);

hipError_t launch_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const void *W,
                          bool bf16, void *Wt, SortedEv srt, int *n_valid, const float *t_in,
                          float *t_out, float *slope, int *q_idx, hipStream_t st);

// Dense backward workspace: per-input events (dW), the row-sorted records
// with derivatives (dt_in), WT, the per-neuron gradient triples and the dW
// split partial sums.
struct DenseBwdWs {
    int *row;
    float *L, *R;
    SortedEv srt;
    int *n_valid;
    void *wt;
    float *gam, *uq;
    int *q;
    float *part;
};
hipError_t launch_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                           const void *W, bool bf16, const float *t_in, const float *t_out,
                           const float *slope, const int *q_idx, const float *grad_t,
                           DenseBwdWs ws, float *grad_W, float *grad_t_in, const Synfire &sf,
                           hipStream_t st);
// The dense forward's bf16 MFMA contraction (App. B.1's w^ as one product
// of the event matrix and W), then the interval scan. ev: 16 B per input;
// wh: [B][M+1][N_out] fp32.
constexpr int kMfmaAutoMaxM = 8;  // largest M the automatic choice sends there (measured)
hipError_t launch_forward_mfma(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                               const uint16_t *W, void *ev, float *wh, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st);
hipError_t launch_softmax_ce(int64_t B, int64_t N, const float *t, const int *labels,
                             float tau_soft, float t_cap, float *grad, float *loss, hipStream_t st);
hipError_t launch_mse(int64_t B, int64_t N, const float *t, const float *y, float *grad,
                      float *loss, hipStream_t st);

// ------------------------------------------------------------------ conv --
// Geometry of a conv layer, derived on the host. The (pooled) input map has
// Hp x Wp cells of P raw pixels; PC = P * C_in raw inputs per cell.
// n / d for 0 <= n < 2^31 by a multiply and a shift (round-up magic number
// of Granlund and Montgomery): s = ceil(log2 d), m = floor(2^32 (2^s - d) / d)
// + 1, n / d = (mulhi(n, m) + n) >> s; set on the host by fast_div().
struct FastDiv {
    uint32_t m;
    int s;
};

struct ConvGeom {
    int C_in, H, W, C_out, KH, KW, stride, pad, pool;
    int Hp, Wp, Ho, Wo, P, PC;
    float inv_P;
    FastDiv dv_pch, dv_w, dv_cin;  // by Wp * P (raw inputs per channel of a cell row), W, C_in
    FastDiv dv_p, dv_kw, dv_pc;    // by P, KW (receptive-field decode) and PC
};

inline FastDiv fast_div(uint32_t d) {
    int s = 0;
    while ((uint64_t(1) << s) < d) ++s;
    return FastDiv{static_cast<uint32_t>(((uint64_t(1) << 32) * ((uint64_t(1) << s) - d)) / d + 1), s};
}

__device__ __forceinline__ int fdiv(int n, FastDiv f) {
    const uint32_t u = static_cast<uint32_t>(n);
    return static_cast<int>((__umulhi(u, f.m) + u) >> f.s);
}

constexpr int kConvMaxK = 7;  // largest kernel height/width

// ints per cell row of the bucket-start table (R = M + 3 event rows)
__host__ __device__ __forceinline__ int conv_off_stride(int R, const ConvGeom &g) {
    return (g.Wp + 1) * R + 1;
}

// Per cell row (b, py): records bucketed by (event row r, cell column px),
// in (r, px) order, key = px * C_in + ci. The bucket starts within the cell
// row's Wp * PC record slots are held column-major, off[cr * noff + px * R +
// r] (cr = b*Hp + py, noff = conv_off_stride), so that lanes = event rows
// read one column contiguously; column px = Wp holds the end of each row r
// (the start of (r + 1, 0)), and the last entry the row's record count.
// The forward sort writes the event weights L, R; the backward sort (or a
// forward that keeps its sort for the backward) writes the record's event
// row and cell column (px = row << 16 | cell column), its input index in the
// cell row (src = px * PC + j') and the event derivatives dL, dR. Unused
// arrays are NULL. P[record][KH*KW] holds the per-tap partial sums of dt_in:
// the entry of tap k is written by the output position that reads the record
// through k, and only where that position passes gradient up to the record's
// event row (rend); the gather reads exactly those entries.
struct ConvSorted {
    int *key; float *L; float *R; int *off; int *px; int *src; float *P; float *dL; float *dR;
};

// Cell-major events of every input (row -1: no events) for the dW reduction,
// written only for cell rows where some input has events; live[cr] says which
// (the dW kernel reads no others). NULL row: not wanted.
struct CellEv { int *row; float *L, *R; int *live; };

struct ConvBwdWs {
    int *row;
    float *L, *R;            // cell-major events (dW), for cell rows with events; L, R
                             //   hold values only where row >= 0
    int *crlive;             // [B][Hp]: the cell row has an input with events
    float *gam, *uq;         // per output neuron, [B][Ho*Wo][C_out]: -g/slope, t - T_q
    int *q;                  //   and its interval (-1: no gradient flows)
    int *rend;               // [B][Ho*Wo]: last event row whose records get gradient
                             //   there (min(R-2, max q + 1) over channels; -1: none)
    float *part;             // dW partial sums [nsplit][C_out][KH*KW*C_in]
    int *zlive;              // [nsplit]: 1 if the split has samples that pass
                             //   gradient (its partials are written only then)
    float *wt;               // [KH*KW*C_in][C_out] weights / P (as the forward)
    ConvSorted srt;          // records sorted as in the forward, with dL, dR
};

// largest C_out the dt_in kernel handles (channel tiles of 64 per lane)
constexpr int kConvMaxCoutDt = 512;

struct ConvDwPlan { int ti, nsplit, s_per_split; };
constexpr int kConvMaxSplitSamples = 4096;  // (b, position) samples per dW block

// the dt_in kernel's LDS row stride (words); odd, so rows r and r+1 of one
// lane fall in different banks
constexpr int kDtStride = kWave + 1;

ConvDwPlan plan_conv_dw(const ConvGeom &g, int64_t B, int M);
int conv_sort_lds_bytes(int M, const ConvGeom &g);
// keep (cs.dL and ev set): the sort also writes what the backward needs
// (derivatives, px, src, cell-major events), even where the walk bins its
// inputs itself.
hipError_t launch_conv_forward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                               bool bf16, float *Wt, ConvSorted cs, CellEv ev, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st);
// reuse: the workspace holds a kept forward sort (records, events, weight
// layout) for these inputs and weights: no cell-row or weight-layout work.
hipError_t launch_conv_backward(const LifConst &C, const ConvGeom &g, int64_t B, const void *W,
                                bool bf16, const float *t_in, const float *t_out,
                                const float *slope, const int *q_idx, const float *grad_t,
                                ConvBwdWs ws, float *grad_W, float *grad_t_in,
                                const Synfire &sf, bool reuse, hipStream_t st);

// Synfire term values (reporting): T and Q of one layer's outputs
// t [B][rows][spatial] and weights [rows][row_len].
int synfire_value_blocks(int64_t n);
hipError_t launch_synfire_value(const Synfire &sf, int64_t B, int64_t rows, int64_t spatial,
                                int64_t row_len, const float *t_out, const void *W, bool bf16,
                                float *ws, float *value, hipStream_t st);

// ------------------------------------------------------------------ skip --
// Skip-and-delay input of an SD block: per sample n1 = C1*HW delayed block
// inputs then n2 = C2*HW second-layer outputs (concatenation along channels),
// and the split of its gradient (acc: add into g1 instead of overwriting).
hipError_t launch_skip_concat(int64_t B, int64_t n1, int64_t n2, const float *t1, float delay,
                              const float *t2, float *out, hipStream_t st);
hipError_t launch_skip_split(int64_t B, int64_t n1, int64_t n2, const float *g, float *g1, int acc,
                             float *g2, hipStream_t st);

// ------------------------------------------------------------ multispike --
// Events of every input spike ([B][N_in][F_in]: row = q + 1 or -1, L, R and
// their time derivatives) and the backward's per-neuron inputs: the forward's
// spikes [B][N_out][F] and the upstream gradient, G [B][M + 1][N_out] out.
struct MsEvents { int *row; float *L, *R, *dL, *dR; };
struct MsGrad {
    const float *t, *slope;
    const int *q;
    const float *cur, *g;
    float *G;
    int64_t n;  // neurons B * N_out (0: no G role)
    int F;
};
constexpr int kMsMaxM = 250;  // (M + 3) rows x 64 lanes of fp32 in 64 KB of LDS
constexpr int kMsMaxF = 64;
// dW for M <= kMsDwMaxM stages G tiles in LDS, with the batch split S ways
// (S from the shapes alone, so the workspace query and the launch agree:
// about 2048 blocks, at most 16 splits);
// S > 1 needs S * N_in * N_out floats of partials in the workspace. 0: the
// one-wave-per-input kernel is used instead.
constexpr int kMsDwMaxM = 64;
inline int ms_dw_splits(int M, int64_t B, int64_t N_in, int64_t N_out) {
    if (M > kMsDwMaxM || B < 1 || N_in < 1 || N_out < 1) return 0;
    const int64_t blocks = ((N_out + 63) / 64) * ((N_in + 63) / 64);
    int64_t s = (2048 + blocks - 1) / blocks;
    s = s < 16 ? s : 16;
    s = s < B ? s : B;
    const int64_t per = (B + s - 1) / s;
    return static_cast<int>((B + per - 1) / per);
}

hipError_t launch_ms_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t F_in,
                             int64_t N_out, int64_t F_out, const void *W, bool bf16, void *Wt,
                             SortedEv srt, int *n_valid, const float *t_in, float *t_out,
                             float *slope, int *q_idx, float *cur, hipStream_t st);
hipError_t launch_ms_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t F_in,
                              int64_t N_out, int64_t F_out, const void *W, bool bf16, void *Wt,
                              MsEvents ev, const float *t_in, const float *t_out,
                              const float *slope, const int *q_idx, const float *cur,
                              const float *grad_t, float *G, float *dw_part, float *grad_W,
                              float *grad_t_in, hipStream_t st);

// ----------------------------------------------------------------- exact --
// Exact spike times by sorting (App. A, Alg. 1). Per sample, the finite
// inputs before t_max in ascending time order as records (SoA, each array
// [B][stride], padded by kExactPad records at the end): input index j, time
// t, candidate-interval length len (to the next input, or to t_max for the
// last record) with e^{-kappa len} and max K on [0, len] (the interval
// filter's bound, rounded up), and in fp64 the decays over len and K(len)
// (they carry the state to the next input). n[b] = number of records of
// sample b.
struct ExactRecs {
    int *j;
    float *t, *len, *r_lo, *kmax;
    double *alpha, *beta, *kl;
    int *n;
    int64_t stride;
};
constexpr int kExactPad = 32;
constexpr int kExactMaxIn = 8192;  // one block sorts a sample in 64 KB of LDS

hipError_t launch_exact_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                                const void *W, bool bf16, void *Wt, ExactRecs rec,
                                const float *t_in, float t_max, float *t_out, float *slope,
                                int *k_idx, hipStream_t st);
// per-neuron gradient data of the exact backward: {gamma = -g/slope, t_out,
// left end of the crossing interval, 0}, as [B][N_out] and [N_out][B]
hipError_t launch_exact_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                                 const void *W, bool bf16, const float *t_in, float t_max,
                                 const float *t_out, const float *slope, const int *k_idx,
                                 const float *grad_t, float4 *P, float4 *PT, float *grad_W,
                                 float *grad_t_in, hipStream_t st);

}  // namespace dstd
