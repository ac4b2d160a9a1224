// dstd_dense.hip -- DSTD-LIF dense-layer kernels for gfx950.
//
// The event matrix S[b, m, j] has at most two nonzeros per (b, j): the DSTD
// kernel has two-point support (App. B.3). The contraction
// w^[b, m, i] = sum_j W[i, j] S[b, m, j] therefore runs over each sample's
// inputs sorted by event row: a wavefront (lanes = neurons) adds W[i, j] L and
// W[i, j] R of every input to the running sums of its row and feeds each
// closed row to the interval scan, instead of a dense (M+1)-row GEMM that
// would spend (M+1)/2 times the method's multiply-adds on zeros. The weighted
// events never go to HBM. The backward walks the same sorted lists for dt_in
// and reduces dW over the batch with per-input events.
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_lif.h"
#include "dstd_walk.h"
#include "dstd_rows.h"
#include "dstd_profile.h"

#include <algorithm>

namespace dstd {

// ----------------------------------------------------------- event sort --
// Per sample, the inputs that have events, sorted by event row (stable: j
// ascending within a row), as structure-of-arrays records {j, row, L, R}
// (with deriv: the derivatives dL, dR in place of L, R), plus the row starts.
// One block of kSortWaves wavefronts per sample; wave w owns a contiguous
// range of inputs. Row histograms per wave (integer LDS atomics, order-free)
// give every (row, wave) pair its start offset (wave 0 scans the row totals
// across its lanes); each wave then places its inputs 64 at a time: a lane's
// rank among the lanes of its batch with the same row comes from a match
// mask built bit by bit from ballots of the row index, and the lowest lane
// of each row advances that row's slot. The fixed order keeps every sum of
// the forward pass bitwise reproducible.
constexpr int kSortWaves = 8;
constexpr int kPrepThreads = kSortWaves * 64;
constexpr int kRowBits = 9;  // row + 1 < 512 covers R = M + 3 rows for every M <= 256
static_assert(DSTD_MAX_M + 3 < (1 << kRowBits), "row keys must fit kRowBits");

// Optional per-input outputs of the sort, in input order [B][N_in]: the
// events (row -1: none) for the dW reduction, and an array set to zero
// (dt_in, whose inputs with events are written later).
struct SortOut { int *row; float *L; float *R; float *zero; };

template <int KS>
__device__ void sort_sample(const LifConst &C, int b, int N_in, const float *__restrict__ t_in,
                            SortedEv srt, int *__restrict__ n_valid, int deriv, SortOut xo,
                            int *sh) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int R = rows_of(C);
    int *hist = sh;  // [kSortWaves][R], then rowstart [R + 1]
    int *rowstart = sh + kSortWaves * R;
    const float *tb = t_in + static_cast<int64_t>(b) * N_in;
    const int per = ((N_in + kSortWaves * kWave - 1) / (kSortWaves * kWave)) * kWave;
    const int j_lo = wave * per, j_hi = min(N_in, j_lo + per);
    for (int k = threadIdx.x; k < kSortWaves * R + R + 1; k += blockDim.x) sh[k] = 0;
    __syncthreads();
    for (int j0 = j_lo; j0 < j_hi; j0 += kWave) {
        const int j = j0 + lane;
        const int r = (j < j_hi) ? bin_row(C, tb[j]) : -1;
        if (r >= 0) atomicAdd(&hist[wave * R + r], 1);
    }
    __syncthreads();
    if (wave == 0) {
        // rowstart[r + 1] = events in rows <= r: an inclusive scan of the row
        // totals, 64 rows per pass
        int acc = 0;
        for (int r0 = 0; r0 < R; r0 += kWave) {
            const int r = r0 + lane;
            int v = 0;
            if (r < R)
                for (int w = 0; w < kSortWaves; ++w) v += hist[w * R + r];
#pragma unroll
            for (int m = 1; m < kWave; m <<= 1) {
                const int o = __shfl_up(v, m);
                if (lane >= m) v += o;
            }
            if (r < R) rowstart[r + 1] = acc + v;
            acc += __shfl(v, kWave - 1);
        }
        if (lane == 0) n_valid[b] = acc;
    }
    __syncthreads();
    for (int r = threadIdx.x; r <= R; r += blockDim.x)
        srt.rs[static_cast<int64_t>(b) * (R + 1) + r] = rowstart[r];
    for (int r = threadIdx.x; r < R; r += blockDim.x) {
        int base = rowstart[r];
        for (int w = 0; w < kSortWaves; ++w) {
            const int h = hist[w * R + r];
            hist[w * R + r] = base;  // becomes this wave's next slot in row r
            base += h;
        }
    }
    __syncthreads();
    const int64_t ob = static_cast<int64_t>(b) * srt.stride;
    const int64_t ib = static_cast<int64_t>(b) * N_in;
    int *next = hist + wave * R;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int j0 = j_lo; j0 < j_hi; j0 += kWave) {
        const int j = j0 + lane;
        Event e{-1, 0.f, 0.f, 0.f, 0.f};
        if (j < j_hi) e = bin_event<KS>(C, tb[j]);
        const int r = e.row;
        if (j < j_hi) {
            if (xo.row) {
                xo.row[ib + j] = r;
                xo.L[ib + j] = e.L;
                xo.R[ib + j] = e.R;
            }
            if (xo.zero) xo.zero[ib + j] = 0.f;
        }
        // lanes with the same row: agree with this lane on every bit of r + 1
        // (lanes without an event, r + 1 = 0, match only each other)
        const unsigned key = static_cast<unsigned>(r + 1);
        uint64_t same = ~0ull;
#pragma unroll
        for (int bit = 0; bit < kRowBits; ++bit) {
            const uint64_t ones = __ballot((key >> bit) & 1u);
            same &= ((key >> bit) & 1u) ? ones : ~ones;
        }
        const int rank = __popcll(same & below);
        int pos = 0;
        if (r >= 0) {
            const int base = next[r];
            pos = base + rank;
            if (rank == 0) next[r] = base + __popcll(same);
        }
        if (r >= 0) {
            const int64_t o = ob + pos;
            srt.j[o] = j;
            srt.r[o] = r;
            srt.L[o] = deriv ? e.dL : e.L;
            srt.R[o] = deriv ? e.dR : e.R;
        }
    }
}

// Independent setup work of a layer call in one launch, by block role:
// blocks [0, n_sort) sort one sample each, the next n_tr blocks transpose one
// weight tile each, then blocks writing the gradient triple (gamma, t - T_q,
// q) of kPrepThreads neurons each (backward only) and, with the synfire
// terms on, blocks counting each neuron's silent samples into sf.dq. One
// launch instead of several: every launch costs a few microseconds even when
// its work is tiny.
struct PrepGrad {
    const float *t_out, *slope, *grad_t;
    const int *q_idx;
    float *gam, *uq;
    int *q;
    Synfire sf;
    int B;
};

template <typename WT, int KS>
__global__ __launch_bounds__(kPrepThreads) void prep_kernel(LifConst C, int n_sort, int n_tr,
                                                            int N_in, int N_out,
                                                            const float *__restrict__ t_in,
                                                            SortedEv srt, int *__restrict__ n_valid,
                                                            int deriv, SortOut xo,
                                                            const WT *__restrict__ W,
                                                            WT *__restrict__ Wt, PrepGrad pg,
                                                            int64_t n_grad) {
    extern __shared__ int sh[];
    __shared__ WT buf[32][33];
    const int blk = blockIdx.x;
    if (blk < n_sort) {
        sort_sample<KS>(C, blk, N_in, t_in, srt, n_valid, deriv, xo, sh);
    } else if (blk < n_sort + n_tr) {
        transpose_tile<WT, kPrepThreads>(N_out, N_in, W, Wt, blk - n_sort, buf);
    } else {
        const int64_t n_gb = (n_grad + kPrepThreads - 1) / kPrepThreads;
        const int64_t gb = blk - n_sort - n_tr;
        if (gb >= n_gb) {
            // silent-sample count of neuron i over the batch (dead-neuron term)
            const int i = static_cast<int>((gb - n_gb) * kPrepThreads + threadIdx.x);
            if (i < N_out) {
                int cnt = 0;
                for (int b = 0; b < pg.B; ++b)
                    cnt += (pg.q_idx[static_cast<int64_t>(b) * N_out + i] < 0) ? 1 : 0;
                pg.sf.dq[i] = -(pg.sf.gq * pg.sf.scale * static_cast<float>(cnt));
            }
            return;
        }
        const int64_t k = gb * kPrepThreads + threadIdx.x;
        if (k < n_grad) {
            const int q = pg.q_idx[k];
            GradPrep gp{0.f, 0.f, -1};
            if (q >= 0) {  // silent neurons: no further loads
                float g = pg.grad_t[k];
                // the spike time only where it is used (no gradient: no load)
                const float t = (pg.sf.on || g != 0.f) ? pg.t_out[k] : 0.f;
                if (pg.sf.on) g += synfire_dt(pg.sf, t);
                if (g != 0.f) gp = grad_prep(C, t, pg.slope[k], q, g);
            }
            pg.gam[k] = gp.gam;
            pg.uq[k] = gp.uq;
            pg.q[k] = gp.q;
        }
    }
}

// --------------------------------------------------------------- forward --
// Lane = neuron i of a 64-neuron tile, one sample per wavefront (4 per block).
// The wave walks its sample's events in grid order: each record adds
// W[i, j] L and W[i, j] R to the running sums of its row (WT row j is one
// coalesced 256-byte load with a scalar base). When a row closes, grid point
// m = row - 1 is complete (its L parts come from this row, its R parts from
// the previous one) and goes straight into the interval scan: the weighted
// events never exist in memory. Once every lane has found its crossing
// interval, later events cannot change the outputs and the wave stops.

template <typename WT, int KS>
__global__ __launch_bounds__(256) void fwd_sorted_kernel(LifConst C, int B, int N_in, int N_out,
                                                         const WT *__restrict__ Wt,
                                                         SortedEv srt,
                                                         const int *__restrict__ n_valid,
                                                         float *__restrict__ t_out,
                                                         float *__restrict__ slope,
                                                         int *__restrict__ q_idx) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int waves = blockDim.x >> 6;
    const int i = blockIdx.x * kWave + lane;
    const bool row_ok = i < N_out;
    const int b = uniform(blockIdx.y * waves + wave);
    if (b >= B) return;  // wave-uniform; the kernel has no block barrier
    const int n = *as_const(n_valid + b);
    Scan<KS> sc;
    walk_sorted_rows<WT, false>(C, N_in, N_out, Wt, srt, b, n, i, row_ok, 1, sc);
    if (!row_ok) return;
    float to, sl;
    int q;
    sc.finish(C, to, sl, q);
    const int64_t o = static_cast<int64_t>(b) * N_out + i;
    t_out[o] = to;
    slope[o] = sl;
    q_idx[o] = q;
}


// ----------------------------------------------------------------- dW ----
// dW[i, j] = sum_b (G[b, r_bj, i] L_bj + G[b, r_bj + 1, i] R_bj).
// Lane = input j (events are coalesced vector loads); a block covers
// 4 x 64 inputs and a tile of TI neurons whose sums stay in registers over
// its share of the batch. G[b, :, tile] is computed in place from the
// gradient triples (each thread owns one neuron and a fixed set of rows, so
// neurons without gradient cost no exponential) and staged in LDS (double
// buffered) as rows of dw_stride floats, G[r][neuron]: a thread reads the
// two halves of its event, rows r and r+1, per neuron (or four neurons per
// 16-byte read, see dw_stride). Rows
// R-1 and R stay zero (R-1 is the point after the grid; slot R-1 serves
// inputs without events). The next sample's G values and events are fetched
// while this one is consumed; a sample whose tile is all zero is skipped.
// Batch splits write partial sums, reduced in order.
// LDS row stride (floats) of the dW kernel's G buffers for a TI-neuron tile.
// One sample group per block reads four neurons per 16-byte LDS read (rows
// padded to stay 16-byte aligned); two groups read one neuron of both halves
// per two-address read over an odd stride (measured faster there: mlp3's
// layers with two groups 0.069 ms against 0.093 ms, the 4096-wide layer
// with one group 1.18 ms against 1.48 ms).
constexpr bool dw_vec(int groups) { return groups == 1; }
constexpr int dw_stride(int ti, int groups) { return dw_vec(groups) ? ti + 4 : ti + 1; }

template <int TI, int NPER, int GW, int KS, int IPT>
__global__ __launch_bounds__(256 * GW) void dw_dense_kernel(LifConst C, int B, int N_in, int N_out,
                                                             int b_per_split,
                                                             const float *__restrict__ gam,
                                                             const float *__restrict__ uq,
                                                             const int *__restrict__ qv,
                                                             const int *__restrict__ ev_row,
                                                             const float *__restrict__ ev_L,
                                                             const float *__restrict__ ev_R,
                                                             const float *__restrict__ dq,
                                                             float *__restrict__ dW_part) {
    // IPT inputs per thread (j, j + 256, ...): the G tile staged per sample
    // serves IPT times as many multiply-adds (one sample group only)
    static_assert(IPT == 1 || GW == 1, "several inputs per thread with one sample group only");
    extern __shared__ float gs[];  // [GW][2][R + 1][dw_stride(TI, GW)]
    __shared__ int wlive[2][4 * GW];
    constexpr int kStr = dw_stride(TI, GW);
    const int R = rows_of(C);
    const int gbuf = (R + 1) * kStr;
    const int grp = threadIdx.x >> 8;  // sample group of this thread
    const int tid = threadIdx.x & 255;
    float *gsg = gs + grp * 2 * gbuf;
    const int jb = blockIdx.x * 256 * IPT + tid;
    const int i0 = blockIdx.y * TI;
    const int ni = min(TI, N_out - i0);
    // the block's samples [b0, b_end); group g takes b0 + g, b0 + g + GW, ...
    const int b0 = blockIdx.z * b_per_split;
    const int b_end = min(B, b0 + b_per_split);
    const int n_it = (b_per_split + GW - 1) / GW;  // iterations, equal for every group
    float acc[IPT][TI];
#pragma unroll
    for (int k = 0; k < IPT; ++k)
#pragma unroll
        for (int ii = 0; ii < TI; ++ii) acc[k][ii] = 0.f;
    const int total = R * TI;
    // element c of this thread: row r = r_first + c * (256 / TI), neuron l
    const int l_own = tid % TI, r_first = tid / TI;
    constexpr int kRowStep = 256 / TI;
    const GStep gst = g_step<KS>(C, kRowStep);
    float pre[NPER];
    auto sample = [&](int it) { return b0 + grp + it * GW; };
    // gradient triple of this thread's neuron in sample b (q = -1: none, or
    // past the block's share); loaded two samples ahead of its use
    struct Tri { float gm, u; int q; };
    auto load_tri = [&](int b) {
        Tri t{0.f, 0.f, -1};
        if (l_own < ni && b < b_end) {
            const int64_t k = static_cast<int64_t>(b) * N_out + i0 + l_own;
            t.gm = gam[k];
            t.u = uq[k];
            t.q = qv[k];
        }
        return t;
    };
    auto fetch = [&](const Tri &t) {
        g_strided<NPER, KS>(C, gst, t.gm, t.u, t.q, r_first - 1, kRowStep, pre);
        bool nz = false;
#pragma unroll
        for (int c = 0; c < NPER; ++c) nz = nz || pre[c] != 0.f;
        return nz;
    };
    auto store = [&](float *buf) {
#pragma unroll
        for (int c = 0; c < NPER; ++c) {
            const int k = tid + c * 256;
            if (k < total) {
                const int r = k / TI, l = k % TI;
                if (r < R - 1) buf[r * kStr + l] = pre[c];
            }
        }
    };
    // event of (b, j): slot (row) and halves; no events: slot R-1, zeros
    auto event = [&](int b, int j, int &slot, float &L, float &Rv) {
        slot = R - 1;
        L = 0.f;
        Rv = 0.f;
        if (j < N_in && b < b_end) {
            const int64_t o = static_cast<int64_t>(b) * N_in + j;
            const int r = ev_row[o];
            if (r >= 0) {
                slot = r;
                L = ev_L[o];
                Rv = ev_R[o];
            }
        }
    };
    // whether any thread of this group has a nonzero G tile for the next
    // sample: wave votes through LDS, double buffered by iteration parity
    auto group_live = [&](bool v, int par) {
        const int wv = threadIdx.x >> 6;
        const bool any = __any(v);
        if ((threadIdx.x & (kWave - 1)) == 0) wlive[par][wv] = any ? 1 : 0;
        __syncthreads();
        const int g0 = grp * 4;
        return (wlive[par][g0] | wlive[par][g0 + 1] | wlive[par][g0 + 2] | wlive[par][g0 + 3]) != 0;
    };
    for (int k = tid; k < 2 * 2 * kStr; k += 256)
        gsg[(k / (2 * kStr)) * gbuf + (R - 1) * kStr + k % (2 * kStr)] = 0.f;
    bool live = false;
    if (n_it > 0) {
        live = fetch(load_tri(sample(0)));
        store(gsg);
    }
    Tri tri_n = load_tri(sample(1));
    int slot_n[IPT];
    float L_n[IPT], R_n[IPT];
#pragma unroll
    for (int k = 0; k < IPT; ++k) event(sample(0), jb + k * 256, slot_n[k], L_n[k], R_n[k]);
    live = group_live(live, 0);
    for (int it = 0; it < n_it; ++it) {
        const float *cur = gsg + (it & 1) * gbuf;
        const bool more = it + 1 < n_it;
        int slot[IPT];
        float L[IPT], Rv[IPT];
#pragma unroll
        for (int k = 0; k < IPT; ++k) {
            slot[k] = slot_n[k];
            L[k] = L_n[k];
            Rv[k] = R_n[k];
            event(sample(it + 1), jb + k * 256, slot_n[k], L_n[k], R_n[k]);
        }
        const Tri tri = tri_n;
        tri_n = load_tri(sample(it + 2));
        bool live_next = false;
        if (more) live_next = fetch(tri);
        if (live) {
            if constexpr (dw_vec(GW)) {
#pragma unroll
                for (int k = 0; k < IPT; ++k) {
                    const float4 *p = reinterpret_cast<const float4 *>(cur + slot[k] * kStr);
                    float *a_k = acc[k];
#pragma unroll
                    for (int i4 = 0; i4 < TI / 4; ++i4) {
                        const float4 a = p[i4], c = p[i4 + kStr / 4];
                        a_k[4 * i4] = fmaf(a.x, L[k], fmaf(c.x, Rv[k], a_k[4 * i4]));
                        a_k[4 * i4 + 1] = fmaf(a.y, L[k], fmaf(c.y, Rv[k], a_k[4 * i4 + 1]));
                        a_k[4 * i4 + 2] = fmaf(a.z, L[k], fmaf(c.z, Rv[k], a_k[4 * i4 + 2]));
                        a_k[4 * i4 + 3] = fmaf(a.w, L[k], fmaf(c.w, Rv[k], a_k[4 * i4 + 3]));
                    }
                }
            } else {
                const float *p = cur + slot[0] * kStr;
#pragma unroll
                for (int ii = 0; ii < TI; ++ii)
                    acc[0][ii] = fmaf(p[ii], L[0], fmaf(p[ii + kStr], Rv[0], acc[0][ii]));
            }
        }
        if (more) store(gsg + ((it + 1) & 1) * gbuf);
        live = group_live(live_next, (it + 1) & 1);
    }
    if (GW > 1) {
        // groups 1 .. GW-1 hand their sums to group 0 through the (now idle)
        // G buffers, kCh per thread per round; group 0 adds them in group order
        constexpr int kCh = (TI < 16) ? TI : 16;
        float *xch = gs;
#pragma unroll
        for (int c0 = 0; c0 < TI; c0 += kCh) {
            __syncthreads();
            if (grp > 0) {
#pragma unroll
                for (int c = 0; c < kCh; ++c) xch[((grp - 1) * kCh + c) * 256 + tid] = acc[0][c0 + c];
            }
            __syncthreads();
            if (grp == 0) {
#pragma unroll
                for (int c = 0; c < kCh; ++c)
                    for (int g = 1; g < GW; ++g) acc[0][c0 + c] += xch[((g - 1) * kCh + c) * 256 + tid];
            }
        }
        if (grp > 0) return;
    }
#pragma unroll
    for (int k = 0; k < IPT; ++k) {
        const int j = jb + k * 256;
        if (j >= N_in) continue;
        float *out = dW_part + static_cast<int64_t>(blockIdx.z) * N_out * N_in +
                     static_cast<int64_t>(i0) * N_in + j;
        // dq: the dead-neuron term of each row, added to the final sums (one
        // split only; with splits the reduction adds it)
#pragma unroll
        for (int ii = 0; ii < TI; ++ii)
            if (ii < ni) out[static_cast<int64_t>(ii) * N_in] = dq ? acc[k][ii] + dq[i0 + ii] : acc[k][ii];
    }
}

// dW[k] = sum of the split partials in split order (+ the row's dead-neuron
// term dq[k / row_len] when dq is set). Thread t takes outputs 4t .. 4t+3:
// one 16-byte load per split where n is a multiple of 4 (every partial
// then starts 16-byte aligned), with the split loop unrolled so that four
// splits' loads are in flight together; the additions keep split order.
__device__ __forceinline__ void reduce_parts4(int64_t n, int nsplit, const float *__restrict__ part,
                                              const float *__restrict__ dq, int row_len,
                                              float *__restrict__ out, int64_t t) {
    const int64_t k = 4 * t;
    if (k >= n) return;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    if ((n & 3) == 0) {
        int z = 0;
        for (; z + 4 <= nsplit; z += 4) {
            float4 a[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                a[u] = *reinterpret_cast<const float4 *>(part + static_cast<int64_t>(z + u) * n + k);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                s[0] += a[u].x;
                s[1] += a[u].y;
                s[2] += a[u].z;
                s[3] += a[u].w;
            }
        }
        for (; z < nsplit; ++z) {
            const float4 a = *reinterpret_cast<const float4 *>(part + static_cast<int64_t>(z) * n + k);
            s[0] += a.x;
            s[1] += a.y;
            s[2] += a.z;
            s[3] += a.w;
        }
    } else {
        for (int z = 0; z < nsplit; ++z)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (k + c < n) s[c] += part[static_cast<int64_t>(z) * n + k + c];
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (k + c < n) out[k + c] = dq ? s[c] + dq[(k + c) / row_len] : s[c];
}

__global__ __launch_bounds__(256) void reduce_splits_kernel(int64_t n, int nsplit,
                                                            const float *__restrict__ part,
                                                            const float *__restrict__ dq,
                                                            int row_len,
                                                            float *__restrict__ out) {
    reduce_parts4(n, nsplit, part, dq, row_len, out,
                  static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x);
}

// -------------------------------------------------------- dt_in (rows) --
// dt_in of every input with events, from its sample's row-sorted records
// {j, row r, dL, dR}: dL sum_i W[i, j] G[b, m = r-1, i] + dR sum_i W[i, j] G[b, m = r, i],
// G evaluated in place from the gradient triples (once per event row for the
// first 4 * NTW tiles of neurons).
// A block takes a contiguous range of whole event rows of one sample
// (kDtRanges ranges per sample, about equal in records); its four waves walk
// the same records, each over its own NTW 64-neuron tiles per group of
// 4 * NTW tiles (lane = neuron: WT row j is one coalesced load per tile).
// Records go 8 at a time: each wave reduces its lanes (fixed butterfly), the
// four wave sums are added in wave order through LDS. Inputs without events
// are not visited (their dt_in was zeroed earlier).
constexpr int kDtRanges = 6;

// The launch may carry extra blocks (blockIdx.y >= B) that finish the dW
// split reduction of the same layer (independent work, one launch less).
struct RedJob { int64_t n; int nsplit; const float *part; float *out; const float *dq; int row_len; };

// VEC: lane l of wave w takes the NTW neighbouring neurons w*NTW*64 + NTW*l
// + t of each group (one NTW-wide weight load per record; N_out % NTW == 0),
// else neurons (w*NTW + t)*64 + l.
template <typename WT, int NTW, int KS, bool VEC>
__global__ __launch_bounds__(256) void dtin_rows_kernel(LifConst C, int B, int N_in, int N_out,
                                                        const WT *__restrict__ Wt, SortedEv srt,
                                                        const float *__restrict__ gam,
                                                        const float *__restrict__ uq,
                                                        const int *__restrict__ qv,
                                                        float *__restrict__ dt_in, RedJob red) {
    __shared__ float part[4][kBatch];
    if (static_cast<int>(blockIdx.y) >= B) {
        reduce_parts4(red.n, red.nsplit, red.part, red.dq, red.row_len, red.out,
                      (static_cast<int64_t>(blockIdx.y - B) * gridDim.x + blockIdx.x) * blockDim.x +
                          threadIdx.x);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int range = blockIdx.x;
    const int b = blockIdx.y;
    const int R = rows_of(C);
    const int *rs = srt.rs + static_cast<int64_t>(b) * (R + 1);
    const int n = *as_const(rs + R);
    const RowRange rg = row_range(rs, R, n, static_cast<int>((static_cast<int64_t>(n) * range) / kDtRanges),
                                  static_cast<int>((static_cast<int64_t>(n) * (range + 1)) / kDtRanges),
                                  range == 0, range == kDtRanges - 1, lane);
    const int r_lo = uniform(rg.ra), r_hi = uniform(rg.rb);
    if (uniform(rg.ka) == uniform(rg.kb)) return;  // block-uniform: no records
    const int64_t eo = static_cast<int64_t>(b) * srt.stride;
    const int *ej = srt.j + eo;
    const float *edl = srt.L + eo;
    const float *edr = srt.R + eo;
    const int64_t nb = static_cast<int64_t>(b) * N_out;
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(Wt, static_cast<uint32_t>(static_cast<int64_t>(N_in) * N_out * sizeof(WT)));
    const int rstride = N_out * static_cast<int>(sizeof(WT));
    const unsigned jmax = static_cast<unsigned>(max(N_in - 1, 0));
    constexpr int kGroup = 4 * NTW * kWave;
    const int ngroups = (N_out + kGroup - 1) / kGroup;
    auto neuron = [&](int grp, int t) {
        return grp * kGroup + (VEC ? (wave * NTW * kWave + NTW * lane + t) : ((wave * NTW + t) * kWave + lane));
    };
    // VEC loads past N_out read the next row's weights or zeros; those
    // neurons have G = 0
    auto voffv = [&](int grp) { return neuron(grp, 0) * static_cast<int>(sizeof(WT)); };
    // this lane's neurons of group 0 (the only group when N_out <= kGroup)
    float gm0[NTW], ua0[NTW];
    int qa0[NTW], voff0[NTW];
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
        const int i = neuron(0, t);
        const int ic = min(i, N_out - 1);
        const bool ok = i < N_out;
        gm0[t] = ok ? gam[nb + ic] : 0.f;
        ua0[t] = ok ? uq[nb + ic] : 0.f;
        qa0[t] = ok ? qv[nb + ic] : -1;
        voff0[t] = ic * static_cast<int>(sizeof(WT));
    }
    for (int r = r_lo; r < r_hi; ++r) {
        const int s = *as_const(rs + r), e = *as_const(rs + r + 1);
        if (s == e) continue;
        // G at grid points r - 1 (L halves) and r (R halves), group 0
        float h0[NTW], h1[NTW];
#pragma unroll
        for (int t = 0; t < NTW; ++t) {
            h0[t] = g_at<KS>(C, gm0[t], ua0[t], qa0[t], r - 1);
            h1[t] = g_at<KS>(C, gm0[t], ua0[t], qa0[t], r);
        }
        for (int k0 = s; k0 < e; k0 += kBatch) {
            const int nk = min(kBatch, e - k0);
            int jo[kBatch];
            float dl[kBatch], dr[kBatch], v[kBatch];
#pragma unroll
            for (int kk = 0; kk < kBatch; ++kk) {
                jo[kk] = static_cast<int>(min(static_cast<unsigned>(as_const(ej + k0)[kk]), jmax)) * rstride;
                dl[kk] = as_const(edl + k0)[kk];
                dr[kk] = as_const(edr + k0)[kk];
                v[kk] = 0.f;
            }
            for (int grp = 0; grp < ngroups; ++grp) {
                float g0[NTW], g1[NTW], w[kBatch][NTW];
                int voff[NTW];
#pragma unroll
                for (int t = 0; t < NTW; ++t) {
                    if (grp == 0) {
                        g0[t] = h0[t];
                        g1[t] = h1[t];
                        voff[t] = voff0[t];
                    } else {
                        const int i = neuron(grp, t);
                        const int ic = min(i, N_out - 1);
                        const bool ok = i < N_out;
                        const float gm = ok ? gam[nb + ic] : 0.f;
                        const float u = ok ? uq[nb + ic] : 0.f;
                        const int q = ok ? qv[nb + ic] : -1;
                        g0[t] = g_at<KS>(C, gm, u, q, r - 1);
                        g1[t] = g_at<KS>(C, gm, u, q, r);
                        voff[t] = ic * static_cast<int>(sizeof(WT));
                    }
                }
                if constexpr (VEC) {
                    const int vo = voffv(grp);
#pragma unroll
                    for (int kk = 0; kk < kBatch; ++kk) BufLoadN<WT, NTW>::get(wr, vo, jo[kk], w[kk]);
                } else {
#pragma unroll
                    for (int kk = 0; kk < kBatch; ++kk)
#pragma unroll
                        for (int t = 0; t < NTW; ++t) w[kk][t] = BufLoad<WT>::get(wr, voff[t], jo[kk]);
                }
#pragma unroll
                for (int kk = 0; kk < kBatch; ++kk)
#pragma unroll
                    for (int t = 0; t < NTW; ++t)
                        v[kk] = fmaf(w[kk][t], fmaf(dl[kk], g0[t], dr[kk] * g1[t]), v[kk]);
            }
            // lane 8kk ends with record kk's sum over this wave's neurons
            static_assert(kBatch == 8, "wave_sum8 reduces eight records");
            const float tot = wave_sum8(v, lane);
            if ((lane & 7) == 0) part[wave][lane >> 3] = tot;
            __syncthreads();
            if (wave == 0 && lane < nk) {
                int jl = 0;
#pragma unroll
                for (int kk = 0; kk < kBatch; ++kk) {
                    const int jk = as_const(ej + k0)[kk];
                    if (lane == kk) jl = jk;
                }
                dt_in[static_cast<int64_t>(b) * N_in + jl] =
                    ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
            }
            __syncthreads();
        }
    }
}

// dt_in for a layer of at most 64 neurons (one tile, lane = neuron): the
// block's four waves take turns over its range's records, kBatch at a time,
// so no wave walks an empty tile and no block-wide combine is needed. G at
// the grid points the range's rows read (points r_lo - 1 .. r_hi - 1) is
// evaluated once per block into LDS; record k of a batch adds
// W[i, j] (dL G[r-1] + dR G[r]) on its lane and the wave sums the lanes.
// The per-record arithmetic and its order are those of dtin_rows_kernel.
template <typename WT, int KS>
__global__ __launch_bounds__(256) void dtin_tile_kernel(LifConst C, int B, int N_in, int N_out,
                                                        const WT *__restrict__ Wt, SortedEv srt,
                                                        const float *__restrict__ gam,
                                                        const float *__restrict__ uq,
                                                        const int *__restrict__ qv,
                                                        float *__restrict__ dt_in, RedJob red) {
    extern __shared__ float gtab[];  // [r - r_lo][64]: G at point r - 1, r_lo <= r <= r_hi
    if (static_cast<int>(blockIdx.y) >= B) {
        reduce_parts4(red.n, red.nsplit, red.part, red.dq, red.row_len, red.out,
                      (static_cast<int64_t>(blockIdx.y - B) * gridDim.x + blockIdx.x) * blockDim.x +
                          threadIdx.x);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int nw = blockDim.x >> 6;
    const int range = blockIdx.x;
    const int b = blockIdx.y;
    const int R = rows_of(C);
    const int *rs = srt.rs + static_cast<int64_t>(b) * (R + 1);
    const int n = *as_const(rs + R);
    const RowRange rg = row_range(rs, R, n, static_cast<int>((static_cast<int64_t>(n) * range) / kDtRanges),
                                  static_cast<int>((static_cast<int64_t>(n) * (range + 1)) / kDtRanges),
                                  range == 0, range == kDtRanges - 1, lane);
    const int r_lo = uniform(rg.ra), r_hi = uniform(rg.rb);
    const int k_lo = uniform(rg.ka), k_hi = uniform(rg.kb);
    if (k_lo == k_hi) return;  // block-uniform: no records
    const int64_t nb = static_cast<int64_t>(b) * N_out;
    const bool ok = lane < N_out;
    const int ic = min(lane, N_out - 1);
    const float gm = ok ? gam[nb + ic] : 0.f;
    const float ua = ok ? uq[nb + ic] : 0.f;
    const int qa = ok ? qv[nb + ic] : -1;
    for (int r = r_lo + wave; r <= r_hi; r += nw) gtab[(r - r_lo) * kWave + lane] = g_at<KS>(C, gm, ua, qa, r - 1);
    __syncthreads();
    const int64_t eo = static_cast<int64_t>(b) * srt.stride;
    const int *ej = srt.j + eo;
    const int *er = srt.r + eo;
    const float *edl = srt.L + eo;
    const float *edr = srt.R + eo;
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(Wt, static_cast<uint32_t>(static_cast<int64_t>(N_in) * N_out * sizeof(WT)));
    const int rstride = N_out * static_cast<int>(sizeof(WT));
    const unsigned jmax = static_cast<unsigned>(max(N_in - 1, 0));
    const int voff = ic * static_cast<int>(sizeof(WT));
    static_assert(kBatch == 8, "wave_sum8 reduces eight records");
    for (int k0 = k_lo + wave * kBatch; k0 < k_hi; k0 += nw * kBatch) {
        const int nk = min(kBatch, k_hi - k0);
        float w[kBatch], v[kBatch];
#pragma unroll
        for (int kk = 0; kk < kBatch; ++kk) {
            const int jo = static_cast<int>(min(static_cast<unsigned>(as_const(ej + k0)[kk]), jmax)) * rstride;
            w[kk] = BufLoad<WT>::get(wr, voff, jo);
        }
#pragma unroll
        for (int kk = 0; kk < kBatch; ++kk) {
            v[kk] = 0.f;
            if (kk < nk) {
                const int r = as_const(er + k0)[kk];
                const float g0 = gtab[(r - r_lo) * kWave + lane];
                const float g1 = gtab[(r - r_lo + 1) * kWave + lane];
                v[kk] = fmaf(w[kk], fmaf(as_const(edl + k0)[kk], g0, as_const(edr + k0)[kk] * g1), 0.f);
            }
        }
        const float tot = wave_sum8(v, lane);
        const int kl = lane >> 3;
        if ((lane & 7) == 0 && kl < nk) dt_in[static_cast<int64_t>(b) * N_in + ej[k0 + kl]] = tot;
    }
}

// ---------------------------------------------------------------- losses --
// One block per sample; block reductions run over a fixed LDS tree, so the
// per-sample losses (loss[1 + b]) and their fixed-order sum (loss[0]) are
// deterministic.
constexpr int kLossThreads = 256;

__device__ __forceinline__ float block_reduce(float v, float *red, bool is_max) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = kLossThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w)
            red[threadIdx.x] = is_max ? fmaxf(red[threadIdx.x], red[threadIdx.x + w])
                                      : red[threadIdx.x] + red[threadIdx.x + w];
        __syncthreads();
    }
    const float r = red[0];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(kLossThreads) void softmax_ce_kernel(int B, int N,
                                                                  const float *__restrict__ t,
                                                                  const int *__restrict__ labels,
                                                                  float tau_soft, float t_cap,
                                                                  float *__restrict__ grad,
                                                                  float *__restrict__ loss) {
    __shared__ float red[kLossThreads];
    const int b = blockIdx.x;
    const float inv = 1.f / tau_soft;
    const float *tb = t + static_cast<int64_t>(b) * N;
    float *gb = grad + static_cast<int64_t>(b) * N;
    float mx = -INFINITY;
    for (int k = threadIdx.x; k < N; k += kLossThreads) {
        const float tk = isfinite(tb[k]) ? tb[k] : t_cap;
        mx = fmaxf(mx, -tk * inv);
    }
    mx = block_reduce(mx, red, true);
    float z = 0.f;
    for (int k = threadIdx.x; k < N; k += kLossThreads) {
        const float tk = isfinite(tb[k]) ? tb[k] : t_cap;
        z += expf(-tk * inv - mx);
    }
    z = block_reduce(z, red, false);
    const int lab = labels[b];
    const float lz = logf(z) + mx;
    for (int k = threadIdx.x; k < N; k += kLossThreads) {
        const bool fired = isfinite(tb[k]);
        const float tk = fired ? tb[k] : t_cap;
        const float sk = expf(-tk * inv - lz);
        const float dl = (sk - (k == lab ? 1.f : 0.f)) * (-inv) / static_cast<float>(B);
        gb[k] = fired ? dl : 0.f;
    }
    if (threadIdx.x == 0) {
        const float tl = isfinite(tb[lab]) ? tb[lab] : t_cap;
        loss[1 + b] = (lz + tl * inv) / static_cast<float>(B);
    }
}

__global__ __launch_bounds__(kLossThreads) void mse_kernel(int B, int N, const float *__restrict__ t,
                                                           const float *__restrict__ y,
                                                           float *__restrict__ grad,
                                                           float *__restrict__ loss) {
    __shared__ float red[kLossThreads];
    const int b = blockIdx.x;
    float acc = 0.f;
    for (int k = threadIdx.x; k < N; k += kLossThreads) {
        const int64_t o = static_cast<int64_t>(b) * N + k;
        const bool fired = isfinite(t[o]);
        const float d = fired ? (t[o] - y[o]) : 0.f;
        grad[o] = d / static_cast<float>(B);
        acc += 0.5f * d * d / static_cast<float>(B);
    }
    acc = block_reduce(acc, red, false);
    if (threadIdx.x == 0) loss[1 + b] = acc;
}

// loss[0] = sum_b loss[1 + b] in a fixed order
__global__ __launch_bounds__(kLossThreads) void loss_total_kernel(int B, float *__restrict__ loss) {
    __shared__ float red[kLossThreads];
    float acc = 0.f;
    for (int b = threadIdx.x; b < B; b += kLossThreads) acc += loss[1 + b];
    acc = block_reduce(acc, red, false);
    if (threadIdx.x == 0) loss[0] = acc;
}

// ------------------------------------------------------------- launchers --
static int tiles32(int64_t N_in, int64_t N_out) {
    return static_cast<int>(((N_in + 31) / 32) * ((N_out + 31) / 32));
}

static size_t sort_lds_bytes(const LifConst &C) {
    const int R = C.M + 3;
    return static_cast<size_t>(kSortWaves * R + R + 1) * sizeof(int);
}

static hipError_t launch_prep(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                              const float *t_in, SortedEv srt, int *n_valid, bool deriv, SortOut xo,
                              const void *W, bool bf16, void *Wt, bool transpose, PrepGrad pg,
                              int64_t n_grad, const char *name, hipStream_t st) {
    const int n_tr = (transpose && N_in * N_out > 0) ? tiles32(N_in, N_out) : 0;
    const int64_t n_gb = (n_grad + kPrepThreads - 1) / kPrepThreads;
    const int64_t n_db = (pg.sf.on && pg.sf.dq) ? (N_out + kPrepThreads - 1) / kPrepThreads : 0;
    const int64_t blocks = B + n_tr + n_gb + n_db;
    if (blocks == 0) return hipSuccess;
    ProfScope prof(name, st);
#define PREP(WTY, KSV)                                                                             \
    hipLaunchKernelGGL((prep_kernel<WTY, KSV>), dim3(static_cast<unsigned>(blocks)),              \
                       dim3(kPrepThreads), sort_lds_bytes(C), st, C, static_cast<int>(B), n_tr,   \
                       static_cast<int>(N_in), static_cast<int>(N_out), t_in, srt, n_valid,        \
                       deriv ? 1 : 0, xo, static_cast<const WTY *>(W), static_cast<WTY *>(Wt), pg, \
                       n_grad)
    const bool gen = C.kind == kGeneral;
    if (bf16) {
        if (gen) PREP(uint16_t, kGeneral); else PREP(uint16_t, kAnyKind);
    } else {
        if (gen) PREP(float, kGeneral); else PREP(float, kAnyKind);
    }
#undef PREP
    return hipGetLastError();
}

hipError_t launch_sort_records(const LifConst &C, int64_t B, int64_t n_rec, const float *t_in,
                               SortedEv srt, int *n_valid, const char *name, hipStream_t st) {
    return launch_prep(C, B, n_rec, 0, t_in, srt, n_valid, false,
                       SortOut{nullptr, nullptr, nullptr, nullptr}, nullptr, false, nullptr, false,
                       PrepGrad{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                Synfire{}, 0},
                       0, name, st);
}

hipError_t launch_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const void *W,
                          bool bf16, void *Wt, SortedEv srt, int *n_valid, const float *t_in,
                          float *t_out, float *slope, int *q_idx, hipStream_t st) {
    const int R = C.M + 3;
    hipError_t e = launch_prep(C, B, N_in, N_out, t_in, srt, n_valid, false,
                               SortOut{nullptr, nullptr, nullptr, nullptr}, W, bf16, Wt, true,
                               PrepGrad{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                        Synfire{}, 0},
                               0, "sort_transpose", st);
    if (e != hipSuccess) return e;
    ProfScope prof("fwd_dense", st);
    if (C.M <= kRowsMaxM) {
        const int nt = rows_nt(N_out, R);
        const int tiles = static_cast<int>((N_out + kWave - 1) / kWave);
        dim3 grid(static_cast<unsigned>((tiles + nt - 1) / nt), static_cast<unsigned>(B));
        const size_t lds = rows_lds(nt, R);
        // NT neighbouring neurons per lane where rows keep NT-wide loads aligned
        const bool vec = (N_out % nt) == 0;
#define FWR_KV(WTY, NTV, KSV, VECV)                                                               \
    hipLaunchKernelGGL((fwd_rows_kernel<WTY, NTV, KSV, VECV, RowOutTtfs>), grid,                 \
                       dim3(kRowWaves * kWave), lds, st, C, static_cast<int>(N_in),               \
                       static_cast<int>(N_out), static_cast<const WTY *>(Wt), srt,                \
                       RowOutTtfs{t_out, slope, q_idx})
#define FWR_K(WTY, NTV, KSV)                      \
    do {                                          \
        if (vec) FWR_KV(WTY, NTV, KSV, true);     \
        else FWR_KV(WTY, NTV, KSV, false);        \
    } while (0)
#define FWR(WTY, NTV)                                                     \
    do {                                                                  \
        if (C.kind == kGeneral) FWR_K(WTY, NTV, kGeneral);                \
        else FWR_K(WTY, NTV, kAnyKind);                                   \
    } while (0)
        if (bf16) {
            if (nt == 4) FWR(uint16_t, 4);
            else if (nt == 2) FWR(uint16_t, 2);
            else FWR(uint16_t, 1);
        } else {
            if (nt == 4) FWR(float, 4);
            else if (nt == 2) FWR(float, 2);
            else FWR(float, 1);
        }
#undef FWR
#undef FWR_K
#undef FWR_KV
        return hipGetLastError();
    }
    constexpr int waves = 4;
    dim3 grid(static_cast<unsigned>((N_out + kWave - 1) / kWave),
              static_cast<unsigned>((B + waves - 1) / waves));
#define FWS(WTY, KSV)                                                                           \
    hipLaunchKernelGGL((fwd_sorted_kernel<WTY, KSV>), grid, dim3(waves * kWave), 0, st, C,      \
                       static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),     \
                       static_cast<const WTY *>(Wt), srt, n_valid, t_out, slope, q_idx)
    const bool gen = C.kind == kGeneral;
    if (bf16) {
        if (gen) FWS(uint16_t, kGeneral); else FWS(uint16_t, kAnyKind);
    } else {
        if (gen) FWS(float, kGeneral); else FWS(float, kAnyKind);
    }
#undef FWS
    return hipGetLastError();
}

// neuron tile: 64, or 32 where two 64-wide G buffers would pass 48 KB of
// LDS; narrower (16 or 32) where the layer has no more neurons than that, so
// a sample's G reads and multiply-adds are not spent on empty columns
static int dw_ti(int M, int64_t N_out) {
    if (N_out <= 16) return 16;
    if (N_out <= 32) return 32;
    return (2 * (M + 4) * dw_stride(64, 1) * 4 <= 48 * 1024) ? 64 : 32;
}

// register slots per thread for staging one tile (R * TI values / 256 threads)
static int dw_nper(int M, int ti) {
    const int need = ((M + 3) * ti + 255) / 256;
    for (int n : {9, 17, 33}) if (need <= n) return n;
    return -1;
}

// Batch splits: enough that the grid holds ~4 groups of 4 waves per CU
// (256 CUs), keeping >= 4 samples per group. Where that takes 4 or more
// splits (and two groups' G buffers fit 64 KB), blocks carry two sample
// groups (8 waves) and half the splits: the same waves in flight, half the
// partials to write and read back.
DwPlan plan_dw(int64_t B, int64_t N_in, int64_t N_out, int M) {
    DwPlan p;
    p.jw = dw_ti(M, N_out);
    p.ipt = 1;
    const int64_t tiles = ((N_in + 255) / 256) * ((N_out + p.jw - 1) / p.jw);
    p.nsplit = 1;
    while (tiles * p.nsplit < 1024 && B / (p.nsplit * 2) >= 4) p.nsplit *= 2;
    const size_t g_lds = 2 * static_cast<size_t>(M + 4) * dw_stride(p.jw, 2) * sizeof(float);  // one of two groups
    const int groups = (p.nsplit >= 4 && 2 * g_lds <= 64 * 1024) ? 2 : 1;
    p.nsplit /= groups;
    p.waves = 4 * groups;
    p.b_per_split = static_cast<int>(std::max<int64_t>(1, (B + p.nsplit - 1) / p.nsplit));
    p.nsplit = static_cast<int>(std::max<int64_t>(1, (B + p.b_per_split - 1) / p.b_per_split));
    // large layers with one sample group and 64-neuron tiles: two inputs per
    // thread, so each staged G tile serves twice the multiply-adds (the G
    // work per sample grows with M; measured on the 4096-wide layer: dW
    // 1.18 -> 0.91 ms at M = 64, slower at M = 8 and 32)
    if (groups == 1 && p.nsplit == 1 && p.jw == 64 && M >= 64 && N_out >= 1024 && N_in >= 1024)
        p.ipt = kDwWideIPT;
    return p;
}

static hipError_t launch_dw(const LifConst &C, const DwPlan &p, int64_t B, int64_t N_in,
                            int64_t N_out, const DenseBwdWs &ws, const float *dq, float *dst,
                            hipStream_t st) {
    const int ti = p.jw;
    dim3 grid(static_cast<unsigned>((N_in + 256 * p.ipt - 1) / (256 * p.ipt)),
              static_cast<unsigned>((N_out + ti - 1) / ti), static_cast<unsigned>(p.nsplit));
    // G buffers of every group; after the samples, the same LDS carries the
    // groups' sums to group 0 (16 per thread per round)
    const int groups = p.waves / 4;
    const size_t lds = std::max(groups * 2 * static_cast<size_t>(C.M + 4) * dw_stride(ti, groups),
                                static_cast<size_t>(groups - 1) * 16 * 256) *
                       sizeof(float);
    ProfScope prof("dw_dense", st);
    const int nper = dw_nper(C.M, ti);
#define DW_LAUNCH_GI(TIV, NP, GWV, KSV, IPTV)                                                      \
    hipLaunchKernelGGL((dw_dense_kernel<TIV, NP, GWV, KSV, IPTV>), grid, dim3(256 * GWV), lds, st,  \
                       C, static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),     \
                       p.b_per_split, ws.gam, ws.uq, ws.q, ws.row, ws.L, ws.R, dq, dst)
#define DW_LAUNCH_G(TIV, NP, GWV, KSV) DW_LAUNCH_GI(TIV, NP, GWV, KSV, 1)
#define DW_LAUNCH_K(TIV, NP, KSV)                                          \
    do {                                                                   \
        if (groups == 2) DW_LAUNCH_G(TIV, NP, 2, KSV);                     \
        else DW_LAUNCH_G(TIV, NP, 1, KSV);                                 \
    } while (0)
#define DW_LAUNCH(TIV, NP)                                                \
    do {                                                                  \
        if (C.kind == kGeneral) DW_LAUNCH_K(TIV, NP, kGeneral);           \
        else DW_LAUNCH_K(TIV, NP, kAnyKind);                              \
    } while (0)
    if (p.ipt > 1) {
        // one group; 64-neuron tiles, kDwWideIPT inputs per thread
#define DW_WIDE(NP)                                                                  \
    do {                                                                             \
        if (C.kind == kGeneral) DW_LAUNCH_GI(64, NP, 1, kGeneral, kDwWideIPT);       \
        else DW_LAUNCH_GI(64, NP, 1, kAnyKind, kDwWideIPT);                          \
    } while (0)
        if (nper == 9) DW_WIDE(9);
        else if (nper == 17) DW_WIDE(17);
        else DW_WIDE(33);
#undef DW_WIDE
    } else if (ti == 64) {
        if (nper == 9) DW_LAUNCH(64, 9);
        else if (nper == 17) DW_LAUNCH(64, 17);
        else DW_LAUNCH(64, 33);
    } else if (ti == 16) {
        if (nper == 9) DW_LAUNCH(16, 9);
        else if (nper == 17) DW_LAUNCH(16, 17);
        else DW_LAUNCH(16, 33);
    } else {
        if (nper == 9) DW_LAUNCH(32, 9);
        else if (nper == 17) DW_LAUNCH(32, 17);
        else DW_LAUNCH(32, 33);
    }
#undef DW_LAUNCH
#undef DW_LAUNCH_K
#undef DW_LAUNCH_G
#undef DW_LAUNCH_GI
    return hipGetLastError();
}

hipError_t launch_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                           const void *W, bool bf16, const float *t_in, const float *t_out,
                           const float *slope, const int *q_idx, const float *grad_t,
                           DenseBwdWs ws, float *grad_W, float *grad_t_in, const Synfire &sf,
                           hipStream_t st) {
    const bool zero_dt = grad_t_in && B * N_in > 0;
    const bool run_dt = zero_dt && N_out > 0;
    const bool run_dw = grad_W && N_out * N_in > 0;
    // sort (per-input events for dW; row-sorted records with derivatives and
    // a zeroed dt_in when dt_in is wanted), transpose W, gradient triples:
    // one launch
    // the dead-neuron term needs dW; without dW only dT/dt is used
    Synfire sfp = sf;
    if (!run_dw) sfp.dq = nullptr;
    const float *dq = (sfp.on && sfp.dq) ? sfp.dq : nullptr;
    hipError_t e = launch_prep(C, B, N_in, N_out, t_in, ws.srt, ws.n_valid, true,
                               SortOut{ws.row, ws.L, ws.R, zero_dt ? grad_t_in : nullptr}, W, bf16,
                               ws.wt, run_dt,
                               PrepGrad{t_out, slope, grad_t, q_idx, ws.gam, ws.uq, ws.q, sfp,
                                        static_cast<int>(B)},
                               B * N_out, "bwd_prep", st);
    if (e != hipSuccess) return e;
    DwPlan p = plan_dw(B, N_in, N_out, C.M);
    const bool split = run_dw && p.nsplit > 1;
    if (run_dw) {
        e = launch_dw(C, p, B, N_in, N_out, ws, split ? nullptr : dq, split ? ws.part : grad_W, st);
        if (e != hipSuccess) return e;
    }
    const RedJob red{split ? N_out * N_in : 0, p.nsplit, ws.part, grad_W, dq,
                     static_cast<int>(N_in)};
    if (run_dt) {
        const int tiles = static_cast<int>((N_out + kWave - 1) / kWave);
        const int tpw = (tiles + 3) / 4;  // tiles per wave
        const int64_t red_rows = ((red.n + 3) / 4 + kDtRanges * 256 - 1) / (kDtRanges * 256);
        dim3 grid(kDtRanges, static_cast<unsigned>(B + red_rows));
        ProfScope prof("dtin_rows", st);
#define DTR_KV(WTY, NTV, KSV, VECV)                                                              \
    hipLaunchKernelGGL((dtin_rows_kernel<WTY, NTV, KSV, VECV>), grid, dim3(256), 0, st, C,       \
                       static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),     \
                       static_cast<const WTY *>(ws.wt), ws.srt, ws.gam, ws.uq, ws.q, grad_t_in, red)
#define DTR_K(WTY, NTV, KSV)                                   \
    do {                                                       \
        if (N_out % NTV == 0) DTR_KV(WTY, NTV, KSV, true);     \
        else DTR_KV(WTY, NTV, KSV, false);                     \
    } while (0)
#define DTR(WTY, NTV)                                                     \
    do {                                                                  \
        if (C.kind == kGeneral) DTR_K(WTY, NTV, kGeneral);                \
        else DTR_K(WTY, NTV, kAnyKind);                                   \
    } while (0)
#define DTR_NT(WTY)                                      \
    do {                                                 \
        if (tpw <= 1) DTR(WTY, 1);                       \
        else if (tpw <= 2) DTR(WTY, 2);                  \
        else DTR(WTY, 4);                                \
    } while (0)
        if (tiles == 1) {
            // one tile: the waves split the records instead of the tiles
            const size_t lds = static_cast<size_t>(C.M + 4) * kWave * sizeof(float);  // R + 1 rows
#define DTT_K(WTY, KSV)                                                                            \
    hipLaunchKernelGGL((dtin_tile_kernel<WTY, KSV>), grid, dim3(256), lds, st, C,                  \
                       static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),       \
                       static_cast<const WTY *>(ws.wt), ws.srt, ws.gam, ws.uq, ws.q, grad_t_in, red)
#define DTT(WTY)                                                          \
    do {                                                                  \
        if (C.kind == kGeneral) DTT_K(WTY, kGeneral);                     \
        else DTT_K(WTY, kAnyKind);                                        \
    } while (0)
            if (bf16) DTT(uint16_t);
            else DTT(float);
#undef DTT
#undef DTT_K
        } else if (bf16) {
            DTR_NT(uint16_t);
        } else {
            DTR_NT(float);
        }
#undef DTR_NT
#undef DTR
#undef DTR_K
#undef DTR_KV
        return hipGetLastError();
    }
    if (split) {
        ProfScope prof("dw_reduce", st);
        hipLaunchKernelGGL(reduce_splits_kernel, dim3(static_cast<unsigned>(((red.n + 3) / 4 + 255) / 256)),
                           dim3(256), 0, st, red.n, p.nsplit, ws.part, dq,
                           static_cast<int>(N_in), grad_W);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_softmax_ce(int64_t B, int64_t N, const float *t, const int *labels,
                             float tau_soft, float t_cap, float *grad, float *loss,
                             hipStream_t st) {
    ProfScope prof("softmax_ce", st);
    if (B > 0)
        hipLaunchKernelGGL(softmax_ce_kernel, dim3(static_cast<unsigned>(B)), dim3(kLossThreads), 0,
                           st, static_cast<int>(B), static_cast<int>(N), t, labels, tau_soft,
                           t_cap, grad, loss);
    hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(kLossThreads), 0, st, static_cast<int>(B),
                       loss);
    return hipGetLastError();
}

hipError_t launch_mse(int64_t B, int64_t N, const float *t, const float *y, float *grad,
                      float *loss, hipStream_t st) {
    ProfScope prof("mse", st);
    if (B > 0)
        hipLaunchKernelGGL(mse_kernel, dim3(static_cast<unsigned>(B)), dim3(kLossThreads), 0, st,
                           static_cast<int>(B), static_cast<int>(N), t, y, grad, loss);
    hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(kLossThreads), 0, st, static_cast<int>(B),
                       loss);
    return hipGetLastError();
}

}  // namespace dstd
