// dstd_exact.hip -- exact continuous-time LIF spike times of a dense layer and
// their gradients (App. A, Alg. 1, Eq. (timing_exact)) on gfx950: the method
// DSTD replaces, kept as the baseline it is measured against.
//
// Forward: one block per sample sorts its finite inputs (bitonic sort of
// (time, index) keys in LDS) and writes per-interval records; then one lane
// per neuron walks the sorted inputs, carrying (v, I) in fp64 from one input
// time to the next, and tests each interval [t~_k, t~_{k+1}) for the first
// crossing with the same interval test and root solve as the DSTD scan (the
// DSTD intervals are the special case of a fixed length). The weight of
// input j for the wave's 64 neurons is row j of the transposed weights: one
// coalesced load per input, with the row offset as a scalar.
// Backward: implicit-function theorem on v(t) = V_th over the causal set of
// the crossing interval (inputs with t_j <= t~_k):
//   dL/dw_ij = gamma_i K(t_i - t_j),  dL/dt_j = -sum_i gamma_i w_ij K'(t_i - t_j)
// with gamma = -g / slope; one kernel per gradient, each pair term evaluated
// directly (the indicator t_j <= t~_k makes the sums non-separable).
#include <algorithm>

#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"

namespace dstd {

namespace {

constexpr int kSortThreads = 1024;
constexpr int kFwdThreads = 4 * kWave;
constexpr int kChunk = 32;      // records per batch of weight and constant loads
constexpr int kGradWaves = 4;   // waves splitting the summed dimension (LDS reduction)
constexpr int kDwTile = 16;     // neurons per dW block (accumulators per lane)
constexpr int kDtSamples = 4;   // samples per dt_in block (accumulators per lane)
constexpr uint64_t kNoKey = ~0ull;

// order-preserving map of a float to an unsigned key (and back)
__device__ __forceinline__ uint32_t time_key(float t) {
    const uint32_t u = __float_as_uint(t);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_time(uint64_t k) {
    const uint32_t h = static_cast<uint32_t>(k >> 32);
    return __uint_as_float((h & 0x80000000u) ? (h & 0x7fffffffu) : ~h);
}

// Sorts sample b's inputs that are finite and before t_max by (time, index)
// into key[0, n) (the rest hold kNoKey); P = power of two >= N_in (and >= 1).
// Returns n, the same in every thread. Ends with a barrier.
__device__ int sort_sample_keys(int b, int N_in, int P, const float *__restrict__ t_in,
                                float t_max, uint64_t *key) {
    const int tid = threadIdx.x;
    for (int x = tid; x < P; x += kSortThreads) {
        uint64_t k = kNoKey;
        if (x < N_in) {
            const float t = t_in[static_cast<int64_t>(b) * N_in + x];
            if (isfinite(t) && t < t_max)
                k = (static_cast<uint64_t>(time_key(t)) << 32) | static_cast<uint32_t>(x);
        }
        key[x] = k;
    }
    __syncthreads();
    // bitonic sort: pair (lo, lo + stride) of each merge stage, ascending
    // where the enclosing block of `size` is ascending
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int x = tid; x < (P >> 1); x += kSortThreads) {
                const int lo = 2 * x - (x & (stride - 1));
                const int hi = lo + stride;
                const bool asc = (lo & size) == 0;
                const uint64_t a = key[lo], c = key[hi];
                if ((a > c) == asc) {
                    key[lo] = c;
                    key[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    // n = first position holding kNoKey (binary search, same in every thread)
    int lo = 0, hi = P;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (key[mid] == kNoKey) hi = mid; else lo = mid + 1;
    }
    return lo;
}

__device__ __forceinline__ int pow2_at_least(int n) {
    int p = 1;
    while (p < n) p <<= 1;
    return p;
}

// K(u) in fp64, u >= 0 (Table "tab:kernel"; u may be +inf)
__device__ __forceinline__ double kern_dd(int kind, double tv, double ti, double u) {
    switch (kind) {
        case kEqual: return u * exp(-u / ti);
        case kInfTau: return -ti * expm1(-u / ti);
        case kInfInf: return u;
        default: {
            const double c = tv * ti / (tv - ti), kap = 1.0 / ti - 1.0 / tv;
            return -c * exp(-u / tv) * expm1(-kap * u);
        }
    }
}

// Blocks [0, B) sort one sample each and write its records; blocks after
// that transpose one 32 x 32 weight tile each (W -> WT [N_in][N_out]).
template <typename WT>
__global__ __launch_bounds__(kSortThreads) void exact_prep_kernel(LifConst C, int B, int N_in,
                                                                   int N_out, float t_max,
                                                                   const float *__restrict__ t_in,
                                                                   const WT *__restrict__ W,
                                                                   WT *__restrict__ Wt,
                                                                   ExactRecs rec) {
    extern __shared__ uint64_t key[];
    const int blk = blockIdx.x;
    if (blk >= B) {
        transpose_tile<WT, kSortThreads>(N_out, N_in, W, Wt, blk - B,
                                         reinterpret_cast<WT(*)[33]>(key));
        return;
    }
    const int b = blk;
    const int n = sort_sample_keys(b, N_in, pow2_at_least(N_in), t_in, t_max, key);
    const double tv = static_cast<double>(C.tv), ti = static_cast<double>(C.ti);
    const double inv_tv = 1.0 / tv, inv_ti = 1.0 / ti;  // 0 for +inf
    const double kap = (C.kind == kGeneral) ? inv_ti - inv_tv : 0.0;
    // K peaks at ln(tv/ti)/kappa (general), tau ((tau, tau)); the other rows increase
    const double upk = (C.kind == kGeneral) ? log(tv / ti) / kap
                       : (C.kind == kEqual) ? ti : INFINITY;
    const int64_t o = static_cast<int64_t>(b) * rec.stride;
    for (int k = threadIdx.x; k < n; k += kSortThreads) {
        const uint64_t kk = key[k];
        const float t = key_time(kk);
        const bool last = (k + 1 == n);
        // the last interval ends at t_max; the others at the next input
        const double len = (last ? static_cast<double>(t_max) : static_cast<double>(key_time(key[k + 1]))) -
                           static_cast<double>(t);
        rec.j[o + k] = static_cast<int>(kk & 0xffffffffu);
        rec.t[o + k] = t;
        rec.len[o + k] = static_cast<float>(len);
        rec.r_lo[o + k] = (C.kind == kGeneral) ? static_cast<float>(exp(-kap * len)) : 0.f;
        rec.alpha[o + k] = last ? 0.0 : exp(-len * inv_tv);
        rec.beta[o + k] = last ? 0.0 : exp(-len * inv_ti);
        rec.kl[o + k] = last ? 0.0 : kern_dd(C.kind, tv, ti, len);
        // rounded up: a bound for the interval filter
        rec.kmax[o + k] = __double2float_ru(kern_dd(C.kind, tv, ti, fmin(len, upk)));
    }
    if (threadIdx.x == 0) rec.n[b] = n;
}

// One lane per neuron of sample blockIdx.y: walk the sample's records in
// time order. At input k the current jumps by w_ik; the interval [t~_k,
// t~_k + len) is tested (zero-length intervals of simultaneous inputs are
// skipped: they add up first); the state is then carried to the next input
// with that interval's fp64 decays. Records come in batches of kChunk (fully
// unrolled); the weights and the interval constants of the next batch are
// loaded during this one. A lane stops testing at its first crossing and the
// wave stops once all its lanes have; the roots are then solved together.
// The last partial batch is walked one record at a time.
template <typename WT, int KS>
__global__ __launch_bounds__(kFwdThreads) void exact_fwd_kernel(LifConst C, int N_in, int N_out,
                                                                const WT *__restrict__ Wt,
                                                                ExactRecs rec,
                                                                float *__restrict__ t_out,
                                                                float *__restrict__ slope,
                                                                int *__restrict__ k_idx) {
    const int b = blockIdx.y;
    const int i = blockIdx.x * kFwdThreads + threadIdx.x;
    const bool act = i < N_out;
    const int n = *as_const(rec.n + b);
    const int64_t o = static_cast<int64_t>(b) * rec.stride;
    const int *rj = rec.j + o;
    const float *rlen = rec.len + o, *rrl = rec.r_lo + o, *rm = rec.kmax + o;
    const double *ra = rec.alpha + o, *rb = rec.beta + o, *rk = rec.kl + o;
    const __amdgpu_buffer_rsrc_t wr =
        make_rsrc(Wt, static_cast<uint32_t>(static_cast<int64_t>(N_in) * N_out * sizeof(WT)));
    const int voff = (act ? i : 0) * static_cast<int>(sizeof(WT));
    const int rstride = N_out * static_cast<int>(sizeof(WT));
    auto wrow = [&](int k) { return as_const(rj)[k] * rstride; };  // k < n: j in [0, N_in)

    double Vd = 0.0, Id = 0.0;
    bool done = !act;
    int kf = -1;
    Seg sf{0.f, 0.f};
    float hi = 0.f, fhi = 0.f;
    const double itv = static_cast<double>(C.inv_tv);
    // one record: the jump of the current, the state carried over the
    // interval, and the interval test where the filter lets it through
    auto step = [&](int k, float wk, double al, double be, double kl, float kmax) {
        Id = Id + static_cast<double>(wk);
        const double vn = fma(Vd, al, Id * kl);
        const double km = static_cast<double>(kmax);
        const double vpos = fmax(Vd, 0.0);
        const double ub = (kind_of<KS>(C) == kInfInf) ? ((Id > 0.0) ? fma(Id, km, vpos) : vpos)
                                                      : fma(fmax(Id, 0.0), km, vpos);
        // bitwise: the bound is formed on every step, not behind a branch on
        // `done`
        if ((ub >= C.theta_lo_d) & !done) {
            // Inside an interval v has at most one critical point, so a
            // crossing needs v near the threshold at an end of the interval
            // or an interior maximum: v rising at the start and falling at
            // the end (v' = -v/tv + I(u), I(u) = I e^{-u/ti}). The last
            // interval's end value is not carried by the recurrence: always
            // tested. Only these lanes run the full test.
            const bool last = k + 1 == n;
            const bool maybe = last || vn >= C.theta_lo_d || Vd >= C.theta_lo_d ||
                               (fma(-Vd, itv, Id) > 0.0 && fma(-vn, itv, Id * be) < 0.0);
            const float len = as_const(rlen)[k];
            if (maybe && len > 0.f &&
                seg_test<KS>(C, Vd, Id, vn, last, len, km, as_const(rrl)[k], sf, hi, fhi)) {
                done = true;
                kf = k;
            }
        }
        Vd = vn;
        Id = Id * be;
    };
    // Per batch, lane u < kChunk holds record u's constants (vector loads
    // issued with the batch's weights, one batch ahead); each step reads them
    // back as scalars with readlane.
    static_assert(kChunk <= kWave, "one record's constants per lane");
    const int lane = threadIdx.x & (kWave - 1);
    const int ul = lane < kChunk ? lane : 0;
    float w[kChunk], wn[kChunk];
    double ca = 0.0, cb = 0.0, ck = 0.0, na = 0.0, nb = 0.0, nk = 0.0;
    float cm = 0.f, nm = 0.f;
    auto load_consts = [&](int kb) {
        na = ra[kb + ul];
        nb = rb[kb + ul];
        nk = rk[kb + ul];
        nm = rm[kb + ul];
    };
    auto lane_d = [](double v, int u) {
        const int lo = __builtin_amdgcn_readlane(__double2loint(v), u);
        const int hi = __builtin_amdgcn_readlane(__double2hiint(v), u);
        return __hiloint2double(hi, lo);
    };
    if (n >= kChunk) {
#pragma unroll
        for (int u = 0; u < kChunk; ++u) wn[u] = BufLoad<WT>::get(wr, voff, wrow(u));
        load_consts(0);
    }
    int k0 = 0;
    for (; k0 + kChunk <= n; k0 += kChunk) {
        if (__all(done)) break;
#pragma unroll
        for (int u = 0; u < kChunk; ++u) w[u] = wn[u];
        ca = na; cb = nb; ck = nk; cm = nm;
        if (k0 + 2 * kChunk <= n) {
#pragma unroll
            for (int u = 0; u < kChunk; ++u) wn[u] = BufLoad<WT>::get(wr, voff, wrow(k0 + kChunk + u));
            load_consts(k0 + kChunk);
        }
#pragma unroll
        for (int u = 0; u < kChunk; ++u)
            step(k0 + u, w[u], lane_d(ca, u), lane_d(cb, u), lane_d(ck, u),
                 __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cm), u)));
    }
    if (!__all(done))
        for (int k = k0; k < n; ++k)
            step(k, BufLoad<WT>::get(wr, voff, wrow(k)), as_const(ra)[k], as_const(rb)[k],
                 as_const(rk)[k], as_const(rm)[k]);
    if (!act) return;
    float to = INFINITY, sl = 0.f;
    if (kf >= 0) {
        float u;
        seg_solve<KS>(C, sf, hi, fhi, u, sl);
        to = static_cast<float>(static_cast<double>(rec.t[o + kf]) + static_cast<double>(u));
    }
    const int64_t oo = static_cast<int64_t>(b) * N_out + i;
    t_out[oo] = to;
    slope[oo] = sl;
    k_idx[oo] = kf;
}

// One block per sample: sort as in the forward (the same order), then the
// gradient data of each of the sample's neurons: gamma = -g / slope (slope
// floored), the spike time, and the time of the crossing interval's left end
// (the causal set is t_j <= that time); zero where no gradient flows.
__global__ __launch_bounds__(kSortThreads) void exact_bwd_prep_kernel(
    LifConst C, int B, int N_in, int N_out, float t_max, const float *__restrict__ t_in,
    const float *__restrict__ t_out, const float *__restrict__ slope,
    const int *__restrict__ k_idx, const float *__restrict__ grad_t, float4 *__restrict__ P,
    float4 *__restrict__ PT) {
    extern __shared__ uint64_t key[];
    const int b = blockIdx.x;
    const int n = sort_sample_keys(b, N_in, pow2_at_least(N_in), t_in, t_max, key);
    for (int i = threadIdx.x; i < N_out; i += kSortThreads) {
        const int64_t o = static_cast<int64_t>(b) * N_out + i;
        const int k = k_idx[o];
        const float g = grad_t[o], to = t_out[o];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (k >= 0 && k < n && g != 0.f && isfinite(to))
            v = make_float4(-g / fmaxf(slope[o], C.slope_floor), to, key_time(key[k]), 0.f);
        P[o] = v;
        PT[static_cast<int64_t>(i) * B + b] = v;
    }
}

// K(d) and K'(d), d >= 0, from the hardware exponential (relative error
// ~1e-6, within the gradients' tolerance)
template <int KS>
__device__ __forceinline__ void kern_pair(const LifConst &C, float d, float &K, float &Kp) {
    switch (kind_of<KS>(C)) {
        case kInfInf: K = d; Kp = 1.f; return;
        case kInfTau: {
            const float ei = __expf(-d * C.inv_ti);
            K = C.ti * (1.f - ei);
            Kp = ei;
            return;
        }
        case kEqual: {
            const float ei = __expf(-d * C.inv_ti);
            K = d * ei;
            Kp = ei * fmaf(-d, C.inv_ti, 1.f);
            return;
        }
        default: {
            const float ev = __expf(-d * C.inv_tv), ei = __expf(-d * C.inv_ti);
            K = C.c * (ev - ei);
            Kp = C.c * fmaf(ei, C.inv_ti, -ev * C.inv_tv);
            return;
        }
    }
}

// grad_W[i][j] = sum_b gamma_bi K(t_bi - t_bj) over t_bj <= tl_bi. Block:
// kDwTile neurons (blockIdx.x) x 64 inputs (blockIdx.y, lane = input); its
// kGradWaves waves take every kGradWaves-th sample and their partial sums
// meet in LDS. The per-neuron data of a sample is read as scalars.
template <int KS>
__global__ __launch_bounds__(kGradWaves * kWave) void exact_dw_kernel(LifConst C, int B, int N_in,
                                                                      int N_out,
                                                                      const float *__restrict__ t_in,
                                                                      const float4 *__restrict__ P,
                                                                      float *__restrict__ grad_W) {
    __shared__ float red[kGradWaves][kDwTile][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int j0 = blockIdx.y * kWave;
    const int j = j0 + lane;
    const int i0 = blockIdx.x * kDwTile;
    const int ni = min(kDwTile, N_out - i0);
    const bool ok = j < N_in;
    float acc[kDwTile];
#pragma unroll
    for (int ii = 0; ii < kDwTile; ++ii) acc[ii] = 0.f;
    for (int b = wave; b < B; b += kGradWaves) {
        float t = ok ? t_in[static_cast<int64_t>(b) * N_in + j] : INFINITY;
        if (!isfinite(t)) t = INFINITY;
        const float *pb = reinterpret_cast<const float *>(P + static_cast<int64_t>(b) * N_out + i0);
#pragma unroll
        for (int ii = 0; ii < kDwTile; ++ii) {
            if (ii < ni) {
                const float gam = as_const(pb)[4 * ii];
                const float th = as_const(pb)[4 * ii + 1], tl = as_const(pb)[4 * ii + 2];
                if (gam != 0.f && t <= tl) {
                    float K, Kp;
                    kern_pair<KS>(C, th - t, K, Kp);
                    acc[ii] = fmaf(gam, K, acc[ii]);
                }
            }
        }
    }
#pragma unroll
    for (int ii = 0; ii < kDwTile; ++ii) red[wave][ii][lane] = acc[ii];
    __syncthreads();
    for (int r = threadIdx.x; r < kDwTile * kWave; r += kGradWaves * kWave) {
        const int ii = r / kWave, l = r % kWave;
        if (ii < ni && j0 + l < N_in) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < kGradWaves; ++w) sum += red[w][ii][l];
            grad_W[static_cast<int64_t>(i0 + ii) * N_in + j0 + l] = sum;
        }
    }
}

// grad_t_in[b][j] = -sum_i gamma_bi w_ij K'(t_bi - t_bj) over t_bj <= tl_bi.
// Block: 64 inputs (blockIdx.x, lane = input) x kDtSamples samples
// (blockIdx.y); its kGradWaves waves take every kGradWaves-th neuron (row i
// of W is one coalesced load) and their partial sums meet in LDS.
template <typename WT, int KS>
__global__ __launch_bounds__(kGradWaves * kWave) void exact_dtin_kernel(
    LifConst C, int B, int N_in, int N_out, const WT *__restrict__ W, const float *__restrict__ t_in,
    const float4 *__restrict__ PT, float *__restrict__ grad_t_in) {
    __shared__ float red[kGradWaves][kDtSamples][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = uniform(threadIdx.x >> 6);
    const int j0 = blockIdx.x * kWave;
    const int j = j0 + lane;
    const int b0 = blockIdx.y * kDtSamples;
    const int nb = min(kDtSamples, B - b0);
    const bool ok = j < N_in;
    float t[kDtSamples], acc[kDtSamples];
#pragma unroll
    for (int bb = 0; bb < kDtSamples; ++bb) {
        float x = (ok && bb < nb) ? t_in[static_cast<int64_t>(b0 + bb) * N_in + j] : INFINITY;
        t[bb] = isfinite(x) ? x : INFINITY;
        acc[bb] = 0.f;
    }
#pragma unroll 2
    for (int i = wave; i < N_out; i += kGradWaves) {
        const float w = ok ? WLoad<WT>::get(W, static_cast<int64_t>(i) * N_in + j) : 0.f;
        const float *pi = reinterpret_cast<const float *>(PT + static_cast<int64_t>(i) * B + b0);
#pragma unroll
        for (int bb = 0; bb < kDtSamples; ++bb) {
            if (bb < nb) {
                const float gam = as_const(pi)[4 * bb];
                const float th = as_const(pi)[4 * bb + 1], tl = as_const(pi)[4 * bb + 2];
                if (gam != 0.f && t[bb] <= tl) {
                    float K, Kp;
                    kern_pair<KS>(C, th - t[bb], K, Kp);
                    acc[bb] = fmaf(-gam * w, Kp, acc[bb]);
                }
            }
        }
    }
#pragma unroll
    for (int bb = 0; bb < kDtSamples; ++bb) red[wave][bb][lane] = acc[bb];
    __syncthreads();
    for (int r = threadIdx.x; r < kDtSamples * kWave; r += kGradWaves * kWave) {
        const int bb = r / kWave, l = r % kWave;
        if (bb < nb && j0 + l < N_in) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < kGradWaves; ++w) sum += red[w][bb][l];
            grad_t_in[static_cast<int64_t>(b0 + bb) * N_in + j0 + l] = sum;
        }
    }
}

size_t sort_lds(int64_t N_in) {
    int64_t p = 1;
    while (p < N_in) p <<= 1;
    return static_cast<size_t>(p) * sizeof(uint64_t);
}

unsigned cdiv(int64_t a, int64_t b) { return static_cast<unsigned>((a + b - 1) / b); }

}  // namespace

hipError_t launch_exact_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                                const void *W, bool bf16, void *Wt, ExactRecs rec,
                                const float *t_in, float t_max, float *t_out, float *slope,
                                int *k_idx, hipStream_t st) {
    const int64_t n_tr = (N_in * N_out > 0) ? static_cast<int64_t>(cdiv(N_in, 32)) * cdiv(N_out, 32) : 0;
    const size_t lds = std::max(sort_lds(N_in), static_cast<size_t>(32 * 33 * sizeof(float)));
    {
        ProfScope prof("exact_sort_transpose", st);
        if (bf16)
            hipLaunchKernelGGL(exact_prep_kernel<uint16_t>, dim3(static_cast<unsigned>(B + n_tr)),
                               dim3(kSortThreads), lds, st, C, static_cast<int>(B),
                               static_cast<int>(N_in), static_cast<int>(N_out), t_max, t_in,
                               static_cast<const uint16_t *>(W), static_cast<uint16_t *>(Wt), rec);
        else
            hipLaunchKernelGGL(exact_prep_kernel<float>, dim3(static_cast<unsigned>(B + n_tr)),
                               dim3(kSortThreads), lds, st, C, static_cast<int>(B),
                               static_cast<int>(N_in), static_cast<int>(N_out), t_max, t_in,
                               static_cast<const float *>(W), static_cast<float *>(Wt), rec);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    ProfScope prof("exact_fwd", st);
    dim3 grid(cdiv(N_out, kFwdThreads), static_cast<unsigned>(B));
#define EXF(WTY, KSV)                                                                           \
    hipLaunchKernelGGL((exact_fwd_kernel<WTY, KSV>), grid, dim3(kFwdThreads), 0, st, C,         \
                       static_cast<int>(N_in), static_cast<int>(N_out),                          \
                       static_cast<const WTY *>(Wt), rec, t_out, slope, k_idx)
    const bool gen = C.kind == kGeneral;
    if (bf16) {
        if (gen) EXF(uint16_t, kGeneral); else EXF(uint16_t, kAnyKind);
    } else {
        if (gen) EXF(float, kGeneral); else EXF(float, kAnyKind);
    }
#undef EXF
    return hipGetLastError();
}

hipError_t launch_exact_backward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                                 const void *W, bool bf16, const float *t_in, float t_max,
                                 const float *t_out, const float *slope, const int *k_idx,
                                 const float *grad_t, float4 *P, float4 *PT, float *grad_W,
                                 float *grad_t_in, hipStream_t st) {
    const bool gen = C.kind == kGeneral;
    if (B * N_out > 0) {
        ProfScope prof("exact_bwd_prep", st);
        hipLaunchKernelGGL(exact_bwd_prep_kernel, dim3(static_cast<unsigned>(B)), dim3(kSortThreads),
                           sort_lds(N_in), st, C, static_cast<int>(B), static_cast<int>(N_in),
                           static_cast<int>(N_out), t_max, t_in, t_out, slope, k_idx, grad_t, P, PT);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (grad_W && N_in * N_out > 0) {
        ProfScope prof("exact_dw", st);
        dim3 grid(cdiv(N_out, kDwTile), cdiv(N_in, kWave));
        if (gen)
            hipLaunchKernelGGL(exact_dw_kernel<kGeneral>, grid, dim3(kGradWaves * kWave), 0, st, C,
                               static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),
                               t_in, P, grad_W);
        else
            hipLaunchKernelGGL(exact_dw_kernel<kAnyKind>, grid, dim3(kGradWaves * kWave), 0, st, C,
                               static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),
                               t_in, P, grad_W);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (grad_t_in && B * N_in > 0) {
        ProfScope prof("exact_dtin", st);
        dim3 grid(cdiv(N_in, kWave), cdiv(B, kDtSamples));
#define EXD(WTY, KSV)                                                                            \
    hipLaunchKernelGGL((exact_dtin_kernel<WTY, KSV>), grid, dim3(kGradWaves * kWave), 0, st, C,  \
                       static_cast<int>(B), static_cast<int>(N_in), static_cast<int>(N_out),      \
                       static_cast<const WTY *>(W), t_in, PT, grad_t_in)
        if (bf16) {
            if (gen) EXD(uint16_t, kGeneral); else EXD(uint16_t, kAnyKind);
        } else {
            if (gen) EXD(float, kGeneral); else EXD(float, kAnyKind);
        }
#undef EXD
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace dstd
