// dstd_synfire.hip -- values of the synfire-chain training terms (App. C.1,
// Eqs. (temporal_penalty), (dead_neuron_penalty)) for gfx950.
//
// The gradients of both terms are fused into the backward kernels (the
// temporal penalty's dT/dt into the per-neuron gradient, the dead-neuron term
// into the dW write); these kernels only report the two values. Every sum has
// a fixed order: per-thread strided partials, then an LDS tree per block,
// then one block adding the block results in index order.
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"

namespace dstd {

namespace {

constexpr int kValThreads = 256;
constexpr int64_t kValChunk = 8192;  // outputs per temporal-penalty block

__device__ float block_sum(float v, float *sh) {
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int h = kValThreads / 2; h > 0; h >>= 1) {
        if (static_cast<int>(threadIdx.x) < h) sh[threadIdx.x] += sh[threadIdx.x + h];
        __syncthreads();
    }
    const float r = sh[0];
    __syncthreads();
    return r;
}

// blocks [0, rows): row i's (silent outputs) * (weight row sum);
// blocks [rows, rows + n_tb): the temporal penalty of kValChunk outputs
// (without the scale). Results go to part[block].
template <typename WT>
__global__ __launch_bounds__(kValThreads) void synfire_value_kernel(
    Synfire sf, int64_t B, int64_t rows, int64_t spatial, int64_t row_len,
    const float *__restrict__ t, const WT *__restrict__ W, float *__restrict__ part) {
    __shared__ float sh[kValThreads];
    const int64_t blk = blockIdx.x;
    if (blk < rows) {
        const int64_t i = blk;
        const int64_t n = B * spatial;
        float cnt = 0.f;  // counts below 2^24 stay exact in fp32
        for (int64_t e = threadIdx.x; e < n; e += kValThreads) {
            const int64_t b = e / spatial, p = e % spatial;
            cnt += isfinite(t[(b * rows + i) * spatial + p]) ? 0.f : 1.f;
        }
        float ws = 0.f;
        for (int64_t j = threadIdx.x; j < row_len; j += kValThreads)
            ws += WLoad<WT>::get(W, i * row_len + j);
        const float c = block_sum(cnt, sh);
        const float w = block_sum(ws, sh);
        if (threadIdx.x == 0) part[blk] = c * w;
        return;
    }
    const int64_t n = B * rows * spatial;
    const int64_t lo = (blk - rows) * kValChunk;
    const int64_t hi = min(n, lo + kValChunk);
    float acc = 0.f;
    for (int64_t e = lo + threadIdx.x; e < hi; e += kValThreads) {
        const float v = t[e];
        if (!isfinite(v)) continue;
        if (v < sf.th) acc += sf.gh * (v - sf.th) * (v - sf.th);
        else if (v > sf.tt) acc += sf.gt * (v - sf.tt) * (v - sf.tt);
    }
    const float s = block_sum(acc, sh);
    if (threadIdx.x == 0) part[blk] = s;
}

// value[0] = scale * (sum of the temporal blocks), value[1] = -gamma_q *
// scale * (sum of the row blocks)
__global__ __launch_bounds__(kValThreads) void synfire_final_kernel(Synfire sf, int64_t rows,
                                                                     int64_t n_tb,
                                                                     const float *__restrict__ part,
                                                                     float *__restrict__ value) {
    __shared__ float sh[kValThreads];
    float q = 0.f, tp = 0.f;
    for (int64_t k = threadIdx.x; k < rows; k += kValThreads) q += part[k];
    for (int64_t k = threadIdx.x; k < n_tb; k += kValThreads) tp += part[rows + k];
    const float qs = block_sum(q, sh);
    const float ts = block_sum(tp, sh);
    if (threadIdx.x == 0) {
        value[0] = sf.scale * ts;
        value[1] = -(sf.gq * sf.scale * qs);
    }
}

}  // namespace

int synfire_value_blocks(int64_t n) { return static_cast<int>((n + kValChunk - 1) / kValChunk); }

hipError_t launch_synfire_value(const Synfire &sf, int64_t B, int64_t rows, int64_t spatial,
                                int64_t row_len, const float *t_out, const void *W, bool bf16,
                                float *ws, float *value, hipStream_t st) {
    const int64_t n_tb = synfire_value_blocks(B * rows * spatial);
    ProfScope prof("synfire_value", st);
    const unsigned blocks = static_cast<unsigned>(rows + n_tb);
    if (blocks > 0) {
        if (bf16)
            hipLaunchKernelGGL(synfire_value_kernel<uint16_t>, dim3(blocks), dim3(kValThreads), 0, st,
                               sf, B, rows, spatial, row_len, t_out,
                               static_cast<const uint16_t *>(W), ws);
        else
            hipLaunchKernelGGL(synfire_value_kernel<float>, dim3(blocks), dim3(kValThreads), 0, st,
                               sf, B, rows, spatial, row_len, t_out,
                               static_cast<const float *>(W), ws);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(synfire_final_kernel, dim3(1), dim3(kValThreads), 0, st, sf, rows, n_tb, ws,
                       value);
    return hipGetLastError();
}

}  // namespace dstd
