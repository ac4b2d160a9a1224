// dstd_skip.hip -- the skip-and-delay connection of an SD block (App. C.3,
// Fig. "skip_connection"): the third layer of the block reads the spikes that
// enter the block, delayed by a fixed 2 tau_shift, alongside the second
// layer's spikes, as one channel-concatenated input map. The delay only
// shifts times, so the backward pass routes the gradient of each channel
// back unchanged. Both directions are elementwise (grid-stride loops over the
// concatenated map) and bound by HBM.
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"

namespace dstd {

namespace {

constexpr int kSkipThreads = 256;

// out[b][c][p] = c < C1 ? t1[b][c][p] + delay : t2[b][c - C1][p]; index over
// the output, n1 = C1 * HW and n2 = C2 * HW floats per sample
__global__ __launch_bounds__(kSkipThreads) void skip_concat_kernel(int64_t n, int64_t n1, int64_t n2,
                                                                   const float *__restrict__ t1,
                                                                   float delay,
                                                                   const float *__restrict__ t2,
                                                                   float *__restrict__ out) {
    const int64_t per = n1 + n2;
    for (int64_t x = static_cast<int64_t>(blockIdx.x) * kSkipThreads + threadIdx.x; x < n;
         x += static_cast<int64_t>(gridDim.x) * kSkipThreads) {
        const int64_t b = x / per, r = x - b * per;
        out[x] = (r < n1) ? t1[b * n1 + r] + delay : t2[b * n2 + (r - n1)];
    }
}

// g1[b][c][p] (+)= g[b][c][p] for c < C1; g2[b][c - C1][p] = g[b][c][p]
// otherwise (either target may be absent)
__global__ __launch_bounds__(kSkipThreads) void skip_split_kernel(int64_t n, int64_t n1, int64_t n2,
                                                                  const float *__restrict__ g,
                                                                  float *__restrict__ g1, int acc,
                                                                  float *__restrict__ g2) {
    const int64_t per = n1 + n2;
    for (int64_t x = static_cast<int64_t>(blockIdx.x) * kSkipThreads + threadIdx.x; x < n;
         x += static_cast<int64_t>(gridDim.x) * kSkipThreads) {
        const int64_t b = x / per, r = x - b * per;
        const float v = g[x];
        if (r < n1) {
            if (g1) {
                const int64_t o = b * n1 + r;
                g1[o] = acc ? g1[o] + v : v;
            }
        } else if (g2) {
            g2[b * n2 + (r - n1)] = v;
        }
    }
}

unsigned skip_blocks(int64_t n) {
    // enough blocks to fill the chip a few times over; the loops stride
    const int64_t want = (n + kSkipThreads - 1) / kSkipThreads;
    return static_cast<unsigned>(want < 8192 ? want : 8192);
}

}  // namespace

hipError_t launch_skip_concat(int64_t B, int64_t n1, int64_t n2, const float *t1, float delay,
                              const float *t2, float *out, hipStream_t st) {
    const int64_t n = B * (n1 + n2);
    if (n == 0) return hipSuccess;
    ProfScope prof("skip_concat", st);
    hipLaunchKernelGGL(skip_concat_kernel, dim3(skip_blocks(n)), dim3(kSkipThreads), 0, st, n, n1,
                       n2, t1, delay, t2, out);
    return hipGetLastError();
}

hipError_t launch_skip_split(int64_t B, int64_t n1, int64_t n2, const float *g, float *g1, int acc,
                             float *g2, hipStream_t st) {
    const int64_t n = B * (n1 + n2);
    if (n == 0 || (!g1 && !g2)) return hipSuccess;
    ProfScope prof("skip_split", st);
    hipLaunchKernelGGL(skip_split_kernel, dim3(skip_blocks(n)), dim3(kSkipThreads), 0, st, n, n1,
                       n2, g, g1, acc, g2);
    return hipGetLastError();
}

}  // namespace dstd
