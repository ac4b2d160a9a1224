// dstd_mfma.hip -- the dense form of the weighted-event contraction on the
// matrix cores of gfx950, for dense layers with bf16 weights.
//
// The weighted events w^_im = sum_j w_ij s_jm of App. B.1 are, over a batch,
// the product w^[(b, m), i] = sum_j S[(b, m), j] W[i, j] with S the event
// matrix [B (M+1)][N_in]: at most two nonzeros per (b, j) column pair, so the
// dense product does (M+1)/2 times the method's multiply-adds (App. B.3). It
// pays only for small M; the library selects it by shape (see the launcher).
//
// Precision: W is exact in bf16. Each event weight s (fp32) is split into
// three bf16 planes s = s1 + s2 + s3 (s1 = bf16(s), s2 = bf16(s - s1),
// s3 = bf16(s - s1 - s2); the residual is below 2^-26 |s|), and the three
// products S_p W^T accumulate in fp32 in the same MFMA accumulators, so w^
// carries the rounding of an fp32 sum, as the event-sparse path does.
//
// Kernels:
//  - mfma_events_kernel: per (b, j) the event row q+1 of bin_event and the
//    three planes of L and R, packed in 16 bytes;
//  - mfma_contract_kernel: 128 x 128 tiles of w^ (rows (b, m), columns i),
//    K tiles of 32 inputs staged in LDS in MFMA fragment order: an S tile is
//    zeroed and each event of the tile's samples writes its two nonzero rows
//    (L at row (b, q), R at row (b, q + 1)) in the three planes; W tiles are
//    copied as 16-byte runs; each of the four waves owns a 64 x 64 quarter
//    (2 x 2 v_mfma_f32_32x32x16_bf16 tiles per plane);
//  - mfma_scan_kernel: one thread per (b, i) runs the interval scan and root
//    solve of the event-sparse forward over w^[(b, 0..M), i].
#include "dstd_internal.h"
#include "dstd_kernels.h"
#include "dstd_profile.h"

namespace dstd {

typedef __bf16 bf16x8_t __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16_t __attribute__((__vector_size__(16 * sizeof(float))));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// round-to-nearest-even fp32 -> bf16 bits (finite inputs)
__device__ __forceinline__ uint32_t bf16_bits(float x) {
    const uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// three bf16 planes of s, as 16-bit patterns
__device__ __forceinline__ void split3(float s, uint32_t &p1, uint32_t &p2, uint32_t &p3) {
    p1 = bf16_bits(s);
    const float r1 = s - __uint_as_float(p1 << 16);
    p2 = bf16_bits(r1);
    const float r2 = r1 - __uint_as_float(p2 << 16);
    p3 = bf16_bits(r2);
}

// packed event of one input: x = event row (q + 1, -1 = none), y = L1 | L2 << 16,
// z = L3 | R1 << 16, w = R2 | R3 << 16
template <int KS>
__global__ __launch_bounds__(256) void mfma_events_kernel(LifConst C, int64_t n,
                                                          const float *__restrict__ t_in,
                                                          u32x4_t *__restrict__ ev) {
    const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const Event e = bin_event<KS>(C, t_in[k]);
    uint32_t l1, l2, l3, r1, r2, r3;
    split3(e.L, l1, l2, l3);
    split3(e.R, r1, r2, r3);
    ev[k] = u32x4_t{static_cast<uint32_t>(e.row), l1 | (l2 << 16), l3 | (r1 << 16), r2 | (r3 << 16)};
}

constexpr int kNT = 128;   // neurons per block tile (rows (b, m) per tile: MT, 128 or 64)
constexpr int kKT = 32;    // inputs per K tile
constexpr int kFrag = 64;  // 16-byte fragments per (32-row block, 16-k step)

// LDS fragment slot of (32-row block rb, k step ks, lane): one 16-byte
// fragment per lane, lanes consecutive (conflict-free 128-bit reads)
__device__ __forceinline__ int frag_slot(int rb, int ks, int lane) { return (rb * 2 + ks) * kFrag + lane; }

// MT rows per tile: each wave owns (MT / 2) x 64 of it, RA = MT / 64 row
// blocks of 32 (64-row tiles give twice the blocks where the grid of 128-row
// tiles would not fill the chip).
template <int MT>
__global__ __launch_bounds__(256) void mfma_contract_kernel(int M, int64_t rows, int N_in, int N_out,
                                                            const u32x4_t *__restrict__ ev,
                                                            const uint16_t *__restrict__ W,
                                                            float *__restrict__ wh) {
    constexpr int RB = MT / 32, RA = MT / 64;  // row blocks per tile and per wave
    __shared__ u32x4_t As[3 * RB * 2 * kFrag];  // [plane][row block][k step][lane]
    __shared__ u32x4_t Bs[4 * 2 * kFrag];       // [col block][k step][lane]
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid >> 6;
    const int64_t row0 = static_cast<int64_t>(blockIdx.y) * MT;
    const int col0 = blockIdx.x * kNT;
    const int M1 = M + 1;
    f32x16_t acc[RA][2];
#pragma unroll
    for (int a = 0; a < RA; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[a][bb][r] = 0.f;
    const int wr = wave >> 1, wc = wave & 1;
    // samples whose rows (b, m) fall in this tile
    const int64_t b_lo = row0 / M1;
    const int64_t b_hi = min((row0 + MT - 1) / M1, (rows - 1) / M1);
    const int ntask = static_cast<int>(b_hi - b_lo + 1) * kKT;  // (sample, input) events per K tile
    uint16_t *As16 = reinterpret_cast<uint16_t *>(As);
    constexpr int kPlane = RB * 2 * kFrag;  // fragments per plane
    for (int k0 = 0; k0 < N_in; k0 += kKT) {
        __syncthreads();
        // ---- S tile: zeroed here, the events' nonzero rows written below
#pragma unroll
        for (int h = 0; h < 3 * RB * 2 * kFrag / 256; ++h) As[tid + h * 256] = u32x4_t{0u, 0u, 0u, 0u};
        // ---- W tile: 16-byte runs of 8 inputs of one neuron
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int pr = tid + h * 256;
            const int i = pr & (kNT - 1), c = pr >> 7;
            const int gi = col0 + i;
            const int j = k0 + c * 8;
            u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
            if (gi < N_out && j < N_in) {
                const uint16_t *src = W + static_cast<int64_t>(gi) * N_in + j;
                if (j + 8 <= N_in && (N_in & 7) == 0) {
                    v = *reinterpret_cast<const u32x4_t *>(src);
                } else {
                    uint32_t w4[4] = {0u, 0u, 0u, 0u};
                    for (int e = 0; e < 8; ++e)
                        if (j + e < N_in) w4[e >> 1] |= static_cast<uint32_t>(src[e]) << ((e & 1) * 16);
                    v = u32x4_t{w4[0], w4[1], w4[2], w4[3]};
                }
            }
            Bs[frag_slot(i >> 5, c >> 1, (i & 31) + 32 * (c & 1))] = v;
        }
        __syncthreads();
        // ---- each event of the tile's samples writes its two nonzero rows
        // (L at row (b, q), R at row (b, q + 1)) in the three planes
        for (int t = tid; t < ntask; t += 256) {
            const int64_t b = b_lo + t / kKT;
            const int kk = t % kKT;
            const int j = k0 + kk;
            if (j >= N_in) continue;
            const u32x4_t x = ev[b * N_in + j];
            const int row = static_cast<int>(x.x);
            if (row < 0) continue;
            // element (r, kk) of a plane: 16-byte fragment (r/32, kk/16, lane
            // (r%32) + 32 ((kk/8)%2)), halfword kk%8
            const int fe = (((kk >> 3) & 1) * 32) * 8 + (kk & 7);
            const int fk = kk >> 4;
            const int64_t rL = b * M1 + (row - 1) - row0, rR = b * M1 + row - row0;
            if (row >= 1 && rL >= 0 && rL < MT) {
                const int r = static_cast<int>(rL);
                const int o = frag_slot(r >> 5, fk, r & 31) * 8 + fe;
                As16[o] = static_cast<uint16_t>(x.y & 0xFFFFu);
                As16[kPlane * 8 + o] = static_cast<uint16_t>(x.y >> 16);
                As16[2 * kPlane * 8 + o] = static_cast<uint16_t>(x.z & 0xFFFFu);
            }
            if (row <= M && rR >= 0 && rR < MT) {
                const int r = static_cast<int>(rR);
                const int o = frag_slot(r >> 5, fk, r & 31) * 8 + fe;
                As16[o] = static_cast<uint16_t>(x.z >> 16);
                As16[kPlane * 8 + o] = static_cast<uint16_t>(x.w & 0xFFFFu);
                As16[2 * kPlane * 8 + o] = static_cast<uint16_t>(x.w >> 16);
            }
        }
        __syncthreads();
        // ---- 2 k steps x 3 planes x (2 x 2) MFMA tiles per wave
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8_t bf[2];
#pragma unroll
            for (int bb = 0; bb < 2; ++bb)
                bf[bb] = __builtin_bit_cast(bf16x8_t, Bs[frag_slot(2 * wc + bb, ks, lane)]);
#pragma unroll
            for (int p = 0; p < 3; ++p) {
#pragma unroll
                for (int a = 0; a < RA; ++a) {
                    const bf16x8_t af =
                        __builtin_bit_cast(bf16x8_t, As[p * kPlane + frag_slot(RA * wr + a, ks, lane)]);
#pragma unroll
                    for (int bb = 0; bb < 2; ++bb)
                        acc[a][bb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf[bb], acc[a][bb], 0, 0, 0);
                }
            }
        }
    }
    // ---- epilogue: accumulator r of lane l is row (r/4)*8 + (l/32)*4 + r%4,
    // column l%32 of its 32 x 32 tile
#pragma unroll
    for (int a = 0; a < RA; ++a)
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            const int col = col0 + 32 * (2 * wc + bb) + (lane & 31);
            if (col >= N_out) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = row0 + 32 * (RA * wr + a) + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (row < rows) wh[row * N_out + col] = acc[a][bb][r];
            }
        }
}

// Interval scan and root solve over w^ [(b, 0..M)][N_out], one thread per
// (b, i); the wave stops once all its lanes have found their interval.
template <int KS>
__global__ __launch_bounds__(256) void mfma_scan_kernel(LifConst C, int N_out,
                                                        const float *__restrict__ wh,
                                                        float *__restrict__ t_out,
                                                        float *__restrict__ slope,
                                                        int *__restrict__ q_idx) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t b = blockIdx.y;
    const bool ok = i < N_out;
    const float *col = wh + b * (C.M + 1) * static_cast<int64_t>(N_out) + (ok ? i : 0);
    Scan<KS> sc;
    float wn = col[0];
    bool done = false;
    for (int m = 0; m < C.M && !done; ++m) {
        const float wc = wn;
        wn = col[static_cast<int64_t>(m + 1) * N_out];
        sc.template step_k<false>(C, m, wc);
        done = __all(sc.found() || !ok);
    }
    if (!done) sc.template step_k<true>(C, C.M, wn);  // the last interval
    if (!ok) return;
    float to, sl;
    int q;
    sc.finish(C, to, sl, q);
    const int64_t o = b * N_out + i;
    t_out[o] = to;
    slope[o] = sl;
    q_idx[o] = q;
}

hipError_t launch_forward_mfma(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out,
                               const uint16_t *W, void *ev, float *wh, const float *t_in,
                               float *t_out, float *slope, int *q_idx, hipStream_t st) {
    const bool gen = C.kind == kGeneral;
    {
        ProfScope prof("mfma_events", st);
        const int64_t n = B * N_in;
        const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
        if (n > 0) {
            if (gen)
                hipLaunchKernelGGL((mfma_events_kernel<kGeneral>), dim3(blocks), dim3(256), 0, st, C, n,
                                   t_in, static_cast<u32x4_t *>(ev));
            else
                hipLaunchKernelGGL((mfma_events_kernel<kAnyKind>), dim3(blocks), dim3(256), 0, st, C, n,
                                   t_in, static_cast<u32x4_t *>(ev));
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t rows = B * (C.M + 1);
    {
        ProfScope prof("fwd_mfma", st);
        // 64-row tiles where 128-row tiles would give fewer than four blocks per CU
        const int64_t nc = (N_out + kNT - 1) / kNT;
        const bool small = nc * ((rows + 127) / 128) < 1024;
        const int mt = small ? 64 : 128;
        dim3 grid(static_cast<unsigned>(nc), static_cast<unsigned>((rows + mt - 1) / mt));
        if (small)
            hipLaunchKernelGGL(mfma_contract_kernel<64>, grid, dim3(256), 0, st, C.M, rows,
                               static_cast<int>(N_in), static_cast<int>(N_out),
                               static_cast<const u32x4_t *>(ev), W, wh);
        else
            hipLaunchKernelGGL(mfma_contract_kernel<128>, grid, dim3(256), 0, st, C.M, rows,
                               static_cast<int>(N_in), static_cast<int>(N_out),
                               static_cast<const u32x4_t *>(ev), W, wh);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    ProfScope prof("mfma_scan", st);
    dim3 grid(static_cast<unsigned>((N_out + 255) / 256), static_cast<unsigned>(B));
    if (gen)
        hipLaunchKernelGGL((mfma_scan_kernel<kGeneral>), grid, dim3(256), 0, st, C, static_cast<int>(N_out), wh,
                           t_out, slope, q_idx);
    else
        hipLaunchKernelGGL((mfma_scan_kernel<kAnyKind>), grid, dim3(256), 0, st, C, static_cast<int>(N_out), wh,
                           t_out, slope, q_idx);
    return hipGetLastError();
}

}  // namespace dstd
