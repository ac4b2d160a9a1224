// dstd_kernels.h -- host-side launchers of the DSTD-LIF kernels (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dstd_internal.h"

namespace dstd {

struct DwPlan { int waves, jw, nsplit, b_per_split; };

// records past the end of a sample's sorted list that the forward kernel may
// read (and mask): the list array is padded by this many records
constexpr int kSortPad = 64;

DwPlan plan_dw(int64_t B, int64_t N_in, int64_t N_out, int M);
size_t dtin_partial_bytes(int M, int64_t B, int64_t N_in, int64_t N_out);

hipError_t launch_bin_events(const LifConst &C, int64_t n, const float *t_in, int *row, float *L,
                             float *R, float *dL, float *dR, hipStream_t st);
hipError_t launch_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const void *W,
                          bool bf16, void *Wt, SortedEv srt, int *n_valid, const float *t_in,
                          float *t_out, float *slope, int *q_idx, hipStream_t st);
hipError_t launch_grad_g(const LifConst &C, int64_t B, int64_t N_out, const float *t_out,
                         const float *slope, const int *q_idx, const float *grad_t, float *G,
                         hipStream_t st);
hipError_t launch_dw(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const float *G,
                     const int *row, const float *L, const float *R, float *dW, float *part,
                     hipStream_t st);
hipError_t launch_dtin(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const float *G,
                       const void *W, bool bf16, const int *row, const float *dL, const float *dR,
                       float *dt_in, float *part, hipStream_t st);
hipError_t launch_softmax_ce(int64_t B, int64_t N, const float *t, const int *labels,
                             float tau_soft, float t_cap, float *grad, float *loss, hipStream_t st);
hipError_t launch_mse(int64_t B, int64_t N, const float *t, const float *y, float *grad,
                      float *loss, hipStream_t st);

}  // namespace dstd
