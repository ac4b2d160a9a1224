// dstd_kernels.h -- host-side launchers of the DSTD-LIF kernels (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "dstd_internal.h"

namespace dstd {

struct FwdPlan { int waves, spw; size_t lds; };
struct DwPlan { int waves, jw, nsplit, b_per_split; };

FwdPlan plan_forward(int M, int64_t B);
DwPlan plan_dw(int64_t B, int64_t N_in, int64_t N_out);
size_t dtin_lds_bytes(int M);

hipError_t launch_bin_events(const LifConst &C, int64_t n, const float *t_in, int *row, float *L,
                             float *R, float *dL, float *dR, hipStream_t st);
hipError_t launch_forward(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const void *W,
                          bool bf16, const int *row, const float *L, const float *R, float *t_out,
                          float *slope, int *q_idx, hipStream_t st);
hipError_t launch_grad_g(const LifConst &C, int64_t B, int64_t N_out, const float *t_out,
                         const float *slope, const int *q_idx, const float *grad_t, float *G,
                         hipStream_t st);
hipError_t launch_dw(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const float *G,
                     const int *row, const float *L, const float *R, float *dW, float *part,
                     hipStream_t st);
hipError_t launch_dtin(const LifConst &C, int64_t B, int64_t N_in, int64_t N_out, const float *G,
                       const void *W, bool bf16, const int *row, const float *dL, const float *dR,
                       float *dt_in, hipStream_t st);
hipError_t launch_softmax_ce(int64_t B, int64_t N, const float *t, const int *labels,
                             float tau_soft, float t_cap, float *grad, float *loss, hipStream_t st);
hipError_t launch_mse(int64_t B, int64_t N, const float *t, const float *y, float *grad,
                      float *loss, hipStream_t st);

}  // namespace dstd
