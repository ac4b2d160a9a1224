/*
 * dstd_lif.h -- C ABI of the MI355X (gfx950) DSTD-LIF layer library.
 *
 * Differentiable spike-time discretization (DSTD) for a time-to-first-spike
 * leaky integrate-and-fire layer with membrane / synaptic time constants
 * (tau_m, tau_s), after Sakemi et al., "Scalable Training of Continuous-Time
 * Spiking Neural Networks with Differentiable Spike-Time Discretization".
 *
 * One layer maps presynaptic spike times t_j to weighted events at the grid
 * points T_m = t0 + m*dt (m = 0..M), contracts them with the weights, scans
 * the M intervals of every postsynaptic neuron for the first threshold
 * crossing and solves for the continuous spike time; the backward pass
 * returns gradients with respect to the weights and the input spike times.
 *
 * Conventions for every call:
 *  - All array pointers are DEVICE pointers owned by the caller; the library
 *    never allocates, frees or keeps device memory between calls (the one
 *    exception is the static scratch array of dstd_lif_forward_noalloc).
 *  - Arrays are dense, row-major, fp32 unless stated (W may be bf16).
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t, passed as
 *    void*; NULL = the default stream); outputs are valid once the stream
 *    reaches that point.
 *  - Scratch memory comes from the caller: `ws` of `ws_bytes` bytes, at
 *    least what the matching *_workspace_size() call returns, 256-byte
 *    aligned. Its contents need not be initialised and are clobbered.
 *  - Arguments are validated on the host before anything is enqueued; on a
 *    non-OK status nothing was enqueued and outputs are untouched (except
 *    DSTD_ERR_HIP, raised by a failed launch: outputs are then undefined).
 *  - Results are deterministic: no floating-point atomics across threads,
 *    fixed reduction orders; repeated calls give identical bits.
 *  - Calls are thread-safe; dstd_last_error() is per thread.
 */
#ifndef DSTD_LIF_H
#define DSTD_LIF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DSTD_OK = 0,
    DSTD_ERR_NULL = -1,        /* a required pointer is NULL */
    DSTD_ERR_SHAPE = -2,       /* negative / inconsistent sizes */
    DSTD_ERR_PARAM = -3,       /* invalid LIF or grid parameter */
    DSTD_ERR_UNSUPPORTED = -4, /* valid but not implemented (e.g. tau_m == tau_s, M too large) */
    DSTD_ERR_WORKSPACE = -5,   /* ws too small or misaligned */
    DSTD_ERR_HIP = -6          /* a HIP launch failed; see dstd_last_error() */
} dstd_status;

typedef enum { DSTD_F32 = 0, DSTD_BF16 = 1 } dstd_dtype;

/*
 * Layer parameters.
 *  tau_m, tau_s : membrane and synaptic time constants (the paper's tau_v,
 *                 tau_I; LIF model Eq. (LIF_model_TTFS)); each > 0, finite
 *                 or +INFINITY. The spike kernel (Table "tab:kernel") is
 *                 symmetric in the pair; its rows are selected by the pair:
 *                 two different finite constants (general row), two equal
 *                 finite constants ((tau, tau)), one infinite ((inf, tau)),
 *                 both infinite ((inf, inf)). Finite constants that differ by
 *                 no more than 1e-3 * max(tau_m, tau_s) without being equal
 *                 are DSTD_ERR_UNSUPPORTED (the general row loses precision
 *                 there and the paper defines no blend).
 *  threshold    : firing threshold V_th > 0. A neuron fires at the first t
 *                 where v(t) >= V_th.
 *  M            : number of DSTD intervals, 1 <= M <= DSTD_MAX_M; the grid
 *                 has M+1 points (App. B.1).
 *  t0, dt       : grid T_m = t0 + m*dt, dt > 0; the random t_offset of
 *                 Alg. 2 is folded into t0 by the caller.
 *  t_max        : end of the last candidate interval [T_M, t_max); +INFINITY
 *                 leaves it open (the exact method's t_{N+1} = inf, App. A).
 *                 Must be > T_M.
 *  flags        : 0, or one of the contraction choices of the dense forward
 *                 (ignored by the dense backward; any other call with a
 *                 contraction flag returns DSTD_ERR_UNSUPPORTED):
 *                  DSTD_FLAG_CONTRACT_SPARSE: the event-sparse contraction
 *                    (two-point event supports, vector ALU);
 *                  DSTD_FLAG_CONTRACT_MFMA: the dense product of the event
 *                    matrix [B(M+1)][N_in] and W on the matrix cores (bf16
 *                    weights only, else DSTD_ERR_UNSUPPORTED; the events are
 *                    split into three bf16 planes, so the products carry fp32
 *                    precision); it does (M+1)/2 times the method's
 *                    multiply-adds (App. B.3).
 *                 With neither, the library picks by shape (the MFMA product
 *                 for bf16 weights, M <= 8 and large layers, where it was
 *                 measured faster). Both set: DSTD_ERR_PARAM.
 *                 Conv calls take instead (see dstd_lif_conv_forward /
 *                 _backward):
 *                  DSTD_FLAG_CONV_KEEP (forward): keep the binned, sorted
 *                    inputs for the backward;
 *                  DSTD_FLAG_CONV_REUSE (backward): use what a forward with
 *                    DSTD_FLAG_CONV_KEEP kept.
 *                 A flag a call does not take gives DSTD_ERR_UNSUPPORTED.
 *                 Other bits must be 0.
 */
typedef struct {
    float tau_m, tau_s;
    float threshold;
    int32_t M;
    float t0, dt;
    float t_max;
    int32_t flags;
} dstd_lif_params;

#define DSTD_MAX_M 256
#define DSTD_FLAG_CONTRACT_SPARSE 0x2
#define DSTD_FLAG_CONTRACT_MFMA 0x4
#define DSTD_FLAG_CONV_KEEP 0x8
#define DSTD_FLAG_CONV_REUSE 0x10

/* ---------------------------------------------------------------- dense -- */

/* Workspace bytes needed by dstd_lif_forward / dstd_lif_backward. Returns 0
   for invalid arguments (the calls then report the precise error). */
size_t dstd_lif_forward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                       int64_t N_out);
size_t dstd_lif_backward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                        int64_t N_out);

/*
 * Forward pass of one dense layer (Eq. (DSTD), App. B.1 definition of the
 * weighted events, Table "tab:timing_DSTD", Eq. (timing_DSTD)).
 *  t_in  [B][N_in]      input spike times; +inf (any non-finite value) = no
 *                       spike. Inputs outside [T_0 - dt, T_M + dt) contribute
 *                       nothing; an input in [T_0 - dt, T_0) only contributes
 *                       its weight at T_0, one in [T_M, T_M + dt) only its
 *                       weight at T_M (Eq. (DSTD_kernel) at the grid ends).
 *  W     [N_out][N_in]  weights w_ij (input j -> neuron i), fp32 or bf16.
 *  t_out [B][N_out]     out: spike time, +inf if the neuron does not fire.
 *  slope [B][N_out]     out: dv/dt at the spike (0 if none); needed by backward.
 *  q_idx [B][N_out]     out: interval index q of the spike (T_q <= t < T_{q+1},
 *                       q = M for [T_M, t_max)), -1 if none.
 * B, N_in, N_out >= 0; zero sizes are valid no-ops (N_in == 0 gives silent
 * outputs). Only the O(B*N_out) outputs are kept for the backward pass.
 */
dstd_status dstd_lif_forward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                             const float *t_in, const void *W, dstd_dtype w_dtype,
                             float *t_out, float *slope, int32_t *q_idx,
                             void *ws, size_t ws_bytes, void *stream);

/*
 * Allocation-free variant of dstd_lif_forward, for callers that cannot
 * allocate device memory or take a workspace: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation. Same arguments,
 * outputs, validation and bits as dstd_lif_forward, without ws / ws_bytes;
 * its scratch is a static device array of DSTD_NOALLOC_SCRATCH_BYTES bytes
 * that the library holds on each GPU it runs on until the process ends (its
 * device address is looked up once per device, on the first call there).
 *  - A layer whose dstd_lif_forward_workspace_size() exceeds
 *    DSTD_NOALLOC_SCRATCH_BYTES is rejected with DSTD_ERR_WORKSPACE before
 *    anything touches the device.
 *  - It calls no hipMalloc / hipFree and no allocating routine.
 *  - All calls on one GPU share that GPU's array: calls that overlap in time
 *    on one GPU (different streams, or different threads without ordering)
 *    race on it and give undefined results. Calls ordered on one stream are
 *    safe; the forward writes every scratch word it reads, so nothing carries
 *    over from the previous call.
 */
#define DSTD_NOALLOC_SCRATCH_BYTES (32u << 20)
dstd_status dstd_lif_forward_noalloc(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                     int64_t N_out, const float *t_in, const void *W,
                                     dstd_dtype w_dtype, float *t_out, float *slope,
                                     int32_t *q_idx, void *stream);

/*
 * Backward pass of one dense layer. t_out, slope, q_idx are the forward's
 * outputs for the same (t_in, W, p). The interval index is piecewise
 * constant, so the spike time's derivative follows from the implicit-function
 * theorem applied to v^(t) = V_th: d t / d w^_m = -K(t - T_m) / slope for
 * m <= q, which equals differentiating the candidates of Table
 * "tab:timing_DSTD".
 *  grad_t_out [B][N_out]  dL/dt_out; ignored where q_idx < 0.
 *  grad_W     [N_out][N_in] out (fp32, overwritten, not accumulated), or NULL
 *                           to skip.
 *  grad_t_in  [B][N_in]   out (overwritten), or NULL to skip (first layer).
 *                         Inputs without events get 0.
 * A spike with slope below 1e-12 * threshold uses that floor (the exact
 * derivative of a tangent crossing is unbounded).
 */
dstd_status dstd_lif_backward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                              const float *t_in, const void *W, dstd_dtype w_dtype,
                              const float *t_out, const float *slope, const int32_t *q_idx,
                              const float *grad_t_out, float *grad_W, float *grad_t_in,
                              void *ws, size_t ws_bytes, void *stream);

/* ----------------------------------------------------------------- conv -- */

/*
 * Convolutional layer geometry. Inputs NCHW [B][C_in][H][W], weights
 * [C_out][C_in][KH][KW], outputs NCHW [B][C_out][H_out][W_out].
 *  pool_in : 1 = none; 2 = average the input EVENTS over 2x2 windows
 *            (H and W must be even) before the convolution; 0 = average them
 *            over the whole H x W map (a global pool: H_p = W_p = 1).
 *            Averaging events is linear, i.e. it averages the synaptic input
 *            currents. The paper's own nets down-sample with stride-2
 *            convolutions (Table "tab:architectures") and do not define spike
 *            pooling; this is the linear reading.
 *  H_out = (H_p + 2*pad - KH)/stride + 1 with H_p the (pooled) input height
 *  (likewise W_out); zero padding: padded positions have no events.
 * Supported: 1 <= KH, KW <= 7, stride >= 1, 0 <= pad <= max(KH, KW),
 * C_in, H, W, C_out >= 1, (M + 3) * W_p <= 16128, per-sample sizes below
 * 2^30 (DSTD_ERR_SHAPE / DSTD_ERR_UNSUPPORTED otherwise).
 */
typedef struct {
    int32_t C_in, H, W, C_out, KH, KW, stride, pad, pool_in;
} dstd_conv_shape;

/* Workspace bytes of dstd_lif_conv_forward / _backward; 0 for invalid
   arguments (the calls then report the precise error). With
   DSTD_FLAG_CONV_KEEP the forward's size is the backward's. */
size_t dstd_lif_conv_forward_workspace_size(const dstd_lif_params *p, const dstd_conv_shape *cs,
                                            int64_t B);
size_t dstd_lif_conv_backward_workspace_size(const dstd_lif_params *p, const dstd_conv_shape *cs,
                                             int64_t B);

/*
 * Forward pass of one conv layer: the dense forward (Eq. (DSTD), App. B.1,
 * Table "tab:timing_DSTD") with the convolution's connectivity, i.e.
 * w^_{(c,y,x), m} sums w_ij s_jm over the receptive field of output neuron
 * (c, y, x) (pooled events weighted by 1/P for a pool of P pixels).
 *  t_in  [B][C_in][H][W]          input spike times (+inf = no spike)
 *  W     [C_out][C_in][KH][KW]    fp32 or bf16 (converted to fp32 inside)
 *  t_out, slope, q_idx [B][C_out][H_out][W_out]  as in dstd_lif_forward.
 * With p->flags = DSTD_FLAG_CONV_KEEP the workspace must have
 * dstd_lif_conv_backward_workspace_size bytes (else DSTD_ERR_WORKSPACE): the
 * call also leaves there what the layer's backward would derive from t_in
 * and W again -- the inputs binned to their events and sorted, with the
 * event weights' derivatives (the events s_jm of Eq. (DSTD_kernel) and
 * ds/dt depend on t_in alone), the cell-major events for dW and the
 * weights' layout -- for a dstd_lif_conv_backward with
 * DSTD_FLAG_CONV_REUSE on the same workspace.
 * B = 0 is a valid no-op.
 */
dstd_status dstd_lif_conv_forward(const dstd_lif_params *p, const dstd_conv_shape *cs, int64_t B,
                                  const float *t_in, const void *W, dstd_dtype w_dtype,
                                  float *t_out, float *slope, int32_t *q_idx,
                                  void *ws, size_t ws_bytes, void *stream);

/*
 * Backward pass of one conv layer (same chain rule as dstd_lif_backward).
 *  grad_W    [C_out][C_in][KH][KW] out (fp32, overwritten; zeros for B = 0),
 *            or NULL to skip.
 *  grad_t_in [B][C_in][H][W] out (overwritten), or NULL to skip; inputs
 *            without events get 0.
 * With p->flags = DSTD_FLAG_CONV_REUSE the workspace must hold what a
 * dstd_lif_conv_forward with DSTD_FLAG_CONV_KEEP wrote for the same t_in, W,
 * shape, B and (apart from flags) parameters, unchanged since; the call then
 * skips binning, sorting and the weight layout. The library cannot check
 * this (the data are on the device): other contents give wrong gradients
 * (indices read from the workspace are clamped, so accesses stay inside the
 * workspace and the outputs). Results are bitwise those of the call without
 * the flag.
 */
dstd_status dstd_lif_conv_backward(const dstd_lif_params *p, const dstd_conv_shape *cs, int64_t B,
                                   const float *t_in, const void *W, dstd_dtype w_dtype,
                                   const float *t_out, const float *slope, const int32_t *q_idx,
                                   const float *grad_t_out, float *grad_W, float *grad_t_in,
                                   void *ws, size_t ws_bytes, void *stream);

/* --------------------------------------------------------------- losses -- */

/*
 * Softmax cross-entropy on the output spike times (App. C.1): logits
 * -t/tau_soft, S = softmax, L = -(1/B) sum_b ln S_{b, label_b}. Neurons that
 * did not fire (t = +inf) enter the softmax at t_cap and get no gradient.
 *  t_out [B][N], labels [B] int32 in [0, N), grad_t [B][N] out = dL/dt,
 *  loss [B + 1] out (device floats): loss[0] = L, loss[1 + b] = sample b's
 *  term -(1/B) ln S_{b, label_b} (summed into loss[0] in a fixed order).
 *  1 <= N < 2^24, 0 <= B <= 65535.
 */
dstd_status dstd_softmax_ce_grad(int64_t B, int64_t N, const float *t_out, const int32_t *labels,
                                 float tau_soft, float t_cap, float *grad_t, float *loss,
                                 void *stream);

/* Mean squared error L = (1/B) sum_{b,i fired} (t - y)^2 / 2 over fired
   outputs; grad_t [B][N] out; loss [B + 1] out (device floats): loss[0] = L,
   loss[1 + b] = sample b's term. 1 <= N < 2^24, 0 <= B <= 65535. */
dstd_status dstd_mse_grad(int64_t B, int64_t N, const float *t_out, const float *target,
                          float *grad_t, float *loss, void *stream);

/* ------------------------------------------------------ synfire terms -- */

/*
 * Synfire-chain training terms of one layer (App. C.1, Eqs.
 * (temporal_penalty) and (dead_neuron_penalty)), for the outputs t of the
 * layer's forward pass.
 *  Temporal penalty  T = scale * sum over neurons that fire (t finite) of
 *      gamma_head (t - t_head)^2 [t < t_head] + gamma_tail (t - t_tail)^2 [t > t_tail];
 *    silent neurons (t = +inf) contribute nothing (the paper's dead-neuron
 *    term exists because T gives them no gradient).
 *  Dead-neuron term  Q = -gamma_q * scale * sum over silent neurons of the
 *      sum of their weight row (dense: row i of W; conv: all weights of the
 *      neuron's output channel), so dQ/dw_ij = -gamma_q * scale * (number of
 *      silent neurons that row i feeds).
 * t_head, t_tail are this layer's window ends, l * tau_shift + t_head and
 * l * tau_shift + tau_width - t_tail in the paper's hyperparameters (the
 * caller forms them). scale folds the mini-batch mean and, for conv layers,
 * the division by the spatial size: 1/B (dense) or 1/(B * H_out * W_out).
 * All gammas >= 0 and finite, t_head and t_tail finite, scale > 0 and finite
 * (DSTD_ERR_PARAM otherwise).
 */
typedef struct {
    float gamma_head, gamma_tail;
    float t_head, t_tail;
    float gamma_q;
    float scale;
} dstd_synfire_params;

/*
 * Backward passes with the synfire terms: as dstd_lif_backward /
 * dstd_lif_conv_backward (same workspace size), except that each firing
 * neuron's gradient is grad_t_out + dT/dt (added inside the kernels that
 * build the per-neuron gradient), and grad_W additionally holds dQ/dW
 * (added where the dW sums are written). sp = NULL gives the plain
 * backward; all gammas zero give the plain backward's results bit for bit.
 */
dstd_status dstd_lif_backward_synfire(const dstd_lif_params *p, const dstd_synfire_params *sp,
                                      int64_t B, int64_t N_in, int64_t N_out,
                                      const float *t_in, const void *W, dstd_dtype w_dtype,
                                      const float *t_out, const float *slope,
                                      const int32_t *q_idx, const float *grad_t_out,
                                      float *grad_W, float *grad_t_in, void *ws,
                                      size_t ws_bytes, void *stream);
dstd_status dstd_lif_conv_backward_synfire(const dstd_lif_params *p, const dstd_synfire_params *sp,
                                           const dstd_conv_shape *cs, int64_t B,
                                           const float *t_in, const void *W, dstd_dtype w_dtype,
                                           const float *t_out, const float *slope,
                                           const int32_t *q_idx, const float *grad_t_out,
                                           float *grad_W, float *grad_t_in, void *ws,
                                           size_t ws_bytes, void *stream);

/*
 * Values of the two terms (for reporting; the gradients come from the
 * backward calls above). The layer's outputs are t_out [B][rows][spatial]
 * (dense: rows = N_out, spatial = 1; conv NCHW: rows = C_out, spatial =
 * H_out * W_out); W holds rows x row_len weights, row-major (dense [N_out]
 * [N_in]; conv [C_out][C_in * KH * KW]), fp32 or bf16.
 *  value [2] out (device floats): value[0] = T, value[1] = Q, each summed in
 *  a fixed order (bitwise reproducible).
 * Workspace: dstd_synfire_penalty_workspace_size(B, rows, spatial) bytes,
 * 256-byte aligned. B, rows, spatial >= 0 with per-layer element counts
 * below 2^31; rows * row_len below 2^31.
 */
size_t dstd_synfire_penalty_workspace_size(int64_t B, int64_t rows, int64_t spatial);
dstd_status dstd_synfire_penalty(const dstd_synfire_params *sp, int64_t B, int64_t rows,
                                 int64_t spatial, int64_t row_len, const float *t_out,
                                 const void *W, dstd_dtype w_dtype, float *value, void *ws,
                                 size_t ws_bytes, void *stream);

/* ------------------------------------------------------------ profiling -- */

/*
 * Opt-in per-kernel timing (not from the paper: an instrument for measuring
 * this library). While enabled, each kernel the library launches is bracketed
 * by hipEvents on its stream; dstd_profile_collect() waits for them and adds
 * the durations to per-kernel totals readable with dstd_profile_entry().
 * Keep it disabled while capturing a stream into a graph.
 *  dstd_profile_enable : on != 0 enables; returns the previous setting.
 *  dstd_profile_entry  : idx in [0, dstd_profile_count()); *name stays valid
 *                        until dstd_profile_reset().
 */
int32_t dstd_profile_enable(int32_t on);
dstd_status dstd_profile_collect(void);
int32_t dstd_profile_count(void);
dstd_status dstd_profile_entry(int32_t idx, const char **name, int64_t *launches,
                               double *total_ms);
void dstd_profile_reset(void);

/* ----------------------------------------------------------- multispike -- */

/*
 * Multi-spike DSTD for a dense layer (App. "multi-spikes", Eq.
 * (Vmem_multiSpikes) and its DSTD form). Every input neuron may fire up to
 * F_in times; each input spike gets its own events (Eq. (DSTD_kernel)) and
 * the weighted events sum them. An output neuron fires whenever v reaches
 * V_th; v is then reset to 0 and the synaptic current is not, so after a
 * spike at t_k the potential is I(t_k) K(t - t_k) plus the events after t_k.
 * The first F_out spikes are computed, in time order (several may fall in
 * one interval).
 *  t_in  [B][N_in][F_in]   input spike times (non-finite = no spike; any order)
 *  W     [N_out][N_in]     fp32 or bf16
 *  t_out, slope, q_idx, cur [B][N_out][F_out]  out: spike times (+inf after
 *          the last), dv/dt at each spike, its interval (-1 after the last)
 *          and the synaptic current at the spike (kept for the backward)
 * 1 <= F_in, F_out <= 64; M <= 250 (DSTD_ERR_UNSUPPORTED beyond); the grid,
 * t_max and other limits as in dstd_lif_forward.
 */
size_t dstd_lif_multispike_forward_workspace_size(const dstd_lif_params *p, int64_t B,
                                                  int64_t N_in, int64_t F_in, int64_t N_out,
                                                  int64_t F_out);
size_t dstd_lif_multispike_backward_workspace_size(const dstd_lif_params *p, int64_t B,
                                                   int64_t N_in, int64_t F_in, int64_t N_out,
                                                   int64_t F_out);
dstd_status dstd_lif_multispike_forward(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                        int64_t F_in, int64_t N_out, int64_t F_out,
                                        const float *t_in, const void *W, dstd_dtype w_dtype,
                                        float *t_out, float *slope, int32_t *q_idx, float *cur,
                                        void *ws, size_t ws_bytes, void *stream);

/*
 * Backward: with the intervals fixed, each spike solves v_k(t_k) = V_th, and
 * v_k depends on the weighted events and, through the reset, on t_{k-1}
 * (d t_k / d t_{k-1} = I(t_{k-1}) (K(d)/tau_I + K'(d)) / slope_k,
 * d = t_k - t_{k-1}). Adjoints run from the last spike back, then dL/dW and
 * dL/dt_in follow through the events as in dstd_lif_backward.
 *  t_out, slope, q_idx, cur  the forward's outputs for the same inputs
 *  grad_t_out [B][N_out][F_out]  dL/dt_out; ignored where q_idx < 0
 *  grad_W [N_out][N_in]          out (fp32, overwritten), or NULL
 *  grad_t_in [B][N_in][F_in]     out (overwritten), or NULL; input spikes
 *                                without events get 0
 */
dstd_status dstd_lif_multispike_backward(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                         int64_t F_in, int64_t N_out, int64_t F_out,
                                         const float *t_in, const void *W, dstd_dtype w_dtype,
                                         const float *t_out, const float *slope,
                                         const int32_t *q_idx, const float *cur,
                                         const float *grad_t_out, float *grad_W,
                                         float *grad_t_in, void *ws, size_t ws_bytes,
                                         void *stream);

/* ----------------------------------------------------------------- skip -- */

/*
 * Skip-and-delay connection of an SD block (App. C.3, Fig. "skip_connection",
 * Table "tab:architectures"): the block's third layer receives the spikes
 * entering the block, delayed by a fixed 2 tau_shift, together with the
 * second layer's spikes. The delay moves those inputs into the third layer's
 * synfire window. The two maps are concatenated along channels (block input
 * first), and the result is the t_in of an ordinary conv call.
 *  t1  [B][C1][HW]       spikes entering the block
 *  t2  [B][C2][HW]       the block's second-layer output (same H x W = HW)
 *  out [B][C1 + C2][HW]  out: t1 + delay, then t2 (non-finite times stay
 *                        silent: +inf + delay = +inf)
 * delay finite; sizes >= 0 with (C1 + C2) * HW < 2^30 and B <= 65535.
 */
dstd_status dstd_skip_delay_concat(int64_t B, int64_t C1, int64_t C2, int64_t HW, const float *t1,
                                   float delay, const float *t2, float *out, void *stream);

/*
 * Its backward: the delay is a constant shift, so each channel's gradient
 * passes back unchanged.
 *  g  [B][C1 + C2][HW]  dL/d(out)
 *  g1 [B][C1][HW]       out: the first C1 channels of g; added to g1's
 *                       contents when accumulate = 1 (the block input also
 *                       feeds the block's first layer, whose dt_in is already
 *                       there), written when 0; NULL to skip
 *  g2 [B][C2][HW]       out (written): the remaining channels; NULL to skip
 */
dstd_status dstd_skip_delay_concat_backward(int64_t B, int64_t C1, int64_t C2, int64_t HW,
                                            const float *g, float *g1, int32_t accumulate,
                                            float *g2, void *stream);

/* ---------------------------------------------------------------- exact -- */

/*
 * Exact spike times of a dense layer without discretization (App. A, Alg. 1,
 * Eq. (timing_exact)): the method DSTD approximates, for measuring it against
 * DSTD. Of dstd_lif_params only tau_m, tau_s, threshold, t_max and flags are
 * used (validated as for the DSTD calls; t_max may be any non-NaN value); M,
 * t0 and dt are ignored. Supported: N_in <= 8192 (DSTD_ERR_UNSUPPORTED
 * beyond: one workgroup sorts a sample's inputs), the other size limits as in
 * dstd_lif_forward.
 */
size_t dstd_exact_forward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                         int64_t N_out);
size_t dstd_exact_backward_workspace_size(const dstd_lif_params *p, int64_t B, int64_t N_in,
                                          int64_t N_out);

/*
 * Forward: per sample the finite inputs with t < t_max are sorted ascending
 * (t~_1 <= t~_2 <= ...); on [t~_k, t~_{k+1}) the potential is
 * sum_{j <= k} w_ij K(t - t~_j), and the spike is the first time it reaches
 * the threshold, the first interval whose candidate lies inside it
 * (Eq. (timing_exact); the last interval ends at t_max, +INFINITY = open).
 * Simultaneous inputs add up before their interval is tested.
 *  t_in  [B][N_in]     input spike times; non-finite = no spike.
 *  W     [N_out][N_in] fp32 or bf16.
 *  t_out [B][N_out]    out: spike time, +inf if none.
 *  slope [B][N_out]    out: dv/dt at the spike (0 if none).
 *  k_idx [B][N_out]    out: position (0-based) in the sorted order of the
 *                      left end of the crossing interval, -1 if none; the
 *                      causal set of the spike is every input with
 *                      t_j <= t~_k.
 */
dstd_status dstd_exact_forward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                               const float *t_in, const void *W, dstd_dtype w_dtype,
                               float *t_out, float *slope, int32_t *k_idx,
                               void *ws, size_t ws_bytes, void *stream);

/*
 * Backward: with the causal set fixed (piecewise-constant, as is the choice
 * of interval), the implicit-function theorem on v(t_i) = V_th gives
 * d t_i / d w_ij = -K(t_i - t_j) / slope_i and
 * d t_i / d t_j = w_ij K'(t_i - t_j) / slope_i for t_j <= t~_k; this equals
 * differentiating the selected candidate of Table "tab:spike_timing".
 *  t_out, slope, k_idx  the forward's outputs for the same (t_in, W, p).
 *  grad_t_out [B][N_out] dL/dt_out; ignored where k_idx < 0.
 *  grad_W [N_out][N_in]  out (fp32, overwritten), or NULL to skip.
 *  grad_t_in [B][N_in]   out (overwritten), or NULL to skip; inputs that
 *                        are not finite get 0.
 * Slopes below 1e-12 * threshold use that floor, as in dstd_lif_backward.
 */
dstd_status dstd_exact_backward(const dstd_lif_params *p, int64_t B, int64_t N_in, int64_t N_out,
                                const float *t_in, const void *W, dstd_dtype w_dtype,
                                const float *t_out, const float *slope, const int32_t *k_idx,
                                const float *grad_t_out, float *grad_W, float *grad_t_in,
                                void *ws, size_t ws_bytes, void *stream);

/* ----------------------------------------------------------------- misc -- */

const char *dstd_status_string(dstd_status s);
/* Detail of the last non-OK status returned on the calling thread. */
const char *dstd_last_error(void);
/* Library ABI version (major * 100 + minor). */
int32_t dstd_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DSTD_LIF_H */
