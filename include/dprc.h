/*
 * dprc.h -- randomized per-sample gradient-norm estimation for DP-SGD with
 * randomized clipping (DP-SGD-RC), for AMD Instinct MI355X (gfx950).
 *
 * The calls follow the problem statement of the paper "Efficient DP-SGD for
 * LLMs with Randomized Clipping":
 *   - Algorithm 2 (Norm-Estimation-Routine): per-sample squared-norm estimates
 *     of a bias-free linear layer S = A W from its activations A[B,T,d] and
 *     output gradients E = dL/dS [B,T,p], by the Hutchinson estimator
 *     (dprc_norm_hutch) or by Hutch++ (dprc_norm_hutchpp);
 *   - Algorithm 1 (DP-SGD-RC step): the squared norms summed over layers, the
 *     clip factors min(1, C/sqrt(n_i)) (dprc_clip_scale), the clipped gradient
 *     sum_i c_i A_i^T E_i that the second backward pass produces for a linear
 *     layer (dprc_clip_accumulate), and the Gaussian noise sigma*C*N(0,I)
 *     (dprc_add_noise).
 *
 * Conventions for every call:
 *   - Pointers named A, E, n2, c, grad, ws, out are DEVICE pointers; the
 *     dprc_layer array itself is HOST memory and is read during the call only.
 *   - Every call is asynchronous on `stream` (0 = the null stream) and returns
 *     after enqueueing; results are valid once the stream reaches that point.
 *   - The library never allocates or frees memory and creates no streams or
 *     events; its only host state is the opt-in, per-thread launch-trace hook
 *     (dprc_trace_launches).  Scratch space is the caller's `ws` buffer of at least the size returned
 *     by the matching *_workspace() query, 256-byte aligned.  Calls that share
 *     a workspace must be ordered (same stream, or synchronised).
 *   - Arguments are validated on the host before anything is enqueued; a
 *     failed check returns a non-zero dprc_status and enqueues nothing.  A
 *     failed launch returns DPRC_ERROR_HIP.  No C++ exception crosses the ABI.
 *   - Tensors are row-major with token rows: element (i, t, j) of A is at
 *     A + (i*T + t)*lda + j.  Pointers must be aligned to their element size
 *     (else DPRC_ERROR_NOT_SUPPORTED).  bf16 rows that start on 16-byte
 *     boundaries (16-byte aligned base, stride a multiple of 8) with a width
 *     that is a multiple of 8 take 16-byte loads; other layouts are correct
 *     but slower (element loads).
 *
 * Probes: +-1 (Rademacher) entries from Philox4x32-10 (Salmon et al., SC'11)
 * keyed by (seed, layer_id, stream), shared by all samples of a layer and
 * fresh per layer; the caller folds the training step into `seed`.  Column j,
 * rows 32w..32w+31 of a layer's probe matrix in stream s is word (w mod 4) of
 * Philox(counter = (w div 4, j, layer_id, s), key = (seed lo, seed hi)); bit b
 * gives row 32w+b, 0 -> +1, 1 -> -1.  Streams: 0 = Hutchinson probes (also
 * the Hutch++ residual probes), 1 = Hutch++ sketch, 2 = Gaussian noise.
 */
#ifndef DPRC_H
#define DPRC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DPRC_SUCCESS = 0,
  DPRC_ERROR_INVALID_VALUE = 1,      /* null pointer, non-positive size, bad enum, ...   */
  DPRC_ERROR_NOT_SUPPORTED = 2,      /* alignment / stride / size outside supported range */
  DPRC_ERROR_WORKSPACE_TOO_SMALL = 3,
  DPRC_ERROR_HIP = 4,                /* a HIP runtime call or launch failed              */
  DPRC_ERROR_SCRATCH_LIMIT = 5       /* dprc_norm_hutch_clip_static: needs more scratch
                                        than DPRC_STATIC_SCRATCH_BYTES                   */
} dprc_status;

typedef enum { DPRC_F32 = 0, DPRC_BF16 = 1 } dprc_dtype;

/* Which dimension the probes sketch.  OUT sketches the p side (Z is p x k,
 * Algorithm 2 as printed), IN sketches the d side (Z is d x k; the text notes
 * the two are equivalent since ||A^T E||_F = ||E^T A||_F), AUTO sketches the
 * larger dimension (the paper's proof sketch projects the larger one), ties
 * going to OUT. */
typedef enum { DPRC_SIDE_OUT = 0, DPRC_SIDE_IN = 1, DPRC_SIDE_AUTO = 2 } dprc_side;

/* Probe family.  RADEMACHER: the counter-generated +-1 probes above.
 * HADAMARD: the deterministic Sylvester-Hadamard signs z(u,j) =
 * (-1)^popcount(u & j) (verification: with k = 2^q >= the sketched dimension
 * the estimate equals the exact squared norm).  GAUSSIAN (Hutchinson only,
 * k <= 32): the normal-law probes of Algorithm 2 (standard normal entries, the
 * estimate divided by k as for the other families), entry (u, j) from Philox
 * stream 3 block (u div 4, j, layer_id, 3) through the Box-Muller transform of
 * dprc_add_noise: words (x0, x1) give rows 4q, 4q+1 and (x2, x3) rows 4q+2,
 * 4q+3.  They are generated into the workspace as bf16 hi + lo pairs (fp32 for
 * fp32 layers) and applied as dense probe columns. */
typedef enum { DPRC_PROBE_RADEMACHER = 0, DPRC_PROBE_HADAMARD = 1, DPRC_PROBE_GAUSSIAN = 2 } dprc_probe;

/* One bias-free linear layer S = A W (section "Proposed Method"). */
typedef struct {
  const void* A;      /* activations [B,T,d], device                       */
  const void* E;      /* output gradients dL/dS [B,T,p], device            */
  int64_t B, T, d, p; /* all >= 1                                          */
  int64_t lda, lde;   /* token-row strides in elements, lda >= d, lde >= p */
  dprc_dtype dtype;   /* both tensors share it                             */
  uint32_t layer_id;  /* probe-key component; unique per layer in a step   */
} dprc_layer;

/* ---- Hutchinson (Algorithm 2, Hutch branch) --------------------------------
 * For each layer and sample i: Y_i = X_i Z (X the sketched operand, T x m,
 * Z the m x k probes), W_i = X'_i^T Y_i (X' the other operand), estimate
 * ||W_i||_F^2 / k, an unbiased estimate of ||A_i^T E_i||_F^2.
 *   n2[B]                 : = (accumulate == 0) or += (accumulate != 0) the
 *                           sum over the layers of the estimates (Algorithm 1,
 *                           layer-wise summation).  fp32, device.
 *   n2_layers[num_layers*B]: optional (may be NULL) per-layer estimates.
 *   k in [1, 256] (GAUSSIAN probes: k <= 32, else DPRC_ERROR_NOT_SUPPORTED).
 *   All layers must have the same B.
 * Workspace: dprc_norm_hutch_workspace() bytes for the same arguments (0 when
 * they are invalid).  When every layer is bf16, up to 32 groups of layers
 * keep their own token-split partials in it at once (their split sums take one
 * launch), and with RADEMACHER or HADAMARD probes also their own projected Y
 * (B x T rounded up to 64, x 2 x the group's columns rounded up to 16, bf16),
 * so their projections and token reductions are batched too; it grows with the
 * number of layers up to that many groups.  Every group's tile sums (B x
 * ceil(reduced width / 128) doubles per layer) stay in it until the per-sample
 * sums of all layers at the end of the call. */
size_t dprc_norm_hutch_workspace(const dprc_layer* layers, int32_t num_layers, int32_t k,
                                 dprc_probe probe, dprc_side side);
dprc_status dprc_norm_hutch(const dprc_layer* layers, int32_t num_layers, int32_t k,
                            dprc_probe probe, uint64_t seed, dprc_side side, float* n2,
                            float* n2_layers, int32_t accumulate, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* Hutchinson estimates followed by the clip factors of Algorithm 1 in the same
 * launches: as dprc_norm_hutch, then c[i] = the dprc_clip_scale factor of the
 * final n2[i] (bitwise the same as calling dprc_clip_scale on n2).  C > 0 and
 * finite; c [B] device.  Workspace: dprc_norm_hutch_workspace(). */
dprc_status dprc_norm_hutch_clip(const dprc_layer* layers, int32_t num_layers, int32_t k,
                                 dprc_probe probe, uint64_t seed, dprc_side side, float C, float* n2,
                                 float* c, float* n2_layers, int32_t accumulate, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* The same call for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): identical arguments and
 * results (bit for bit) to dprc_norm_hutch_clip, without the workspace.  Its scratch
 * is a static device array of DPRC_STATIC_SCRATCH_BYTES that the library's code
 * object holds on every device it runs on until the process ends; the call allocates
 * nothing and frees nothing.  A call whose dprc_norm_hutch_workspace() exceeds that
 * size returns DPRC_ERROR_SCRATCH_LIMIT and enqueues nothing (the 113-layer
 * Llama-3.2-1B stack at B = 8, T = 4096, k = 32 needs 136 MiB).  `stream` must belong
 * to the current device (else DPRC_ERROR_INVALID_VALUE); the first call on a device
 * looks up that device's copy of the array (hipGetSymbolAddress) and keeps its
 * address for the process, so make that first call outside graph capture.  Every
 * call on one device shares the array: calls that overlap on one device (different
 * streams, or host threads without ordering between their streams) race on it and
 * must be serialised by the caller.  Nothing in it needs to start cleared; it keeps
 * the last call's contents. */
#define DPRC_STATIC_SCRATCH_BYTES (256u << 20)
dprc_status dprc_norm_hutch_clip_static(const dprc_layer* layers, int32_t num_layers, int32_t k,
                                        dprc_probe probe, uint64_t seed, dprc_side side, float C,
                                        float* n2, float* c, float* n2_layers, int32_t accumulate,
                                        hipStream_t stream);

/* ---- Hutch++ (Algorithm 2, Hutch++ branch; estimator section) --------------
 * With M_i = X'_i^T X_i (m probed columns): sketch O S = M_i^T (M_i S) with s
 * sketch probes (stream 1), Q = orthonormal basis of its columns (Householder
 * QR), U = M_i Q, V = M_i P - U (Q^T P) with r residual probes P (stream 0),
 * estimate ||U||_F^2 + ||V||_F^2 / r.  s in [0, 32], r in [1, 256],
 * s + r <= 256, s <= the sketched dimension.  s = 0 gives Hutchinson with r
 * probes.  A sketched dimension above 2^21 rows returns DPRC_ERROR_NOT_SUPPORTED
 * (the QR tree of 128-row blocks is at most eight levels deep).  Outputs as for
 * dprc_norm_hutch.  With several bf16 layers and s > 0, up to eight layers keep
 * their sketches, QR trees and partials in the workspace at once (each level of
 * their QR trees is one launch for all of them), so dprc_norm_hutchpp_workspace()
 * grows with the number of layers up to eight.  Everything is enqueued on
 * `stream` alone. */
size_t dprc_norm_hutchpp_workspace(const dprc_layer* layers, int32_t num_layers, int32_t s,
                                   int32_t r, dprc_side side);
dprc_status dprc_norm_hutchpp(const dprc_layer* layers, int32_t num_layers, int32_t s, int32_t r,
                              uint64_t seed, dprc_side side, float* n2, float* n2_layers,
                              int32_t accumulate, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- clip factors (Algorithm 1, scaled loss) ---------------------------------
 * c[i] = min(1, C / sqrt(n2[i])); n2 = 0 gives 1; a NaN, infinite or negative
 * n2 gives 0 (the sample is dropped).  C > 0 and finite.  Device n2[B], c[B]. */
dprc_status dprc_clip_scale(const float* n2, int64_t B, float C, float* c, hipStream_t stream);

/* ---- clipped accumulation (Algorithm 1, second backward pass) ----------------
 * grad[j*ldg + u] (=|+=) sum_i c[i] * sum_t A[i,t,j] * E[i,t,u]   (d x p, fp32)
 * i.e. the weight gradient of S = A W for the loss sum_i c_i L_i with the c_i
 * held constant.  Samples with c[i] == 0 are skipped entirely.  bf16 inputs
 * run on bf16 matrix cores with fp32 accumulation; the per-sample factor is
 * applied to the fp32 accumulator, never to the bf16 inputs.  ldg >= p. */
size_t dprc_clip_accumulate_workspace(const dprc_layer* layer);
dprc_status dprc_clip_accumulate(const dprc_layer* layer, const float* c, float* grad,
                                 int64_t ldg, int32_t accumulate, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* The same for num_layers bf16 layers of one batch (same B; T, d and p free):
 * grads[l][j*ldg[l] + u] (=|+=) the sum above for layer l.  No layer is split over its
 * tokens, so no workspace is needed: a layer with at least 256 output tiles of
 * 256 x 256 takes a launch of its own, and the smaller ones share launches (up to 64
 * layers each) where dprc_clip_accumulate would split them.  grads and ldg
 * are host arrays of num_layers entries (device pointers, row strides >= p); the
 * gradients must not overlap.  Each layer's result is the one dprc_clip_accumulate
 * gives with one token split, up to the order of the fp32 sums.  Any fp32 layer gives
 * DPRC_ERROR_NOT_SUPPORTED. */
dprc_status dprc_clip_accumulate_layers(const dprc_layer* layers, int32_t num_layers, const float* c,
                                        float* const* grads, const int64_t* ldg, int32_t accumulate,
                                        hipStream_t stream);

/* ---- Gaussian noise (Algorithm 1) ---------------------------------------------
 * grad[e] += sigma * C * xi_e for e in [0, numel), xi_e standard normal from
 * Philox (stream 2) keyed by (seed, tensor_id): element e uses words of
 * block e div 4 through the Box-Muller transform with uniforms
 * (floor(x / 2^9) + 1/2) * 2^-23.  sigma >= 0, C > 0, both finite. */
dprc_status dprc_add_noise(float* grad, int64_t numel, float sigma, float C, uint64_t seed,
                           uint32_t tensor_id, hipStream_t stream);

/* ---- Private AdamW step (Algorithm 1: noise addition and optimizer step) --------
 * One AdamW step (Adam with decoupled weight decay, the optimizer of the
 * paper's private runs) on one layer's fp32 master weights, fed the private
 * gradient
 *   g[r][c] = (G[r][c] + sigma * C * xi_e) * inv_batch,   e = r * p + c,
 * where G [d, p] (row stride ldg) is the clipped gradient sum from
 * dprc_clip_accumulate and xi_e is the value dprc_add_noise(seed, tensor_id)
 * would add to element e of a contiguous [d, p] buffer (sigma = 0: none).
 * With t = hp->step (1-based), for every element:
 *   theta *= 1 - lr * weight_decay;
 *   m = beta1 m + (1 - beta1) g;   v = beta2 v + (1 - beta2) g^2;
 *   theta -= lr / (1 - beta1^t) * m / (sqrt(v) / sqrt(1 - beta2^t) + eps).
 * theta, m, v: fp32 [d, p] with row stride ldt >= p, updated in place; G is
 * read only.  w (may be NULL) receives bf16(theta) transposed, w[c][r] with
 * row stride ldw >= d (the [p, d] weight of a linear layer), rounded to
 * nearest even.  Device pointers, fp32 ones 4-byte aligned, w 2-byte aligned;
 * 16-byte aligned rows with p a multiple of 4 take vector accesses.
 * hp: host pointer; lr >= 0, 0 <= beta1, beta2 < 1, eps > 0, step >= 1. */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
  int32_t step;
} dprc_adamw_params;
dprc_status dprc_private_adamw(float* theta, float* m, float* v, int64_t ldt, const float* G, int64_t ldg,
                               int64_t d, int64_t p, float sigma, float C, uint64_t seed,
                               uint32_t tensor_id, float inv_batch, const dprc_adamw_params* hp,
                               uint16_t* w, int64_t ldw, hipStream_t stream);

/* ---- Envelope CDF of the Hutchinson estimate (privacy accounting) ------------------
 * Proposition on the extremal envelope and the appendix algorithms cdf-grid and
 * binary-search-xplus.  dprc_envelope_middle evaluates MiddleRegionCDF at nx
 * points: best[e] = the largest P(S <= x[e]) over the two-level forms
 *   S(i, j, lam) = lam/(ik) chi^2(ik) + (1-lam)/(jk) chi^2(jk),
 *   i, j >= 1, i + j <= d, lam = l / (2 (n_lambda - 1)), l = 0 .. n_lambda - 1
 * (lam = 0 only when n_lambda = 1), in fp64.  arg (may be NULL) receives
 * (i, j, l) of the maximiser, the first in (i, j, l) order among equal values.
 * Each form's CDF is a convolution integral evaluated by composite
 * Gauss-Legendre quadrature (16 panels of 16 nodes) with regularised incomplete
 * gamma functions; about 1e-12 absolute.  x, best, arg: device.  Limits:
 * 1 <= nx <= 65535, k >= 1, 2 <= d, k * d < 2^31, 1 <= n_lambda <= 4096.
 * Workspace: dprc_envelope_middle_workspace() bytes. */
size_t dprc_envelope_middle_workspace(int32_t nx, int32_t d, int32_t n_lambda);
dprc_status dprc_envelope_middle(const double* x, int32_t nx, int32_t k, int32_t d, int32_t n_lambda,
                                 double* best, int32_t* arg, void* ws, size_t ws_bytes,
                                 hipStream_t stream);

/* out[e] = P(chi^2(dof) <= x[e] * scale) for e < n (the extremal parts of the
 * envelope: dof = k, scale = k for the single coordinate; dof = scale = k d for
 * uniform weights).  dof > 0, scale > 0; x, out: device, fp64. */
dprc_status dprc_chi2_cdf(const double* x, int64_t n, double dof, double scale, double* out,
                          hipStream_t stream);

/* ---- privacy accountant (appendix: Algorithm accounting) ---------------------------
 * The accountant for DP-SGD-RC runs Poisson-subsampled Gaussian steps whose
 * effective scale a = 1/sqrt(Y) is averaged over the envelope law of Y, and
 * composes their privacy-loss distributions (PLD).  All arrays are fp64, device.
 *
 * dprc_envelope_bins: the envelope law as bins.  F[0..n_bins] holds the envelope
 * CDF at y_j = y_min + j (y_max - y_min) / n_bins; the CDF is made monotone by a
 * running maximum and clipped to [0, 1], w[j] = its increment over bin j (clamped
 * at zero) divided by the sum of the increments, ybar[j] = the bin's midpoint.  A
 * CDF with no increase on the range gives NaN weights.  n_bins >= 1, y_max > y_min.
 *
 * dprc_pld_step: one step's PLD on the cell-centred grid t_j = (j - n_half + 1) h,
 * j < 2 n_half - 1 (q, normalised with q_inf to total one), from the survival
 * function S(t) = P(L > t) at the cuts (c - n_half + 1/2) h, c < 2 n_half:
 *   S(t) = p betabar(t + s(t)) + (1 - p) alpha(t + s(t)),
 *   s(t) = log(1/p - (1 - p)/p e^-t), for t > log(1 - p); S = 1 at and below it,
 *   alpha(u) = sum_i w_i Phi(-u/mu_i - mu_i/2), betabar(u) = sum_i w_i Phi(-u/mu_i + mu_i/2),
 *   mu_i = 1 / (sigma sqrt(ybar_i))   (n_bins = 0: one term, w = 1, mu = 1/sigma).
 * q_j = S(cut j) - S(cut j + 1) clamped at zero; the mass below the first cut
 * joins q_0 and S at the last cut is the atom q_inf[0] at +infinity.  sigma > 0,
 * 0 < p <= 1, h > 0.  Workspace: dprc_pld_step_workspace(n_half) bytes (S).
 *
 * dprc_pld_fold: the composition of two PLDs on the same grid of L cells (L odd)
 * with atoms *ainf and *binf, given r[0 .. 2L - 2], their linear convolution
 * (r[j] sits at cell j - (L - 1)/2 of the result grid): negatives clipped; the
 * L centred cells kept, the mass below them added to the lowest one; the atom
 * becomes 1 - (1 - ainf)(1 - binf) plus the mass above them, rescaled with the
 * cells so that the total stays one.  q [L] and q_inf [1] must not overlap r.
 *
 * dprc_pld_delta: delta[e] = sum over t_j >= eps[e] of q_j (1 - e^(eps[e] - t_j))
 * + q_inf[0], clipped to [0, 1], t_j = (j - (L - 1)/2) h, for 1 <= n_eps <= 65535.
 */
dprc_status dprc_envelope_bins(const double* F, int32_t n_bins, double y_min, double y_max, double* ybar,
                               double* w, hipStream_t stream);
size_t dprc_pld_step_workspace(int64_t n_half);
dprc_status dprc_pld_step(double sigma, double p, double h, int64_t n_half, const double* ybar,
                          const double* w, int32_t n_bins, double* q, double* q_inf, void* ws,
                          size_t ws_bytes, hipStream_t stream);
dprc_status dprc_pld_fold(const double* r, int64_t L, const double* ainf, const double* binf, double* q,
                          double* q_inf, hipStream_t stream);
dprc_status dprc_pld_delta(const double* q, int64_t L, double h, const double* q_inf, const double* eps,
                           int32_t n_eps, double* delta, hipStream_t stream);

/* ---- probe bits (verification) -------------------------------------------------
 * out[j*ceil(m/32) + w] = packed probe word w of column j (k columns), bits of
 * rows >= m cleared.  probe selects the family; for HADAMARD, seed, layer_id
 * and stream_id are ignored.  Device out. */
dprc_status dprc_probe_bits(dprc_probe probe, uint64_t seed, uint32_t layer_id,
                            uint32_t stream_id, int64_t m, int32_t k, uint32_t* out,
                            hipStream_t stream);

/* ---- Gaussian probe values (verification) ----------------------------------------
 * out[j*m + u] = the GAUSSIAN probe entry (u, j) in fp32, u < m, j < k (k in
 * [1, 256]).  Device out. */
dprc_status dprc_probe_gaussian(uint64_t seed, uint32_t layer_id, int64_t m, int32_t k, float* out,
                                hipStream_t stream);

/* ---- per-launch timing (diagnostics, for profilers and benchmarks) ------------
 * While `events` is non-NULL, every kernel that a dprc call enqueues from THIS
 * host thread is launched with hipExtLaunchKernelGGL and start/stop events that
 * the dispatch itself stamps (no extra packets): launch j (counted from this
 * call) uses events[2j] (start) and events[2j+1] (stop),
 * kinds[j] (if kinds is non-NULL) receives its dprc_kernel_kind, and the host
 * integer *count is advanced; recording stops once *count reaches `capacity`
 * (the events array must hold 2*capacity created events).  *count is reset
 * to 0 here.  events == NULL switches the hook off.  The state is per host
 * thread and holds the caller's pointers until switched off. */
typedef enum {
  DPRC_KERNEL_PROJECT = 1,            /* Y = X Z (bf16 matrix cores)          */
  DPRC_KERNEL_TOKEN_REDUCE = 2,       /* X'^T Y, estimate or store            */
  DPRC_KERNEL_QR = 3,                 /* Hutch++ QR of 128-row blocks of O S  */
  DPRC_KERNEL_HUTCHPP_FINAL = 4,      /* Hutch++ V = W_P - U Q^T P, estimate  */
  DPRC_KERNEL_CLIP_SCALE = 5,
  DPRC_KERNEL_ACCUMULATE = 6,         /* clipped accumulation GEMM            */
  DPRC_KERNEL_SPLITK_REDUCE = 7,
  DPRC_KERNEL_NOISE = 8,
  DPRC_KERNEL_PROBE_BITS = 9,
  DPRC_KERNEL_PROJECT_F32 = 10,
  DPRC_KERNEL_TOKEN_REDUCE_F32 = 11,
  DPRC_KERNEL_SAMPLE_SQ = 12,
  DPRC_KERNEL_ACCUMULATE_F32 = 13,
  DPRC_KERNEL_TOKEN_SPLITS = 14,      /* sum of token splits per tile          */
  DPRC_KERNEL_SAMPLE_SUM = 15,        /* per-sample sum of tile squares         */
  DPRC_KERNEL_QR_COMBINE = 16,        /* QR of stacked block R factors (upper tree levels) */
  DPRC_KERNEL_QR_EXPAND = 17,         /* rows of Q per tree level; Q^T P at the first */
  DPRC_KERNEL_HUTCHPP_SUM = 18,       /* per-sample Hutch++ estimate            */
  DPRC_KERNEL_PROBE_GAUSS = 19,       /* Gaussian probe columns                  */
  DPRC_KERNEL_ADAMW = 20,             /* private AdamW step                      */
  DPRC_KERNEL_ENVELOPE = 21,          /* MiddleRegionCDF candidates and reduction */
  DPRC_KERNEL_CHI2_CDF = 22,          /* chi-squared CDF values                  */
  DPRC_KERNEL_PLD = 23                /* accountant: bins, step PLD, fold, delta */
} dprc_kernel_kind;
dprc_status dprc_trace_launches(hipEvent_t* events, int32_t* kinds, int32_t capacity,
                                int32_t* count);

const char* dprc_status_string(dprc_status status);
const char* dprc_version(void);

#ifdef __cplusplus
}
#endif
#endif /* DPRC_H */
