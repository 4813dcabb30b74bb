/*
 * prm.h -- C ABI of the Periodic Row-wise Muon (PRM) optimizer step for AMD
 * MI355X (gfx950).  Library: libprm.so.
 *
 * The operation is Alg. 1 ("Periodic Row-wise Muon") of "Scaling Muon for
 * Diffusion Transformers", applied to a fixed list of 2-D weight matrices on one
 * GPU.  For every matrix W (m x n) with gradient G and momentum M, step t does
 *
 *   M <- beta*M + G                     (heavy-ball; optional dampening
 *                                        M <- beta*M + (1-beta)*G)
 *   U  = M, or G + beta*M with Nesterov
 *   rho_t = 1[t mod K = 0]              (Sec. 3.3, eq. periodic-direction)
 *   U~ = U if m <= n else U^T           (orientation, Sec. 3.1; r = min, c = max)
 *   D~ = NS5(U~)                 if rho_t   (eq. app-ns-recurrence, five iterations of
 *                                            G = XX^T, B = bG + cG^2, X <- aX + BX on
 *                                            X0 = U~/(||U~||_F + eps_ns))
 *      = gamma * RowNorm_eps(U~) otherwise  (eq. rownorm: row / max(||row||_2, eps))
 *   D  = s(W) * O^{-1}(D~)
 *   W <- (1 - eta*lambda)*W - eta*D     (eq. periodic-direction; Alg. 1)
 *
 * Numerics: momentum, RowNorm and the parameter write are fp32; NS5 runs as
 * bf16-input / fp32-accumulate matrix products (MFMA), with the diagonals of
 * G and B carried in fp32 and only their off-diagonal parts rounded to bf16
 * for the next product; W is rounded to its storage type (RNE).
 *
 * Memory: every matrix buffer is a DEVICE pointer to a contiguous row-major
 * m x n array owned by the caller.  W and M are updated in place, G is only
 * read.  Buffers of different matrices, and W / G / M of one matrix, must not
 * overlap.  Pointer arrays (the `const*` arguments) are HOST arrays read
 * during the call only.  The library owns its workspace (allocated by
 * prm_init, freed by prm_destroy) and never frees caller memory.
 *
 * Streams: prm_step and prm_step_debug only enqueue work on the stream given
 * to prm_init (a hipStream_t; NULL = the default stream) and never wait for
 * the GPU, except that a call whose pointer arrays differ from the previous
 * call's waits for that previous call's small pointer-table upload to finish.
 *
 * Errors: every entry point returns PRM_OK (0) or a negative PRM_E* code and
 * stores a message readable with prm_last_error() (per thread).  Arguments are
 * validated before anything is enqueued, so a failed call has no effect on
 * the caller's buffers.  Buffer pointers that differ from the previous call's
 * are checked with hipPointerGetAttributes: host memory, or memory of another
 * device than the context's, is refused with PRM_EINVAL (a kernel reading it
 * would fault).  A context is not thread-safe; separate contexts are.
 */
#ifndef PRM_H
#define PRM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PRM_OK 0
#define PRM_EINVAL (-1)  /* bad argument: K < 1, beta outside [0,1), shape < 1, NULL, host pointer, t < 0, ... */
#define PRM_EDTYPE (-2)  /* unsupported storage type */
#define PRM_EALIGN (-3)  /* a device pointer is not 16-byte aligned */
#define PRM_ENOMEM (-4)  /* workspace does not fit the budget or the device */
#define PRM_EHIP   (-5)  /* a HIP runtime call failed; the message carries its error string */

typedef enum prm_dtype { PRM_F32 = 0, PRM_BF16 = 1 } prm_dtype;

/* Shape scale s(W) of eq. (periodic-direction); the paper names it a
 * scale that depends on the matrix shape, without a formula. */
typedef enum prm_scale_mode {
  PRM_SCALE_ONE = 0,          /* s = 1 */
  PRM_SCALE_SQRT_ASPECT = 1,  /* s = sqrt(max(1, m/n)) (default) */
  PRM_SCALE_RMS_0P2 = 2       /* s = 0.2 * sqrt(max(m, n)) */
} prm_scale_mode;

typedef struct prm_config {
  int32_t K;             /* refresh period, >= 1 (Sec. 3.3) */
  float beta;            /* momentum, in [0, 1) */
  float lr;              /* eta used when prm_step gets lr < 0; >= 0 */
  float wd;              /* decoupled weight decay lambda, >= 0 */
  float gamma;           /* RowNorm multiplier (> 0); scales only the RowNorm branch */
  float eps_rownorm;     /* RowNorm clamp, > 0 (applied after the square root) */
  float eps_ns;          /* NS input normalization X0 = U/(||U||_F + eps_ns), > 0
                            (a zero momentum then gives a zero direction) */
  float ns_a, ns_b, ns_c;/* quintic coefficients (3.4445, -4.7750, 2.0315) */
  int32_t nesterov;      /* 0: U = M;  1: U = G + beta*M (after the momentum update) */
  int32_t ema_dampening; /* 0: M = beta*M + G;  1: M = beta*M + (1-beta)*G */
  int32_t scale_mode;    /* prm_scale_mode */
  int32_t param_dtype;   /* prm_dtype of W (momentum is always fp32) */
  int32_t grad_dtype;    /* prm_dtype of G */
  int32_t never_refresh; /* ablation: RowNorm on every step (K ignored) */
  int32_t gamma_on_refresh; /* ablation: gamma also scales the NS5 direction */
  int32_t ns_plain;      /* 0 (default): matrices with c >= 2r (oriented) evaluate NS5
                            through the factored form described at prm_step; 1: the
                            five iterations as written for every matrix */
  int32_t ns_precise;    /* 0 (default); 1: the five iterations as written, with every
                            iterate carried as two bf16 parts (hi + lo, 16 mantissa bits):
                            the Gram sums X_hi X_hi^T + X_hi X_lo^T + X_lo X_hi^T and the
                            apply takes both parts.  It follows the exact NS5 map within
                            2e-2 also for momenta of low numerical rank, which the bf16
                            iterate amplifies in its smallest directions,
                            at 3.3x the default's refresh time at DiT-4B (2.2x the plain
                            path's) and twice the iterate workspace.  Not available in
                            prm_step_noalloc. */
  uint64_t workspace_budget_bytes; /* NS5 workspace cap; 0 = automatic (48 GiB) */
} prm_config;

typedef struct prm_ctx prm_ctx; /* opaque */

/* Fill *cfg with the paper's defaults: K = 3, beta = 0.95, lr = 5e-3,
 * wd = 0.01, gamma = 0.15 (optimizer hyperparameter table), eps_rownorm = 1e-8,
 * eps_ns = 1e-7, (a,b,c) = (3.4445, -4.7750, 2.0315), heavy-ball momentum,
 * s = sqrt(max(1, m/n)), bf16 W and G. */
void prm_config_default(prm_config* cfg);

/* Create a context for n_mats matrices of shapes rows[i] x cols[i] (host
 * arrays, each in [1, 2^24]; n_mats >= 0): the fixed set W_M of 2-D weight
 * matrices that Alg. 1 loops over, with the hyperparameters of eq.
 * (periodic-direction) in cfg (K, beta, lr, wd, gamma, ...).  Validates cfg,
 * groups the matrices by oriented NS5 shape, plans and allocates the device
 * workspace (hipMalloc on the current device) and records `hip_stream` for
 * later calls.  On success *out owns the workspace until prm_destroy.
 * Errors: PRM_EINVAL / PRM_EDTYPE for a bad cfg or shape, PRM_ENOMEM when the
 * workspace does not fit, PRM_EHIP for a failed HIP call; *out is then NULL
 * and nothing stays allocated. */
int prm_init(prm_ctx** out, int32_t n_mats, const int64_t* rows, const int64_t* cols,
             const prm_config* cfg, void* hip_stream);

/* One optimizer step t (0-based, >= 0) over every matrix: the body of the
 * loop over t in Alg. 1 (momentum update, rho_t of eq. periodic-direction,
 * NS5 refresh or gamma RowNorm, shape scale, decoupled weight decay and the
 * parameter write), enqueued on the context's stream.
 * NS5 (eq. app-ns-recurrence) is evaluated in one of two exact forms.  For a
 * matrix whose oriented shape has c >= 2r (unless cfg.ns_plain or cfg.ns_precise): every B_j
 * is a polynomial in A_0, so the factors P_j = aI + B_j commute, and the
 * step computes X_2 = (P_1 P_0) X_0, A_1 = P_0^2 A_0, A_3 = P_2^2 A_2,
 * A_4 = P_3^2 A_3 and X_5 = (P_4 P_3 P_2) X_2 with r x r products, forming
 * the Gram matrix X X^T only at j = 0 and 2 (4 r^2 c + 14 r^3 multiply-adds
 * instead of 10 r^2 c + 5 r^3, and two bf16 roundings of the iterate instead
 * of five).  Square and nearly square matrices run the five iterations.
 * params[i]: W (param_dtype), grads[i]: G (grad_dtype),
 * momentum[i]: M (fp32); all device pointers, 16-byte aligned.  lr < 0 uses
 * cfg->lr.  *did_refresh (nullable) receives rho_t, computed on the host.
 * Runs on the device the context was created on; the caller's current device
 * is restored before returning.  A call whose pointer arrays equal the
 * previous call's enqueues kernels only (no allocation, memset or upload), so
 * it may be captured into a HIP graph and replayed for the same rho_t. */
int prm_step(prm_ctx* ctx, void* const* params, const void* const* grads,
             float* const* momentum, int64_t step, float lr, int32_t* did_refresh);

/* prm_step that also writes the direction D = s(W) * O^{-1}(D~) of eq.
 * (periodic-direction) (fp32, m x n, row-major, device, caller-owned) into
 * direction_out[i] for every matrix whose entry is not NULL (NULL: that
 * matrix's direction is not written).  W and M end bitwise as with prm_step.
 * Parity checking only. */
int prm_step_debug(prm_ctx* ctx, void* const* params, const void* const* grads,
                   float* const* momentum, int64_t step, float lr, int32_t* did_refresh,
                   float* const* direction_out);

/* The refresh indicator rho_t of the context's schedule (Sec. 3.3, eq.
 * periodic-direction; Alg. 1): 1[t mod K = 0] for 0-based t, or 0 for every t
 * with cfg.never_refresh.  Returns 1 or 0 (what prm_step would report in
 * *did_refresh), or PRM_EINVAL for a NULL ctx or t < 0.  Host only. */
int prm_is_refresh(const prm_ctx* ctx, int64_t step);

/* Device bytes the context holds for the step of Alg. 1 (NS5 workspace,
 * tall-matrix statistics of eq. sharded-tall-rownorm and small per-matrix
 * scalars; not the descriptor and work-list tables) in *out_bytes.
 * PRM_EINVAL for a NULL argument.  Host only. */
int prm_workspace_bytes(const prm_ctx* ctx, size_t* out_bytes);

/* The same two quantities without a context, for planning: rho_t =
 * 1[t mod K = 0] (PRM_EINVAL for K < 1 or t < 0), and the device bytes
 * prm_init would allocate for these shapes and cfg (same validation and error
 * codes as prm_init; no device call). */
int prm_schedule_is_refresh(int64_t step, int32_t K);
int prm_plan_workspace_bytes(int32_t n_mats, const int64_t* rows, const int64_t* cols,
                             const prm_config* cfg, uint64_t* out_bytes);

/* Per-kernel-class timing on the context's stream, for measurement.
 * prm_profile_enable(ctx, 1) makes later steps record a HIP event pair around
 * every kernel launch (on the same stream); prm_profile_read synchronizes the
 * stream and fills out[0 .. min(n, PRM_NUM_KERNEL_CLASSES)) with, per kernel
 * class, the launch count, total GPU milliseconds, and the algorithmic bytes
 * and FLOPs of those launches, then clears the counters.  Classes, in order:
 * rw_wide, rw_generic, rw_tall_stats, rw_tall_finalize, rw_tall_apply,
 * ns_prologue, ns_alpha, ns_gram, ns_poly, ns_apply, ns_sprod.  Algorithmic
 * bytes count each element of G, M and W once per read or write the method
 * needs (the tall-matrix re-read of M is not counted).  Algorithmic FLOPs are
 * 2 x the multiply-adds of the product a launch forms, per matrix: 2r^2c
 * (Gram, apply: r x r times r x c), 2r^3 (square, and the r x r split
 * products of the factored form).  Executed FLOPs are what the matrix cores
 * actually run: padded 256 x 256 tiles, only the upper tiles of symmetric
 * results, and the diagonal-term MFMAs of the apply. */
#define PRM_NUM_KERNEL_CLASSES 11
typedef struct prm_kernel_stats {
  char name[32];
  int64_t launches;
  double total_ms;
  double alg_bytes;
  double alg_flops;
  double exec_flops;
} prm_kernel_stats;
int prm_profile_enable(prm_ctx* ctx, int32_t enable);
int prm_profile_read(prm_ctx* ctx, prm_kernel_stats* out, int32_t n);

/* Free the workspace (after synchronizing the context's stream) and the
 * context.  NULL is a no-op. */
int prm_destroy(prm_ctx* ctx);

/* ---- Auxiliary AdamW group ------------------------------------------------
 * The paper updates every parameter that is not a 2-D hidden weight matrix
 * (biases, normalization scales and shifts, embedders) with AdamW and
 * decoupled weight decay (Sec. 2, Muon setup; App. "Optimizer and Training
 * Hyperparameters": aux LR 1e-4, betas (0.9, 0.95), eps 1e-8, weight decay
 * 0.01).  This context applies that update to a fixed list of flat tensors in
 * one fused launch.  Per element, in fp32, for the t-th update (t >= 1):
 *
 *   m <- beta1*m + (1-beta1)*g          v <- beta2*v + (1-beta2)*g^2
 *   p <- p - lr*( (m/(1-beta1^t)) / (sqrt(v/(1-beta2^t)) + eps) + wd*p )
 *
 * and p is rounded to its storage type (RNE).  Tensors are DEVICE pointers to
 * contiguous arrays of numel[i] elements owned by the caller: p (param_dtype)
 * and the moments m, v (fp32) are updated in place, g (grad_dtype) is only
 * read; they must be 16-byte aligned and must not overlap.  Same stream, device and
 * error rules as prm_step (validation before anything is enqueued; the call
 * only enqueues, except that new pointer arrays wait for the previous call's
 * small pointer-table upload). */
typedef struct prm_adamw_config {
  float lr;              /* used when prm_adamw_step gets lr < 0; >= 0 */
  float beta1, beta2;    /* in [0, 1) */
  float eps;             /* > 0, added to the square root */
  float wd;              /* decoupled weight decay, >= 0 */
  int32_t param_dtype;   /* prm_dtype of p */
  int32_t grad_dtype;    /* prm_dtype of g */
  int32_t reserved;
} prm_adamw_config;

typedef struct prm_adamw_ctx prm_adamw_ctx; /* opaque */

/* Fill *cfg with the paper's aux-AdamW settings: lr = 1e-4, betas = (0.9,
 * 0.95), eps = 1e-8, wd = 0.01, bf16 p and g. */
void prm_adamw_config_default(prm_adamw_config* cfg);

/* Create a context for n_tensors >= 0 flat tensors of numel[i] >= 0 elements
 * (host array).  Allocates the chunk table (one entry per 2048 elements) and
 * the pointer table on the current device and records `hip_stream`. */
int prm_adamw_init(prm_adamw_ctx** out, int32_t n_tensors, const int64_t* numel,
                   const prm_adamw_config* cfg, void* hip_stream);

/* The t-th AdamW update (t >= 1: the number of updates so far, this one
 * included) of every tensor, enqueued on the context's stream.  lr < 0 uses
 * cfg->lr.  Pointers of empty tensors may be NULL. */
int prm_adamw_step(prm_adamw_ctx* ctx, void* const* params, const void* const* grads,
                   float* const* exp_avg, float* const* exp_avg_sq, int64_t t, float lr);

/* Free the context (after synchronizing its stream).  NULL is a no-op. */
int prm_adamw_destroy(prm_adamw_ctx* ctx);

/* Calibration probes (not part of the optimizer step).  They measure the
 * ceilings the step's kernels are compared against, on the device current on
 * the calling thread, with the instructions the step uses; each call
 * synchronizes `hip_stream` and allocates and frees its own device buffers.
 *
 * prm_peak_mfma: sustained bf16 MFMA rate.  Every wave runs 8 independent
 * 32x32x16 accumulator chains for `iters` iterations (1 <= iters <= 2^24; 16
 * waves per compute unit, no memory traffic) on pseudo-random operands that
 * change from one MFMA to the next, as a GEMM's do.  *tflops = executed FLOPs over
 * the HIP-event time; *clock_ghz = the shader clock during the loop (shader
 * cycles over 100 MHz reference ticks), which drops below the nominal
 * 2.4 GHz when the power limit is reached.
 *
 * prm_peak_hbm: HBM stream rates over two buffers of `bytes` bytes each
 * (>= 1 MiB, a multiple of 16): a read-only pass, a write-only pass and a copy,
 * with one 16-byte nontemporal access per thread, and a pass with the
 * row-wise step's element traffic (bf16 gradient, fp32 momentum and bf16
 * weight read, momentum and weight written: 14 bytes per element, bytes/4
 * elements, each access instruction contiguous across a wave).  Each rate is
 * the best of three timed repetitions, in GB/s of bytes moved (reads plus
 * writes).
 *
 * Errors: PRM_EINVAL for NULL outputs or out-of-range sizes, PRM_ENOMEM when
 * the buffers cannot be allocated, PRM_EHIP for a failed HIP call. */
int prm_peak_mfma(void* hip_stream, int32_t iters, double* tflops, double* clock_ghz);
int prm_peak_hbm(void* hip_stream, uint64_t bytes, double* read_gbs, double* write_gbs, double* copy_gbs,
                 double* rowwise_gbs);

/* ---- Allocation-free step ------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  One
 * optimizer step t of ONE matrix (rows x cols, W param, G grad, M momentum:
 * device pointers, 16-byte aligned, as in prm_step) without a context: the
 * same kernels as prm_step on a context created for that matrix alone, with
 * bitwise the same W and M.  Nothing is allocated (no hipMalloc, hipFree or
 * allocating library call) and nothing waits for the GPU: after validation the
 * call enqueues a small set-up kernel and the step's kernels on `hip_stream`,
 * on the CURRENT device.  *did_refresh (nullable) receives rho_t.
 *
 * Scratch: the descriptor, work lists and workspace (the NS5 iterates and Gram
 * factors on refresh steps, a tall matrix's column statistics on row-wise
 * steps) live in one static device array of PRM_NOALLOC_SCRATCH_BYTES per GPU,
 * which the library holds on every GPU it runs on until the process ends.  A
 * step that needs more is refused with PRM_ENOMEM before anything is enqueued
 * (a refresh step needs 4 rp cp + 8 rp^2 bytes in the factored form, c >= 2r,
 * and 4 rp cp + 4 rp^2 otherwise, with rp x cp the oriented shape padded to
 * 256: 3072 x 12288 and 5120 x 5120 fit, 3072 x 18432 does not; row-wise steps of wide
 * matrices need no workspace).  Every call on one GPU uses the same array:
 * calls that overlap in time on one GPU (on other streams or threads) RACE
 * and give wrong results; calls ordered on one stream are safe, and every byte
 * a kernel reads from the array is written earlier in the same call.
 * cfg->workspace_budget_bytes is ignored.  Errors as in prm_init / prm_step. */
#define PRM_NOALLOC_SCRATCH_BYTES (256ull << 20)
int prm_step_noalloc(const prm_config* cfg, int64_t rows, int64_t cols, void* param, const void* grad,
                     float* momentum, int64_t step, float lr, int32_t* did_refresh, void* hip_stream);

/* Message of the last failing call on this thread ("" if none). */
const char* prm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* PRM_H */
