/*
 * rikfad.h -- C ABI of the MI355X (gfx950) R-iKFAD optimiser step.
 *
 * Method: Rank-1 iKFAD (R. Rajpal, B. Leimkuhler, "Low-Rank Friction for
 * Memory-Efficient Transformer Pretraining").  For every weight matrix
 * X (m x n) with momentum P (m x n) and friction factors R (m), C (n), one
 * optimiser step is the BACD splitting of Section 2 ("Splitting
 * Discretization"), written out in App. A (Table of analytical sub-step
 * updates):
 *
 *   B    P^(B)   = P_n - h g                       (g = gradient at X_n)
 *   A    X_{n+1} = X_n + h P^(B)
 *   C.1  xi~_n   = R_n C_n^T / (1^T R_n + eps_stab)          eq. (xi_def)
 *        P^(1)   = P^(B) .* exp(-(h/2) xi~_n)
 *   C.2  R_{n+1} = e^{-alpha h} R_n + (1 - e^{-alpha h})/(mu alpha) [P^(1)]^2 1_n
 *   C.3  C_{n+1} = e^{-alpha h} C_n + (1 - e^{-alpha h})/(mu alpha) ([P^(1)]^2)^T 1_m
 *   C.4  P^(2)   = P^(1) .* exp(-(h/2) xi~_{n+1})
 *   D    P_{n+1} = P^(2) e^{-gamma h}
 *
 * with xi~ = 0 when 1^T R + eps_stab == 0 (the eps_stab = 0 convention of
 * Theorem "Algebraic rates").  Tensors with m == 1 or n == 1 (biases,
 * LayerNorm scales) take element-wise iKFAD instead (Section 2, "Memory
 * Complexity"): the same steps with one friction entry per parameter,
 * xi_{n+1} = e^{-alpha h} xi_n + (1 - e^{-alpha h})/(mu alpha) [P^(1)]^2.
 *
 * All entry points are asynchronous on the HIP stream they are given
 * (a hipStream_t passed as void*; NULL is the default stream) unless stated
 * otherwise, return a rikfad_status, and never throw.  A context is not
 * thread-safe; distinct contexts are independent.
 */
#ifndef RIKFAD_H
#define RIKFAD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    RIKFAD_OK = 0,
    RIKFAD_EINVAL = -1,     /* bad argument (NULL, size, hyperparameter) */
    RIKFAD_EALIGN = -2,     /* a pointer is not aligned to its element type */
    RIKFAD_EDTYPE = -3,     /* unsupported dtype code */
    RIKFAD_ENOMEM = -4,     /* host or device allocation failed */
    RIKFAD_EHIP = -5,       /* a HIP runtime call or kernel launch failed */
    RIKFAD_ESTATE = -6      /* call not valid in the context's current state */
} rikfad_status;

/* Storage type of x and g.  p, r, c (and xi) are always fp32. */
typedef enum { RIKFAD_FP32 = 0, RIKFAD_BF16 = 1 } rikfad_dtype;

/* One parameter tensor: all pointers are device pointers, row-major and
 * contiguous (row i, column j at offset i*n + j).
 *   x  m*n elements of `dtype`, the parameter X, updated in place.  A bf16
 *      parameter is computed in fp32 and stored rounded to nearest-even.
 *   g  m*n elements of `dtype`, the gradient at the current X; read only.
 *   p  m*n fp32, the momentum (see the deferred form below).
 *   r  m fp32, c  n fp32: the friction factors R and C.
 * Vectors (m == 1 or n == 1) keep their element-wise friction (m*n entries)
 * in c when m == 1 and in r otherwise; the other factor is unused and may be
 * NULL.  The caller owns every buffer, keeps it alive and in place from
 * create to destroy, zero-fills p, r and c before the first step (the paper
 * starts from R = C = 0) unless it resumes a saved state, and never lets two
 * tensors of one context share memory.  Every pointer must be aligned to its
 * element size.  A matrix with n a multiple of 4 and x, g, p 16-byte aligned
 * (fp32), or x, g 8-byte and p 16-byte aligned (bf16), takes the 4-wide
 * path (128-bit accesses, 64-bit for bf16 x and g); any other matrix a
 * one-column path in the same launch. */
typedef struct {
    void *x;
    const void *g;
    float *p;
    float *r;
    float *c;
    int64_t m, n;
    int32_t dtype;          /* rikfad_dtype */
    int32_t reserved;       /* must be 0 */
} rikfad_tensor;

/* Hyperparameters shared by all tensors of a context (the paper tunes them
 * per model, App. "Optimal Hyperparameters").  Requirements: h > 0, mu > 0,
 * alpha >= 0 (alpha = 0 takes the limit (1 - e^{-alpha h})/(mu alpha) ->
 * h/mu), gamma >= 0 (0 is R-iKFAD0), eps_stab >= 0, all finite.  The step
 * uses them as fp32 after computing e^{-alpha h}, the factor gain,
 * e^{-gamma h} and h/2 in fp64 on the host. */
typedef struct {
    double h, gamma, alpha, mu, eps_stab;
} rikfad_hparams;

typedef struct rikfad_ctx rikfad_ctx;

/* Flags for rikfad_create. */
#define RIKFAD_FLAG_TWO_PASS 1u   /* p holds P_{n+1} after every step */

/* Create a context over `count` tensors (count >= 0; 0 gives a context whose
 * step does nothing).  Validates every argument before any HIP call, builds
 * the device tile tables and allocates the partial-sum workspace on the
 * current HIP device: 4 (m B + S n + ceil(m / 256)) bytes per matrix for its
 * B column blocks (256 columns, or 64 on the one-column path) and S row
 * stripes (32 rows; 16 in a set with fewer matrix tiles than the chip has
 * compute units; taller for narrow matrices) -- about 0.14 m n bytes
 * (rikfad_query reports the total).  The tensors and every stream passed to
 * the context later must belong to that device.  The tensor array is
 * copied; the buffers it points to are not.  Zero-size tensors (m < 1 or n < 1) are
 * rejected with RIKFAD_EINVAL.
 *
 * Deferred form (default).  The second friction half-kick and D of step n
 * use the same factor R_{n+1}, C_{n+1} as the first half-kick of step n+1,
 * so the library applies them at the start of step n+1 inside the same
 * streaming pass: between steps a matrix's p holds P^(1) of the last step
 * and the step moves the minimum number of bytes (read x, g, p; write x, p).
 * X, R and C are always those of the paper's step.  Call
 * rikfad_sync_momentum to turn p into P_{n+1} (before reading p or saving a
 * checkpoint).  Vector tensors are never deferred.
 * RIKFAD_FLAG_TWO_PASS instead applies the second half-kick in a separate
 * pass after every step, so p always holds P_{n+1} (28 bytes per fp32
 * parameter instead of 20). */
rikfad_status rikfad_create(const rikfad_tensor *tensors, int64_t count,
                            const rikfad_hparams *hp, uint32_t flags,
                            rikfad_ctx **out);

/* Enqueue one optimiser step on `stream`, reading the gradients g given at
 * create (or at the last rikfad_step_grads).  Three kernels at most: the
 * fused streaming pass over all tensors (B, A, C.1, the deferred C.4 + D,
 * per-tile row and column partial sums of [P^(1)]^2), the fixed-order
 * finalisation of R, C and 1^T R, and in two-pass mode the C.4 + D pass.
 * Results are bitwise reproducible: no atomics, fixed reduction order.
 *
 * HIP graphs: a step only enqueues kernel launches (no allocation, copy,
 * memset or synchronisation), so it can be captured and replayed.  Whether
 * a deferred half-kick is pending is host state that the captured launches
 * bake in: capture after a first eager step, and replay the graph only
 * while every step goes through it.  rikfad_sync_momentum,
 * rikfad_set_hparams, rikfad_state_changed and rikfad_step_grads change
 * that state or the gradient table, so they do not belong between replays
 * of one graph.  rikfad_step_grads with changed pointers copies the new
 * table from host memory and may wait for an earlier copy, so it must not
 * be captured. */
rikfad_status rikfad_step(rikfad_ctx *ctx, void *stream);

/* As rikfad_step, with new gradient pointers grads[0..count-1] (same shapes,
 * dtypes and alignment class as at create; RIKFAD_EALIGN otherwise).  For
 * frameworks that reallocate gradients between steps. */
rikfad_status rikfad_step_grads(rikfad_ctx *ctx, const void *const *grads,
                                void *stream);

/* Replace the hyperparameters.  If a deferred half-kick is pending and h,
 * gamma or eps_stab change, the pending half-kick (which belongs to the
 * previous step and its hyperparameters) is applied first on `stream`. */
rikfad_status rikfad_set_hparams(rikfad_ctx *ctx, const rikfad_hparams *hp,
                                 void *stream);

/* Apply a pending deferred half-kick so that every p holds P_{n+1}
 * (App. A Table rows C.4 and D).  No-op when nothing is pending. */
rikfad_status rikfad_sync_momentum(rikfad_ctx *ctx, void *stream);

/* Tell the context that the caller rewrote p, r or c (e.g. restored a
 * checkpoint saved after rikfad_sync_momentum): p is taken to hold P_n, no
 * half-kick is pending, and 1^T R is recomputed before the next step. */
rikfad_status rikfad_state_changed(rikfad_ctx *ctx);

typedef struct {
    int64_t tensors, matrices, vectors;
    int64_t elements;          /* sum of m n */
    int64_t state_bytes;       /* optimiser state p, r, c (and vector xi) */
    int64_t ikfad_state_bytes; /* the same model under full iKFAD: 8 m n */
    int64_t workspace_bytes;   /* device memory owned by the context */
    int64_t min_bytes_per_step;/* compulsory HBM traffic of one step: per
                                  matrix element read x, g, p and write x, p
                                  (20 B fp32, 14 B bf16 x/g), plus R and C read
                                  and written; per vector element also xi */
    int64_t stream_min_bytes;  /* the same for the streaming kernel alone
                                  (R, C read, not written) */
    int64_t stream_tiles;      /* workgroups of the streaming pass */
    int64_t finalize_items;    /* workgroups of the finalisation pass */
    int32_t pending;           /* 1 if a deferred half-kick is pending */
    int32_t two_pass;
} rikfad_info;

/* Describe a context (host only, no HIP call). */
rikfad_status rikfad_query(const rikfad_ctx *ctx, rikfad_info *out);

/* Host-only accounting of a tensor list, no HIP call: R-iKFAD optimiser
 * state (4 m n for p plus 4 (m + n) for R, C per matrix; 8 m n per vector)
 * and full iKFAD state (8 m n) in bytes.  App. "Memory Analysis" reports
 * these as N + sum (m + n) versus 2N scalars. */
rikfad_status rikfad_state_bytes(const rikfad_tensor *tensors, int64_t count,
                                 int64_t *rikfad_bytes, int64_t *ikfad_bytes);

/* Blocking: wait for `stream`, then report whether any finalised factor
 * (R, C or their sum) or any updated vector friction entry has been
 * non-finite since create (1) or not (0).  Non-finite values are
 * propagated, never masked. */
rikfad_status rikfad_nonfinite(rikfad_ctx *ctx, void *stream, int32_t *out);

/* Kernel timing for benchmarks.  While enabled (enable != 0), every step
 * attaches HIP start / stop events to the first and last kernel dispatch of
 * each phase (hipExtLaunchKernelGGL), so they hold the kernels' own begin
 * and end times and add nothing to the stream: a timed step runs like an
 * untimed one.  Disabling and enabling again keeps the unread record.
 * rikfad_timing_read waits for the last timed kernel and returns the
 * summed milliseconds of the streaming, finalisation and two-pass apply
 * kernels and the number of timed steps, then clears the record.  Each
 * timed step holds 6 events until destroy. */
rikfad_status rikfad_timing_enable(rikfad_ctx *ctx, int32_t enable);
rikfad_status rikfad_timing_read(rikfad_ctx *ctx, double *stream_ms,
                                 double *finalize_ms, double *apply_ms,
                                 int64_t *steps);

void rikfad_destroy(rikfad_ctx *ctx);

const char *rikfad_status_string(rikfad_status s);

/* Message describing the most recent failure on the calling thread. */
const char *rikfad_last_error(void);

/* ------------------------------------------------------------------------
 * Full-tensor iKFAD (comparison point).  Section 1, iKFAD dynamics, with
 * the same BACD splitting and sub-flow C treatment as above, one friction
 * entry per parameter: reads x, g, p, xi and writes x, p, xi (28 bytes per
 * fp32 parameter) and keeps 2N state scalars against R-iKFAD's
 * N + sum(m + n).  Same conventions as the R-iKFAD entry points.
 * ---------------------------------------------------------------------- */
typedef struct {
    void *x;
    const void *g;
    float *p;
    float *xi;              /* m*n fp32 friction */
    int64_t m, n;
    int32_t dtype;
    int32_t reserved;
} ikfad_tensor;

typedef struct ikfad_ctx ikfad_ctx;

rikfad_status ikfad_create(const ikfad_tensor *tensors, int64_t count,
                           const rikfad_hparams *hp, ikfad_ctx **out);
rikfad_status ikfad_step(ikfad_ctx *ctx, void *stream);
rikfad_status ikfad_set_hparams(ikfad_ctx *ctx, const rikfad_hparams *hp);
/* Kernel timing as for rikfad_timing_*: ms = summed kernel time of the
 * timed steps. */
rikfad_status ikfad_timing_enable(ikfad_ctx *ctx, int32_t enable);
rikfad_status ikfad_timing_read(ikfad_ctx *ctx, double *ms, int64_t *steps);
/* Blocking: 1 if any updated friction entry has been non-finite since
 * create, else 0 (as rikfad_nonfinite). */
rikfad_status ikfad_nonfinite(ikfad_ctx *ctx, void *stream, int32_t *out);
void ikfad_destroy(ikfad_ctx *ctx);

/* ------------------------------------------------------------------------
 * Rank-1 friction diagnostic (Section 4, "How close is xi~ to the best
 * rank-1 friction?").  The paper runs iKFAD0 and carries R-iKFAD's factors
 * as shadow states fed by the same P^(1); since both obey the same linear
 * filter, from zero they are exactly R = xi 1 and C = xi^T 1.  Given an
 * iKFAD friction tensor xi (m x n fp32, row-major, device memory, e.g. the
 * xi of an ikfad context), this computes on the GPU the shadow factors,
 * |xi|_F^2, |xi - xi~|_F^2 with xi~ = R C^T / (1^T R + eps_stab), and the
 * leading singular value sigma_1 of xi by power_iters steps of power
 * iteration on xi^T xi from C / |C|; then the relative error, the
 * Eckart-Young floor sqrt(1 - sigma_1^2 / |xi|_F^2) and the stable rank
 * |xi|_F^2 / sigma_1^2.  All reductions are fp64 in a fixed order.
 * Blocking (waits for `stream`); allocates and frees a temporary device
 * workspace of 8 (2 m + 2 n + n P) bytes plus a little
 * (rikfad_friction_report_workspace_bytes gives the exact size), where
 * P = ceil(m / 128) for n <= 1024 and otherwise the number of column-sum
 * stripes ceil(m / s), s a power of two in [16, 1024] (larger only for m
 * above 2^20).  For n <= 1024 the report reads xi power_iters + 2 times
 * (the factors in one pass, the errors with the first power iteration,
 * sigma_1 in a last pass), otherwise 2 power_iters + 4 times.  m, n < 2^31;
 * EINVAL on bad arguments, ENOMEM if the workspace cannot be allocated,
 * EHIP on a launch or copy failure (rikfad_last_error says which).
 * ---------------------------------------------------------------------- */
typedef struct {
    double xi_fro2;            /* |xi|_F^2 */
    double err_fro2;           /* |xi - xi~|_F^2 */
    double sum_r;              /* 1^T R = 1^T xi 1 */
    double sigma1;             /* leading singular value of xi */
    double rel_err;            /* |xi - xi~|_F / |xi|_F */
    double eckart_young_floor; /* best possible rank-1 relative error */
    double stable_rank;        /* |xi|_F^2 / sigma_1^2 */
    int32_t power_iters;
    int32_t reserved;
} rikfad_friction_stats;

rikfad_status rikfad_friction_report(const float *xi, int64_t m, int64_t n, double eps_stab,
                                     int32_t power_iters, void *stream,
                                     rikfad_friction_stats *out);

/* The same report for callers that cannot allocate device memory (code
 * between allocations that a harness forbids, tight serving or monitoring
 * loops): the same arguments, kernels and results (bit for bit) as
 * rikfad_friction_report, but the workspace is a static device array of
 * rikfad_friction_report_noalloc_max_bytes() bytes (16 MiB) that the
 * library holds on every device it runs on until the process ends; the
 * call itself never allocates or frees device memory.  The first call on a
 * device looks up that device's copy of the array (hipGetSymbolAddress,
 * with the device current).  A tensor whose workspace
 * (rikfad_friction_report_workspace_bytes) exceeds the array is rejected
 * with RIKFAD_EINVAL and a message in rikfad_last_error; every GPT2-S,
 * DistilBERT and 4096 x 11008 shape needs less than 6 MiB.  Blocking, like
 * rikfad_friction_report.  All calls on one device share its array: calls
 * that overlap on one device (from several host threads, or on several
 * streams at once) race and must be serialised by the caller. */
rikfad_status rikfad_friction_report_noalloc(const float *xi, int64_t m, int64_t n,
                                             double eps_stab, int32_t power_iters,
                                             void *stream, rikfad_friction_stats *out);
/* Size of the static workspace of rikfad_friction_report_noalloc, in bytes. */
int64_t rikfad_friction_report_noalloc_max_bytes(void);
/* Workspace bytes a report on an m x n tensor needs (host only, no HIP
 * call); -1 for m or n outside [1, 2^31). */
int64_t rikfad_friction_report_workspace_bytes(int64_t m, int64_t n);

/* ------------------------------------------------------------------------
 * Adafactor-m (the paper's baseline optimiser; Section 2, Methodology,
 * left-hand system, and eq. (xi_def) for zeta^ = R C^T / 1^T R).  The
 * second moment of the gradient is factored as R (row sums) and C (column
 * sums), the first moment M is kept in full, and the factors act in the
 * position equation.  Discrete step t (t = 1, 2, ...; Section 3 and App.
 * "Hyperparameters": beta2_t = 1 - t^{-0.8}, no relative step, no warm-up),
 * the factored algorithm of Shazeer & Stern (2018) with update clipping:
 *   b = 1 - t^decay_rate;  Q = G^2 + eps1
 *   R <- b R + (1-b) Q 1_n;  C <- b C + (1-b) Q^T 1_m
 *   U = G / sqrt(R C^T / 1^T R)               (U = 0 where that is 0)
 *   s = h * (scale_parameter ? max(eps2, RMS(X)) : 1) / max(1, RMS(U) / d)
 *       (no clipping when d = clip_threshold <= 0; RMS = root mean square
 *        over the tensor, X before the step)
 *   M <- beta1 M + (1 - beta1) s U;  X <- X - M (bf16 x: rounded to nearest even)
 * Vectors (m == 1 or n == 1) keep the unfactored second moment v (m*n fp32,
 * in c when m == 1, else in r) and use U = G / sqrt(v).
 *
 * Tensors reuse rikfad_tensor: p is the first moment M (m*n fp32), r and c
 * the factors (zero-filled by the caller before the first step).  The
 * caller owns every buffer; the context owns its tables and workspace.
 * Three passes stream the gradient (statistics, RMS of U, update), so a
 * step moves 28 bytes per fp32 parameter (18 with bf16 x and g; +4 / +2
 * with scale_parameter).  Every call enqueues on `stream` and returns;
 * same error conventions as the R-iKFAD entry points.  The step's
 * coefficients depend on t and are passed to the kernels by value, so a
 * step captured in a HIP graph would replay the same t: capture is not
 * supported for Adafactor-m.
 * ---------------------------------------------------------------------- */
typedef struct {
    double h;                /* step size (learning rate), > 0 */
    double beta1;            /* first-moment decay, 0 <= beta1 < 1 */
    double decay_rate;       /* beta2_t = 1 - t^decay_rate, <= 0 (paper: -0.8) */
    double eps1;             /* added to G^2, >= 0 (1e-30) */
    double eps2;             /* floor of RMS(X) in the parameter scale, >= 0 (1e-3) */
    double clip_threshold;   /* update clipping d, <= 0 disables it (1.0) */
    int32_t scale_parameter; /* 0 or 1 */
    int32_t reserved;        /* must be 0 */
} adafm_hparams;

typedef struct adafm_ctx adafm_ctx;

/* Validates like rikfad_create; the step counter starts at 0. */
rikfad_status adafm_create(const rikfad_tensor *tensors, int64_t count,
                           const adafm_hparams *hp, adafm_ctx **out);
/* Enqueues step t = (steps taken) + 1. */
rikfad_status adafm_step(adafm_ctx *ctx, void *stream);
/* As adafm_step with new gradient pointers (same rules as rikfad_step_grads). */
rikfad_status adafm_step_grads(adafm_ctx *ctx, const void *const *grads, void *stream);
rikfad_status adafm_set_hparams(adafm_ctx *ctx, const adafm_hparams *hp);
/* Steps taken so far (for resuming from a checkpoint), >= 0. */
rikfad_status adafm_set_step(adafm_ctx *ctx, int64_t steps_taken);
rikfad_status adafm_get_step(const adafm_ctx *ctx, int64_t *steps_taken);
/* Bytes the step must move (read x, g, M and g twice; write x, M; R, C). */
rikfad_status adafm_min_bytes(const adafm_ctx *ctx, int64_t *min_bytes_per_step,
                              int64_t *update_min_bytes, int64_t *state_bytes);
/* 1 if a non-finite R or C value was produced since create (blocks). */
rikfad_status adafm_nonfinite(adafm_ctx *ctx, void *stream, int32_t *out);
/* Kernel timing as for rikfad_timing_*: ms5[5] = statistics pass, factor
 * finalisation, RMS pass (0 when clipping is off or there are no
 * matrices), scale kernel, update pass, summed over the timed steps since
 * the last read. */
rikfad_status adafm_timing_enable(adafm_ctx *ctx, int32_t enable);
rikfad_status adafm_timing_read(adafm_ctx *ctx, double *ms5, int64_t *steps);
void adafm_destroy(adafm_ctx *ctx);

/* ------------------------------------------------------------------------
 * Bandwidth probes (measurement aids for the HBM roofline).
 *   rikfad_probe_stream: d[i] = a[i] + b[i], e[i] = a[i] * c[i] over nfloat
 *     fp32 elements -- the 3-read / 2-write mix of the fp32 step, with no
 *     other work.  All five pointers 16-byte aligned, nfloat % 4 == 0.
 *   rikfad_probe_copy: dst[i] = src[i] over nbytes (16-byte aligned,
 *     nbytes % 16 == 0), a plain copy of known size for calibrating
 *     hardware byte counters.
 *   rikfad_probe_mix: the step's own access mix without its arithmetic --
 *     read x, g (nelem elements of `dtype`, a rikfad_dtype) and p (nelem
 *     fp32), write x and p: 20 bytes per element for fp32 x/g, 14 for
 *     bf16.  x <- x + g (fp32) or the bitwise xor of x and g (bf16),
 *     p <- p / 2.  shape 0: contiguous, 4096 elements per workgroup of 256
 *     threads, every load of a workgroup before its first store; shape 1:
 *     the streaming kernel's workgroup (8 waves, each walking 4 rows of
 *     256 elements with the same ring of row loads).  nelem % 256 == 0;
 *     x, g 16-byte (fp32) or 8-byte (bf16) aligned, p 16-byte aligned.
 *   rikfad_probe_read: reads nbytes from src (16-byte aligned, nbytes % 16
 *     == 0) in four 16-byte loads per lane; writes *out (one float) only in
 *     the event that a workgroup's sum has one particular NaN bit pattern,
 *     which finite data never produces -- a read-only stream.
 *   rikfad_probe_write: fills nbytes at dst (16-byte aligned, nbytes % 16
 *     == 0) with the 32-bit pattern `value`, four 16-byte non-temporal
 *     stores per lane -- a write-only stream.
 * ---------------------------------------------------------------------- */
rikfad_status rikfad_probe_stream(const float *a, const float *b, const float *c,
                                  float *d, float *e, int64_t nfloat, void *stream);
rikfad_status rikfad_probe_copy(const void *src, void *dst, int64_t nbytes,
                                void *stream);
rikfad_status rikfad_probe_mix(void *x, const void *g, float *p, int64_t nelem,
                               int32_t dtype, int32_t shape, void *stream);
rikfad_status rikfad_probe_read(const void *src, int64_t nbytes, float *out,
                                void *stream);
rikfad_status rikfad_probe_write(void *dst, int64_t nbytes, uint32_t value, void *stream);

#ifdef __cplusplus
}
#endif
#endif
