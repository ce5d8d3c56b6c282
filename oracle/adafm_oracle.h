/*
 * adafm_oracle.h -- plain fp64 CPU oracle for the Adafactor-m step.
 *
 * TEST INFRASTRUCTURE.  Correctness reference for the GPU Adafactor-m
 * kernels; only the test suite and the benchmark's CPU-baseline leg may
 * load it.  It shares no source with the GPU path.
 *
 * Adafactor-m is the paper's baseline: Adafactor's factored second moment
 * with a full first moment kept (Section 2, Methodology, left-hand system
 * and eq. (xi_def) for zeta^ = R C^T / 1^T R).  Its discrete schedule is the
 * one the paper states it uses (Section 3 and App. "Hyperparameters"):
 * beta2_t = 1 - t^{-0.8}, beta1 > 0, no relative step size and no warm-up,
 * i.e. the factored algorithm of Shazeer & Stern (2018) with its update
 * clipping, a plain step size h and momentum on the clipped update.  The
 * readings of the points the paper leaves open are listed with the
 * functions below.
 */
#ifndef ADAFM_ORACLE_H
#define ADAFM_ORACLE_H

#include <stdint.h>

#include "rikfad_oracle.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    double h;               /* step size (learning rate) */
    double beta1;           /* first-moment decay, 0 <= beta1 < 1 */
    double decay_rate;      /* beta2_t = 1 - t^decay_rate, decay_rate <= 0 (paper: -0.8) */
    double eps1;            /* added to G^2 before the second-moment update (>= 0) */
    double eps2;            /* floor of RMS(X) in the parameter scale (>= 0) */
    double clip_threshold;  /* update clipping threshold d; <= 0 disables clipping */
    int32_t scale_parameter;/* 1: step h * max(eps2, RMS(X_{t-1})); 0: step h */
    int32_t reserved;       /* must be 0 */
} orc_adafm_hparams;

/* beta2_t = 1 - t^decay_rate for step t >= 1 (beta2_1 = 0). */
double orc_adafm_beta2(int64_t t, double decay_rate);

/* Step t (t >= 1 counts steps including this one) on an m x n matrix with
 * the factored second moment (R: m row sums, C: n column sums):
 *   Q = G^2 + eps1;  R <- b R + (1-b) Q 1_n;  C <- b C + (1-b) Q^T 1_m  (b = beta2_t)
 *   V = R C^T / (1^T R)             (V = 0 where 1^T R = 0)
 *   U = G / sqrt(V)                 (U = 0 where V = 0)
 *   U^ = U / max(1, RMS(U) / d)     (no clipping when d <= 0)
 *   a_t = h * (scale ? max(eps2, RMS(X_{t-1})) : 1)
 *   M <- beta1 M + (1 - beta1) a_t U^;   X <- X - M   (bf16: rounded to nearest)
 * RMS(Y) = sqrt(mean of Y^2).  x_unrounded (optional) receives X - M before
 * the bf16 rounding. */
int orc_adafm_matrix_step(int64_t m, int64_t n, int64_t t, int32_t x_bf16, double *x,
                          double *x_unrounded, const double *g, double *mom, double *r,
                          double *c, const orc_adafm_hparams *hp);

/* The same step for a non-2D parameter of k entries with the unfactored
 * second moment v (k entries): v <- b v + (1-b)(G^2 + eps1), U = G / sqrt(v). */
int orc_adafm_vector_step(int64_t k, int64_t t, int32_t x_bf16, double *x,
                          double *x_unrounded, const double *g, double *mom, double *v,
                          const orc_adafm_hparams *hp);

/* One Adafactor-m step t over a parameter list: p holds the first moment
 * M; matrices keep R, C in r, c; a vector (m == 1 or n == 1) keeps v in c
 * when m == 1 and in r otherwise. */
int orc_adafm_step_list(int64_t count, const orc_tensor *t, int64_t step,
                        const orc_adafm_hparams *hp, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
