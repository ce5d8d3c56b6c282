/*
 * rikfad_oracle.h -- plain fp64 CPU oracle for the R-iKFAD optimiser step.
 *
 * TEST INFRASTRUCTURE.  This library is the correctness reference against
 * which the GPU implementation is checked.  Only the test suite, the
 * package's smoke check and the benchmark's CPU-baseline leg may load it;
 * the GPU product path never calls it and shares no source with it.
 *
 * Source: R. Rajpal, B. Leimkuhler, "Low-Rank Friction for Memory-Efficient
 * Transformer Pretraining" (Rank-1 iKFAD).  Notation follows the paper:
 * parameter X (m x n, row-major), momentum P, row factor R (m), column
 * factor C (n), hyperparameters h, gamma, alpha, mu, eps_stab.
 *
 * All arithmetic is IEEE fp64 with no contraction (built with
 * -ffp-contract=off), sums are sequential in index order, and the rank-1
 * friction is materialised as a full m x n matrix, as the paper writes it.
 */
#ifndef RIKFAD_ORACLE_H
#define RIKFAD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    double h;        /* step size */
    double gamma;    /* linear damping (0 = R-iKFAD0) */
    double alpha;    /* factor relaxation rate */
    double mu;       /* friction mass: forcing of the factors is P^2 / mu */
    double eps_stab; /* stabiliser in the denominator of the rank-1 friction */
} orc_hparams;

/* One parameter tensor as the oracle holds it: every array is fp64.
 * x_bf16 != 0 means the parameter is stored in bfloat16: after the drift
 * the new X is rounded to the nearest bf16 value (ties to even).
 * x_unrounded (optional, may be NULL) receives X_n + h P^(B) before that
 * rounding.  For a vector (m == 1 or n == 1) the element-wise friction xi
 * lives in c when m == 1 and in r otherwise; the other factor is unused. */
typedef struct {
    double *x, *x_unrounded;
    const double *g;
    double *p, *r, *c;
    int64_t m, n;
    int32_t x_bf16;
    int32_t reserved;
} orc_tensor;

/* Status codes: 0 ok, -1 bad argument, -4 out of memory. */

/* Coefficients of the exact sub-flows over one step (App. A, Table of
 * sub-step updates, rows C and D): out[0] = exp(-alpha h), out[1] =
 * (1 - exp(-alpha h)) / (mu alpha) (limit h / mu at alpha = 0),
 * out[2] = exp(-gamma h). */
int orc_coefficients(const orc_hparams *hp, double out[3]);

/* Rank-1 friction xi~_ij = R_i C_j / (sum_k R_k + eps_stab), eq. (xi_def),
 * with xi~ = 0 when the denominator is zero (the eps_stab = 0 convention of
 * Theorem "Algebraic rates").  xi: m x n row-major output. */
int orc_rank1_friction(int64_t m, int64_t n, const double *r, const double *c,
                       double eps_stab, double *xi);

/* One BACD step of R-iKFAD on an m x n matrix (App. A Table; Section 2,
 * "Splitting Discretization").  Updates x, p, r, c in place. */
int orc_rikfad_matrix_step(int64_t m, int64_t n, int32_t x_bf16, double *x,
                           double *x_unrounded, const double *g, double *p,
                           double *r, double *c, const orc_hparams *hp);

/* One step of element-wise iKFAD on k entries (Section 1 iKFAD dynamics,
 * discretised by the same BACD splitting with the element-wise friction in
 * place of xi~).  R-iKFAD applies it to non-2D parameters (Section 2,
 * "Memory Complexity"); it is also the full-tensor comparison method. */
int orc_ikfad_step(int64_t k, int32_t x_bf16, double *x, double *x_unrounded,
                   const double *g, double *p, double *xi,
                   const orc_hparams *hp);

/* One R-iKFAD optimiser step over a parameter list: matrices take the
 * rank-1 step, vectors (m == 1 or n == 1) the element-wise iKFAD step.
 * Tensors are independent; nthreads > 1 spreads them over OpenMP threads. */
int orc_rikfad_step_list(int64_t count, const orc_tensor *t,
                         const orc_hparams *hp, int nthreads);

/* Nearest bfloat16 value of v, ties to even, rounding once from fp64. */
double orc_round_bf16(double v);
void orc_round_bf16_array(const double *in, double *out, int64_t k);

/* Strongly convex quadratic f(X) = 1/2 vec(X)^T A vec(X) (Section 3,
 * "Numerical validation of proved results"), integrated by the R-iKFAD
 * matrix step with gradient A vec(X).  A is d x d (d = m n), row-major,
 * vec(X) is X in row-major order.  Runs nsteps steps from (x, p, r, c),
 * updated in place.  Every `every` steps (and at step 0) it appends the
 * energy E = f + |P|^2/2 to energy[] (nsteps/every + 1 entries).
 * mod_increase (optional) receives the largest relative increase, over all
 * consecutive steps, of the modified energy f + |P|^2/2 - (h/2)<P, grad f>. */
int orc_quadratic_run(int64_t m, int64_t n, const double *A, double *x,
                      double *p, double *r, double *c, const orc_hparams *hp,
                      int64_t nsteps, int64_t every, double *energy,
                      double *mod_increase);

#ifdef __cplusplus
}
#endif
#endif
