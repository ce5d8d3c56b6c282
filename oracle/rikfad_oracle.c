/*
 * rikfad_oracle.c -- plain fp64 CPU oracle for the R-iKFAD optimiser step.
 *
 * TEST INFRASTRUCTURE.  This is the correctness reference for the GPU
 * implementation.  Only the test suite, the package's smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no source, header,
 * table or helper with the GPU path, and the GPU path never calls it.
 *
 * Written from R. Rajpal, B. Leimkuhler, "Low-Rank Friction for
 * Memory-Efficient Transformer Pretraining":
 *   - Section 2, eqs. (rikfad_x)-(rikfad_C): the continuous R-iKFAD system;
 *   - Section 2, eq. (xi_def): the rank-1 friction xi~ = R C^T/(1^T R + eps);
 *   - Section 2, "Splitting Discretization", and App. A, Table of analytical
 *     sub-step updates: the BACD step B -> A -> C -> D;
 *   - Section 2, "Memory Complexity": non-2D parameters use element-wise iKFAD;
 *   - Theorem "Algebraic rates" and App. "Numerical Setup": xi~ = 0 when the
 *     denominator vanishes (eps_stab = 0 and 1^T R = 0).
 *
 * Everything is fp64, sums run sequentially in index order, and xi~ is
 * materialised as an m x n matrix exactly as the Table writes it.  Nothing
 * here is blocked, fused or reordered.
 */
#include "rikfad_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int valid_hparams(const orc_hparams *hp)
{
    if (!hp) return 0;
    if (!(isfinite(hp->h) && isfinite(hp->gamma) && isfinite(hp->alpha) &&
          isfinite(hp->mu) && isfinite(hp->eps_stab)))
        return 0;
    return hp->h > 0.0 && hp->mu > 0.0 && hp->alpha >= 0.0 &&
           hp->gamma >= 0.0 && hp->eps_stab >= 0.0;
}

/* App. A Table: R_{n+1} = e^{-alpha h} R_n + (1 - e^{-alpha h})/(mu alpha) [P^(1)]^2 1
 * (and the same for C); D multiplies the momentum by e^{-gamma h}.
 * 1 - e^{-alpha h} is evaluated as -expm1(-alpha h), the same number without
 * the cancellation.  At alpha = 0 the factor ODE has no decay and the exact
 * flow over h adds (h / mu) [P]^2 1, the alpha -> 0 limit of the formula. */
int orc_coefficients(const orc_hparams *hp, double out[3])
{
    if (!valid_hparams(hp) || !out) return -1;
    const double ah = hp->alpha * hp->h;
    out[0] = exp(-ah);
    out[1] = (hp->alpha > 0.0) ? (-expm1(-ah)) / (hp->mu * hp->alpha)
                               : hp->h / hp->mu;
    out[2] = exp(-hp->gamma * hp->h);
    return 0;
}

/* eq. (xi_def): xi~_ij = R_i C_j / (1_m^T R + eps_stab); zero when the
 * denominator is zero (convention for eps_stab = 0 at R = 0). */
int orc_rank1_friction(int64_t m, int64_t n, const double *r, const double *c,
                       double eps_stab, double *xi)
{
    if (m < 1 || n < 1 || !r || !c || !xi) return -1;
    double s = 0.0;
    for (int64_t i = 0; i < m; ++i) s += r[i];
    const double denom = s + eps_stab;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j)
            xi[i * n + j] = (denom == 0.0) ? 0.0 : (r[i] * c[j]) / denom;
    return 0;
}

/* Sub-steps B and A of the Table: P^(B) = P_n - h grad f(X_n), then
 * X_{n+1} = X_n + h P^(B) (the drift uses the kicked momentum).  A bf16
 * parameter is stored rounded to nearest bf16. */
static void kick_and_drift(int64_t k, double h, int32_t x_bf16, double *x,
                           double *x_unrounded, const double *g,
                           const double *p, double *pb)
{
    for (int64_t e = 0; e < k; ++e) {
        pb[e] = p[e] - h * g[e];
        const double xu = x[e] + h * pb[e];
        if (x_unrounded) x_unrounded[e] = xu;
        x[e] = x_bf16 ? orc_round_bf16(xu) : xu;
    }
}

int orc_rikfad_matrix_step(int64_t m, int64_t n, int32_t x_bf16, double *x,
                           double *x_unrounded, const double *g, double *p,
                           double *r, double *c, const orc_hparams *hp)
{
    double coef[3];
    if (m < 1 || n < 1 || !x || !g || !p || !r || !c) return -1;
    if (orc_coefficients(hp, coef) != 0) return -1;
    const double a = coef[0], kappa = coef[1], d = coef[2], h = hp->h;
    const int64_t k = m * n;

    double *pb = (double *)malloc(sizeof(double) * k);    /* P^(B) */
    double *p1 = (double *)malloc(sizeof(double) * k);    /* P^(1) */
    double *xi = (double *)malloc(sizeof(double) * k);    /* xi~   */
    double *rowsq = (double *)calloc((size_t)m, sizeof(double));
    double *colsq = (double *)calloc((size_t)n, sizeof(double));
    if (!pb || !p1 || !xi || !rowsq || !colsq) {
        free(pb); free(p1); free(xi); free(rowsq); free(colsq);
        return -4;
    }

    /* B, A */
    kick_and_drift(k, h, x_bf16, x, x_unrounded, g, p, pb);

    /* C: xi~_n from the current factors; first half-kick
     * P^(1) = P^(B) .* exp(-(h/2) xi~_n). */
    orc_rank1_friction(m, n, r, c, hp->eps_stab, xi);
    for (int64_t e = 0; e < k; ++e) p1[e] = pb[e] * exp(-0.5 * h * xi[e]);

    /* C: exact factor update with the momentum held at P^(1):
     * row sums [P^(1)]^2 1_n and column sums ([P^(1)]^2)^T 1_m. */
    for (int64_t i = 0; i < m; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j) s += p1[i * n + j] * p1[i * n + j];
        rowsq[i] = s;
    }
    for (int64_t i = 0; i < m; ++i)            /* colsq[j] accumulates in i order */
        for (int64_t j = 0; j < n; ++j) colsq[j] += p1[i * n + j] * p1[i * n + j];
    for (int64_t i = 0; i < m; ++i) r[i] = a * r[i] + kappa * rowsq[i];
    for (int64_t j = 0; j < n; ++j) c[j] = a * c[j] + kappa * colsq[j];

    /* C: xi~_{n+1} from the updated factors; second half-kick
     * P^(2) = P^(1) .* exp(-(h/2) xi~_{n+1}).  D: P_{n+1} = P^(2) e^{-gamma h}. */
    orc_rank1_friction(m, n, r, c, hp->eps_stab, xi);
    for (int64_t e = 0; e < k; ++e) {
        const double p2 = p1[e] * exp(-0.5 * h * xi[e]);
        p[e] = p2 * d;
    }

    free(pb); free(p1); free(xi); free(rowsq); free(colsq);
    return 0;
}

/* Element-wise iKFAD: the iKFAD friction ODE xi' = P^2/mu - alpha xi
 * (Section 1) with the same BACD splitting and the same half-kick / exact
 * friction update / half-kick treatment of sub-flow C, one friction entry
 * per parameter. */
int orc_ikfad_step(int64_t k, int32_t x_bf16, double *x, double *x_unrounded,
                   const double *g, double *p, double *xi,
                   const orc_hparams *hp)
{
    double coef[3];
    if (k < 1 || !x || !g || !p || !xi) return -1;
    if (orc_coefficients(hp, coef) != 0) return -1;
    const double a = coef[0], kappa = coef[1], d = coef[2], h = hp->h;

    double *pb = (double *)malloc(sizeof(double) * k);
    if (!pb) return -4;
    kick_and_drift(k, h, x_bf16, x, x_unrounded, g, p, pb);
    for (int64_t e = 0; e < k; ++e) {
        const double p1 = pb[e] * exp(-0.5 * h * xi[e]);
        xi[e] = a * xi[e] + kappa * (p1 * p1);
        const double p2 = p1 * exp(-0.5 * h * xi[e]);
        p[e] = p2 * d;
    }
    free(pb);
    return 0;
}

int orc_rikfad_step_list(int64_t count, const orc_tensor *t,
                         const orc_hparams *hp, int nthreads)
{
    if (count < 0 || (count > 0 && !t) || !valid_hparams(hp)) return -1;
    int err = 0;
#ifdef _OPENMP
    if (nthreads < 1) nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads) reduction(min : err)
#endif
    for (int64_t i = 0; i < count; ++i) {
        const orc_tensor *T = &t[i];
        int e;
        if (T->m == 1 || T->n == 1) {
            double *xi = (T->m == 1) ? T->c : T->r;
            e = orc_ikfad_step(T->m * T->n, T->x_bf16, T->x, T->x_unrounded,
                               T->g, T->p, xi, hp);
        } else {
            e = orc_rikfad_matrix_step(T->m, T->n, T->x_bf16, T->x,
                                       T->x_unrounded, T->g, T->p, T->r, T->c,
                                       hp);
        }
        if (e < err) err = e;
    }
    (void)nthreads;
    return err;
}

/* bfloat16 keeps 8 significant bits and fp32's exponent range: normal
 * numbers down to 2^-126, subnormals in steps of 2^-133, largest finite
 * (2 - 2^-7) 2^127.  Round |v| to a multiple of its quantum with
 * nearbyint (ties to even in the default rounding mode). */
double orc_round_bf16(double v)
{
    if (isnan(v) || isinf(v) || v == 0.0) return v;
    const double av = fabs(v);
    int e;
    frexp(av, &e);                      /* av = f 2^e, f in [0.5, 1) */
    const int unbiased = e - 1;         /* av in [2^unbiased, 2^(unbiased+1)) */
    const int qexp = (unbiased >= -126 ? unbiased : -126) - 7;
    const double q = nearbyint(ldexp(av, -qexp));
    double out = ldexp(q, qexp);
    if (out >= ldexp(1.0, 128)) out = INFINITY;
    return copysign(out, v);
}

void orc_round_bf16_array(const double *in, double *out, int64_t k)
{
    for (int64_t e = 0; e < k; ++e) out[e] = orc_round_bf16(in[e]);
}

static double quad_energy_terms(int64_t d, const double *A, const double *x,
                                const double *p, double *grad, double *f,
                                double *kin, double *pg)
{
    double fx = 0.0, kk = 0.0, dot = 0.0;
    for (int64_t i = 0; i < d; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < d; ++j) s += A[i * d + j] * x[j];
        grad[i] = s;
    }
    for (int64_t i = 0; i < d; ++i) {
        fx += 0.5 * x[i] * grad[i];
        kk += 0.5 * p[i] * p[i];
        dot += p[i] * grad[i];
    }
    *f = fx; *kin = kk; *pg = dot;
    return fx + kk;
}

int orc_quadratic_run(int64_t m, int64_t n, const double *A, double *x,
                      double *p, double *r, double *c, const orc_hparams *hp,
                      int64_t nsteps, int64_t every, double *energy,
                      double *mod_increase)
{
    if (m < 1 || n < 1 || !A || !x || !p || !r || !c || nsteps < 0 ||
        every < 1 || !energy || !valid_hparams(hp))
        return -1;
    const int64_t d = m * n;
    double *grad = (double *)malloc(sizeof(double) * d);
    if (!grad) return -4;
    double f, kin, pg;
    double E = quad_energy_terms(d, A, x, p, grad, &f, &kin, &pg);
    double H = E - 0.5 * hp->h * pg;    /* modified energy of the kick-drift pair */
    double worst = -INFINITY;
    int64_t rec = 0;
    energy[rec++] = E;
    int err = 0;
    for (int64_t s = 1; s <= nsteps && !err; ++s) {
        /* grad holds grad f(X_n) from the energy evaluation at X_n */
        err = orc_rikfad_matrix_step(m, n, 0, x, NULL, grad, p, r, c, hp);
        E = quad_energy_terms(d, A, x, p, grad, &f, &kin, &pg);
        const double Hn = E - 0.5 * hp->h * pg;
        const double inc = (Hn - H) / fabs(H);
        if (inc > worst) worst = inc;
        H = Hn;
        if (s % every == 0) energy[rec++] = E;
    }
    if (mod_increase) *mod_increase = worst;
    free(grad);
    return err;
}
