/*
 * adafm_oracle.c -- plain fp64 CPU oracle for the Adafactor-m step.
 *
 * TEST INFRASTRUCTURE.  Correctness reference for the GPU Adafactor-m
 * kernels; only the test suite and the benchmark's CPU-baseline leg load
 * it.  It shares no source, table or helper with the GPU path.
 *
 * Written from the paper's definition of Adafactor-m (Section 2,
 * Methodology: Adafactor's factored second moment zeta^ = R C^T / 1^T R,
 * eq. (xi_def), with the momentum P kept) and its stated discrete schedule
 * (Section 3 and App. "Hyperparameters": beta2_t = 1 - t^{-0.8}, beta1 > 0,
 * no relative step and no warm-up), which is the factored Adafactor
 * algorithm of Shazeer & Stern (2018) with update clipping.  Everything is
 * fp64; the second-moment estimate V and the update U are materialised as
 * full arrays, sums run sequentially in index order.
 */
#include "adafm_oracle.h"

#include <math.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int valid(const orc_adafm_hparams *hp)
{
    if (!hp || hp->reserved != 0) return 0;
    if (!(isfinite(hp->h) && isfinite(hp->beta1) && isfinite(hp->decay_rate) &&
          isfinite(hp->eps1) && isfinite(hp->eps2) && isfinite(hp->clip_threshold)))
        return 0;
    return hp->h > 0.0 && hp->beta1 >= 0.0 && hp->beta1 < 1.0 && hp->decay_rate <= 0.0 &&
           hp->eps1 >= 0.0 && hp->eps2 >= 0.0 &&
           (hp->scale_parameter == 0 || hp->scale_parameter == 1);
}

double orc_adafm_beta2(int64_t t, double decay_rate)
{
    return 1.0 - pow((double)t, decay_rate);
}

/* Step size a_t: h, or h * max(eps2, RMS(X_{t-1})) with parameter scaling. */
static double step_size(int64_t k, const double *x, const orc_adafm_hparams *hp)
{
    if (!hp->scale_parameter) return hp->h;
    double s = 0.0;
    for (int64_t e = 0; e < k; ++e) s += x[e] * x[e];
    const double rms = sqrt(s / (double)k);
    return hp->h * (rms > hp->eps2 ? rms : hp->eps2);
}

/* Update clipping U^ = U / max(1, RMS(U)/d), then the first moment and the
 * parameter: M <- beta1 M + (1 - beta1) a U^, X <- X - M. */
static void clip_and_apply(int64_t k, const double *u, double a, int32_t x_bf16, double *x,
                           double *x_unrounded, double *mom, const orc_adafm_hparams *hp)
{
    double s = 0.0;
    for (int64_t e = 0; e < k; ++e) s += u[e] * u[e];
    const double rms = sqrt(s / (double)k);
    double div = 1.0;
    if (hp->clip_threshold > 0.0 && rms / hp->clip_threshold > 1.0)
        div = rms / hp->clip_threshold;
    for (int64_t e = 0; e < k; ++e) {
        const double uhat = u[e] / div;
        mom[e] = hp->beta1 * mom[e] + (1.0 - hp->beta1) * (a * uhat);
        const double xu = x[e] - mom[e];
        if (x_unrounded) x_unrounded[e] = xu;
        x[e] = x_bf16 ? orc_round_bf16(xu) : xu;
    }
}

int orc_adafm_matrix_step(int64_t m, int64_t n, int64_t t, int32_t x_bf16, double *x,
                          double *x_unrounded, const double *g, double *mom, double *r,
                          double *c, const orc_adafm_hparams *hp)
{
    if (m < 1 || n < 1 || t < 1 || !x || !g || !mom || !r || !c || !valid(hp)) return -1;
    const int64_t k = m * n;
    double *q = (double *)malloc(sizeof(double) * k);   /* G^2 + eps1 */
    double *v = (double *)malloc(sizeof(double) * k);   /* V = R C^T / 1^T R */
    double *u = (double *)malloc(sizeof(double) * k);   /* U = G / sqrt(V) */
    if (!q || !v || !u) {
        free(q); free(v); free(u);
        return -4;
    }
    const double a = step_size(k, x, hp);
    const double b = orc_adafm_beta2(t, hp->decay_rate);
    for (int64_t e = 0; e < k; ++e) q[e] = g[e] * g[e] + hp->eps1;

    /* Factor updates with the row sums Q 1_n and the column sums Q^T 1_m. */
    for (int64_t i = 0; i < m; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < n; ++j) s += q[i * n + j];
        r[i] = b * r[i] + (1.0 - b) * s;
    }
    for (int64_t j = 0; j < n; ++j) {
        double s = 0.0;
        for (int64_t i = 0; i < m; ++i) s += q[i * n + j];
        c[j] = b * c[j] + (1.0 - b) * s;
    }

    /* Rank-1 second moment and the normalised update. */
    double sr = 0.0;
    for (int64_t i = 0; i < m; ++i) sr += r[i];
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j)
            v[i * n + j] = (sr == 0.0) ? 0.0 : (r[i] * c[j]) / sr;
    for (int64_t e = 0; e < k; ++e) u[e] = (v[e] == 0.0) ? 0.0 : g[e] / sqrt(v[e]);

    clip_and_apply(k, u, a, x_bf16, x, x_unrounded, mom, hp);
    free(q); free(v); free(u);
    return 0;
}

int orc_adafm_vector_step(int64_t k, int64_t t, int32_t x_bf16, double *x,
                          double *x_unrounded, const double *g, double *mom, double *v,
                          const orc_adafm_hparams *hp)
{
    if (k < 1 || t < 1 || !x || !g || !mom || !v || !valid(hp)) return -1;
    double *u = (double *)malloc(sizeof(double) * k);
    if (!u) return -4;
    const double a = step_size(k, x, hp);
    const double b = orc_adafm_beta2(t, hp->decay_rate);
    for (int64_t e = 0; e < k; ++e) {
        v[e] = b * v[e] + (1.0 - b) * (g[e] * g[e] + hp->eps1);
        u[e] = (v[e] == 0.0) ? 0.0 : g[e] / sqrt(v[e]);
    }
    clip_and_apply(k, u, a, x_bf16, x, x_unrounded, mom, hp);
    free(u);
    return 0;
}

int orc_adafm_step_list(int64_t count, const orc_tensor *t, int64_t step,
                        const orc_adafm_hparams *hp, int nthreads)
{
    if (count < 0 || (count > 0 && !t) || step < 1 || !valid(hp)) return -1;
    int status = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) \
    reduction(min : status)
#endif
    for (int64_t i = 0; i < count; ++i) {
        const orc_tensor *T = &t[i];
        int s;
        if (T->m == 1 || T->n == 1)
            s = orc_adafm_vector_step(T->m * T->n, step, T->x_bf16, T->x, T->x_unrounded, T->g,
                                      T->p, T->m == 1 ? T->c : T->r, hp);
        else
            s = orc_adafm_matrix_step(T->m, T->n, step, T->x_bf16, T->x, T->x_unrounded, T->g,
                                      T->p, T->r, T->c, hp);
        if (s < status) status = s;
    }
    (void)nthreads;
    return status;
}
