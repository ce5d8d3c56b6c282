/*
 * c_abi_step.c -- a plain C program that drives the R-iKFAD library through
 * its C ABI alone (include/rikfad.h, no Python and no PyTorch) and checks
 * every result against the fp64 oracle.  Test infrastructure: it links the
 * oracle, which the product never does.
 *
 * The set: fp32 and bf16 matrices (one whose rows break 16-byte alignment,
 * so it takes the one-column path) and fp32 vectors of both orientations,
 * seeded momentum and factors (so the friction acts from the first step),
 * friction-strong hyperparameters, new gradients every step.  The library
 * runs in its default deferred form; rikfad_sync_momentum materialises
 * P_{n+1} before the final comparison.
 *
 * Bars (App. A Table, computed in fp32 on the GPU against fp64): for fp32 x
 * and p the element-wise error with an rms floor and the normwise error,
 * both <= 1e-5; for R, C and a vector's xi the plain relative error
 * <= 1e-5; for a bf16 parameter, after every step, the stored value against
 * the oracle's unrounded update from the same bf16 start, with the rms
 * floor, <= 4e-3 (rounding to bf16 costs at most 2^-8 relative).
 *
 * Usage: c_abi_step [seed] [steps].  Exit status 0: every bar met; 1: a bar
 * missed; 2: a library or HIP call failed; 77: no GPU.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "rikfad.h"
#include "rikfad_oracle.h"

/* ---------------------------------------------------------------- inputs */

/* splitmix64 (Steele, Lea, Flood 2014) and Box-Muller normals. */
static uint64_t sm64(uint64_t *s)
{
    uint64_t z = (*s += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

static double unif(uint64_t *s) /* (0, 1) */
{
    return ((double)(sm64(s) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

static double normal(uint64_t *s)
{
    const double u = unif(s), v = unif(s);
    return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

/* bf16 storage of an input value: the upper half of its fp32 bits. */
static uint16_t bf16_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

static double bf16_value(uint16_t b)
{
    const uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* ------------------------------------------------------------- the set */

typedef struct {
    int64_t m, n;
    int bf16;
} Shape;

static const Shape kShapes[] = {
    {300, 520, 0},  /* fp32, 16-byte rows, ragged column block and stripe */
    {97, 129, 0},   /* fp32, n odd: one-column path */
    {64, 1000, 1},  /* bf16 x and g */
    {40, 2052, 1},  /* bf16, several column blocks */
    {1, 333, 0},    /* vector, xi in c */
    {77, 1, 0},     /* vector, xi in r */
};
#define NT ((int)(sizeof kShapes / sizeof kShapes[0]))

typedef struct {
    int64_t m, n, k;
    int bf16;
    double *x, *xu, *g, *p, *r, *c;  /* oracle state, fp64 */
    double *srow, *scol;             /* gradient scales */
    void *hx, *hg;                   /* host staging of x and g (fp32 or bf16 bits) */
    float *hp, *hr, *hc;
    void *dx, *dg;                   /* device buffers */
    float *dp, *dr, *dc;
} T;

#define HIP(call)                                                                \
    do {                                                                         \
        hipError_t e_ = (call);                                                  \
        if (e_ != hipSuccess) {                                                  \
            fprintf(stderr, "HIP error %s at %s:%d\n", hipGetErrorString(e_), \
                    __FILE__, __LINE__);                                         \
            exit(2);                                                             \
        }                                                                        \
    } while (0)

#define LIB(call)                                                                      \
    do {                                                                               \
        rikfad_status s_ = (call);                                                     \
        if (s_ != RIKFAD_OK) {                                                         \
            fprintf(stderr, "%s failed: %s (%s)\n", #call, rikfad_status_string(s_), \
                    rikfad_last_error());                                              \
            exit(2);                                                                   \
        }                                                                              \
    } while (0)

static void *xmalloc(size_t bytes)
{
    void *q = calloc(bytes ? bytes : 1, 1);
    if (!q) {
        fprintf(stderr, "out of host memory\n");
        exit(2);
    }
    return q;
}

/* New gradients of every tensor, g_ij = s_i t_j z_ij, stored (fp32 or bf16)
 * and given to the oracle as the stored values. */
static void new_gradients(T *ts, uint64_t *rng)
{
    for (int i = 0; i < NT; ++i) {
        T *t = &ts[i];
        for (int64_t a = 0; a < t->m; ++a)
            for (int64_t b = 0; b < t->n; ++b) {
                const int64_t e = a * t->n + b;
                const float v = (float)(t->srow[a] * t->scol[b] * normal(rng));
                if (t->bf16) {
                    ((uint16_t *)t->hg)[e] = bf16_bits(v);
                    t->g[e] = bf16_value(((uint16_t *)t->hg)[e]);
                } else {
                    ((float *)t->hg)[e] = v;
                    t->g[e] = (double)v;
                }
            }
        HIP(hipMemcpy(t->dg, t->hg, (size_t)t->k * (t->bf16 ? 2 : 4), hipMemcpyHostToDevice));
    }
}

/* ---------------------------------------------------------------- metrics */

static double rms(const double *b, int64_t k)
{
    double s = 0.0;
    for (int64_t i = 0; i < k; ++i) s += b[i] * b[i];
    return k ? sqrt(s / (double)k) : 0.0;
}

static double err_rms_floor(const float *a32, const double *a64, const double *b, int64_t k)
{
    const double fl = rms(b, k);
    double worst = 0.0;
    for (int64_t i = 0; i < k; ++i) {
        const double a = a32 ? (double)a32[i] : a64[i];
        if (!isfinite(a)) return INFINITY;
        double den = fabs(b[i]) > fl ? fabs(b[i]) : fl;
        if (den == 0.0) den = 1.0;
        const double e = fabs(a - b[i]) / den;
        if (e > worst) worst = e;
    }
    return worst;
}

static double err_norm(const float *a, const double *b, int64_t k)
{
    double d = 0.0, s = 0.0;
    for (int64_t i = 0; i < k; ++i) {
        if (!isfinite(a[i])) return INFINITY;
        const double e = fabs((double)a[i] - b[i]);
        if (e > d) d = e;
        if (fabs(b[i]) > s) s = fabs(b[i]);
    }
    return s > 0.0 ? d / s : (d == 0.0 ? 0.0 : INFINITY);
}

static int cmp_double(const void *a, const void *b)
{
    const double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/* Median over a matrix's elements of (h/2) xi~_ij = (h/2) R_i C_j / (1^T R + eps). */
static double median_half_kick(const T *t, double h, double eps)
{
    double sr = 0.0;
    for (int64_t a = 0; a < t->m; ++a) sr += t->r[a];
    double *v = xmalloc(sizeof(double) * t->k);
    for (int64_t a = 0; a < t->m; ++a)
        for (int64_t b = 0; b < t->n; ++b)
            v[a * t->n + b] = 0.5 * h * t->r[a] * t->c[b] / (sr + eps);
    qsort(v, (size_t)t->k, sizeof(double), cmp_double);
    const double med = v[t->k / 2];
    free(v);
    return med;
}

static double err_plain(const float *a, const double *b, int64_t k)
{
    double worst = 0.0;
    for (int64_t i = 0; i < k; ++i) {
        if (!isfinite(a[i])) return INFINITY;
        const double d = fabs((double)a[i] - b[i]);
        if (d == 0.0) continue;
        const double e = b[i] != 0.0 ? d / fabs(b[i]) : INFINITY;
        if (e > worst) worst = e;
    }
    return worst;
}

/* ------------------------------------------------------------------ main */

int main(int argc, char **argv)
{
    const uint64_t seed = argc > 1 ? strtoull(argv[1], NULL, 10) : 1;
    const int steps = argc > 2 ? atoi(argv[2]) : 12;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        printf("no GPU\n");
        return 77;
    }
    HIP(hipSetDevice(0));
    uint64_t rng = seed * 0x2545f4914f6cdd1dull + 17;

    T ts[NT];
    rikfad_tensor lt[NT];
    orc_tensor ot[NT];
    memset(ts, 0, sizeof ts);
    for (int i = 0; i < NT; ++i) {
        T *t = &ts[i];
        t->m = kShapes[i].m;
        t->n = kShapes[i].n;
        t->k = t->m * t->n;
        t->bf16 = kShapes[i].bf16;
        const size_t es = t->bf16 ? 2 : 4;
        t->x = xmalloc(sizeof(double) * t->k);
        t->xu = xmalloc(sizeof(double) * t->k);
        t->g = xmalloc(sizeof(double) * t->k);
        t->p = xmalloc(sizeof(double) * t->k);
        t->r = xmalloc(sizeof(double) * t->m);
        t->c = xmalloc(sizeof(double) * t->n);
        t->srow = xmalloc(sizeof(double) * t->m);
        t->scol = xmalloc(sizeof(double) * t->n);
        t->hx = xmalloc(es * t->k);
        t->hg = xmalloc(es * t->k);
        t->hp = xmalloc(sizeof(float) * t->k);
        t->hr = xmalloc(sizeof(float) * t->m);
        t->hc = xmalloc(sizeof(float) * t->n);
        for (int64_t a = 0; a < t->m; ++a) t->srow[a] = exp(0.5 * normal(&rng));
        for (int64_t b = 0; b < t->n; ++b) t->scol[b] = exp(0.5 * normal(&rng));
        for (int64_t e = 0; e < t->k; ++e) {
            const float xv = (float)(0.02 * normal(&rng));
            if (t->bf16) {
                ((uint16_t *)t->hx)[e] = bf16_bits(xv);
                t->x[e] = bf16_value(((uint16_t *)t->hx)[e]);
            } else {
                ((float *)t->hx)[e] = xv;
                t->x[e] = (double)xv;
            }
            t->hp[e] = (float)(0.05 * normal(&rng));
            t->p[e] = (double)t->hp[e];
        }
        /* Seeded non-negative factors (a vector's xi lives in c when m == 1
         * and in r otherwise; the other factor is unused but still held). */
        for (int64_t a = 0; a < t->m; ++a) {
            t->hr[a] = (float)(0.2 * unif(&rng));
            t->r[a] = (double)t->hr[a];
        }
        for (int64_t b = 0; b < t->n; ++b) {
            t->hc[b] = (float)(0.2 * unif(&rng));
            t->c[b] = (double)t->hc[b];
        }
        HIP(hipMalloc(&t->dx, es * t->k));
        HIP(hipMalloc(&t->dg, es * t->k));
        HIP(hipMalloc((void **)&t->dp, sizeof(float) * t->k));
        HIP(hipMalloc((void **)&t->dr, sizeof(float) * t->m));
        HIP(hipMalloc((void **)&t->dc, sizeof(float) * t->n));
        HIP(hipMemcpy(t->dx, t->hx, es * t->k, hipMemcpyHostToDevice));
        HIP(hipMemcpy(t->dp, t->hp, sizeof(float) * t->k, hipMemcpyHostToDevice));
        HIP(hipMemcpy(t->dr, t->hr, sizeof(float) * t->m, hipMemcpyHostToDevice));
        HIP(hipMemcpy(t->dc, t->hc, sizeof(float) * t->n, hipMemcpyHostToDevice));
        lt[i] = (rikfad_tensor){t->dx, t->dg, t->dp, t->dr, t->dc, t->m, t->n,
                                t->bf16 ? RIKFAD_BF16 : RIKFAD_FP32, 0};
        ot[i] = (orc_tensor){t->x, t->xu, t->g, t->p, t->r, t->c, t->m, t->n, t->bf16, 0};
    }

    /* Friction strong enough that (h/2) xi~ is of order 0.1. */
    const rikfad_hparams hp = {0.1, 0.0, 0.1, 0.1, 1e-8};
    const orc_hparams ohp = {hp.h, hp.gamma, hp.alpha, hp.mu, hp.eps_stab};
    hipStream_t stream;
    HIP(hipStreamCreate(&stream));
    rikfad_ctx *ctx = NULL;
    LIB(rikfad_create(lt, NT, &hp, 0, &ctx));
    rikfad_info info;
    LIB(rikfad_query(ctx, &info));
    printf("c_abi_step: seed %llu, %d steps, %lld tensors (%lld matrices, %lld vectors), "
           "%lld elements, %lld streaming workgroups\n",
           (unsigned long long)seed, steps, (long long)info.tensors, (long long)info.matrices,
           (long long)info.vectors, (long long)info.elements, (long long)info.stream_tiles);
    fflush(stdout);

    int bad = 0;
    double worst_bf16 = 0.0;
    for (int s = 0; s < steps; ++s) {
        new_gradients(ts, &rng);
        LIB(rikfad_step(ctx, stream));
        if (orc_rikfad_step_list(NT, ot, &ohp, 1) != 0) {
            fprintf(stderr, "oracle step failed\n");
            return 2;
        }
        HIP(hipStreamSynchronize(stream));
        /* bf16 parameters: the stored value against the unrounded update,
         * then the oracle continues from the stored value. */
        for (int i = 0; i < NT; ++i) {
            T *t = &ts[i];
            if (!t->bf16) continue;
            HIP(hipMemcpy(t->hx, t->dx, 2 * (size_t)t->k, hipMemcpyDeviceToHost));
            for (int64_t e = 0; e < t->k; ++e) t->x[e] = bf16_value(((uint16_t *)t->hx)[e]);
            const double err = err_rms_floor(NULL, t->x, t->xu, t->k);
            if (err > worst_bf16) worst_bf16 = err;
            if (!(err <= 4e-3)) {
                printf("step %d tensor %d (%lldx%lld bf16): x %.3e > 4e-3\n", s, i,
                       (long long)t->m, (long long)t->n, err);
                bad = 1;
            }
        }
    }
    LIB(rikfad_sync_momentum(ctx, stream));
    int32_t nonfinite = -1;
    LIB(rikfad_nonfinite(ctx, stream, &nonfinite));
    HIP(hipStreamSynchronize(stream));
    if (nonfinite != 0) {
        printf("non-finite flag set: %d\n", nonfinite);
        bad = 1;
    }

    double median_kick = 0.0;
    for (int i = 0; i < NT; ++i) {
        T *t = &ts[i];
        const int vec = t->m == 1 || t->n == 1;
        HIP(hipMemcpy(t->hp, t->dp, sizeof(float) * t->k, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(t->hr, t->dr, sizeof(float) * t->m, hipMemcpyDeviceToHost));
        HIP(hipMemcpy(t->hc, t->dc, sizeof(float) * t->n, hipMemcpyDeviceToHost));
        double ex = 0.0, exn = 0.0;
        if (!t->bf16) {
            HIP(hipMemcpy(t->hx, t->dx, sizeof(float) * t->k, hipMemcpyDeviceToHost));
            ex = err_rms_floor((const float *)t->hx, NULL, t->x, t->k);
            exn = err_norm((const float *)t->hx, t->x, t->k);
        }
        const double ep = err_rms_floor(t->hp, NULL, t->p, t->k);
        const double epn = err_norm(t->hp, t->p, t->k);
        double er = 0.0, ec = 0.0;
        if (!vec || t->n == 1) er = err_plain(t->hr, t->r, t->m);
        if (!vec || t->m == 1) ec = err_plain(t->hc, t->c, t->n);
        const int ok = ex <= 1e-5 && exn <= 1e-5 && ep <= 1e-5 && epn <= 1e-5 && er <= 1e-5 &&
                       ec <= 1e-5;
        if (i == 0) median_kick = median_half_kick(t, hp.h, hp.eps_stab);
        printf("tensor %d %lldx%lld %s: x %.2e/%.2e p %.2e/%.2e R %.2e C %.2e %s\n", i,
               (long long)t->m, (long long)t->n, t->bf16 ? "bf16" : "fp32", ex, exn, ep, epn, er,
               ec, ok ? "ok" : "FAIL");
        if (!ok) bad = 1;
    }
    printf("bf16 x, worst step: %.2e; median (h/2) xi~ of the first matrix: %.3e\n",
           worst_bf16, median_kick);
    if (!(median_kick > 1e-2)) {
        printf("friction too weak to exercise the half-kicks\n");
        bad = 1;
    }
    rikfad_destroy(ctx);
    for (int i = 0; i < NT; ++i) {
        T *t = &ts[i];
        HIP(hipFree(t->dx));
        HIP(hipFree(t->dg));
        HIP(hipFree(t->dp));
        HIP(hipFree(t->dr));
        HIP(hipFree(t->dc));
        free(t->x); free(t->xu); free(t->g); free(t->p); free(t->r); free(t->c);
        free(t->srow); free(t->scol); free(t->hx); free(t->hg);
        free(t->hp); free(t->hr); free(t->hc);
    }
    HIP(hipStreamDestroy(stream));
    printf(bad ? "c_abi_step: FAIL\n" : "c_abi_step: all bars met\n");
    return bad;
}
