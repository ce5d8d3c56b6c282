// diag.hip -- rank-1 friction diagnostic on gfx950.
//
// Section 4 of the paper ("How Close is xi~ to the Best Rank-1 Friction?")
// runs iKFAD0 while updating R-iKFAD's factors R, C as shadow states fed by
// the same P^(1), then compares the full friction xi with the rank-1
// xi~ = R C^T / (1^T R + eps) against the Eckart-Young floor
// sqrt(1 - sigma_1^2 / |xi|_F^2), and reports the stable rank
// |xi|_F^2 / sigma_1^2.  Both xi and the shadow factors obey the same
// linear filter driven by [P^(1)]^2, so from R = C = xi = 0 the shadows are
// exactly R = xi 1 and C = xi^T 1: this file computes them from xi directly.
//
// Every quantity is a deterministic reduction (fixed partition, fixed
// order): row sums one wave per row, column sums in row stripes then
// folded in stripe order, squared norms per workgroup then folded in order.
// sigma_1 comes from power iteration on xi^T xi started at C / |C| (xi >= 0,
// so the leading singular vectors are non-negative), normalised on the GPU:
// the column fold also writes per-workgroup squared-norm partials, from
// which every wave of the next row pass derives the same scale.  For
// n <= 1024 an iteration reads xi once (u = xi v and xi^T u in one pass).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>
#include <mutex>
#include <string>

#include "../../include/rikfad.h"
#include "kernels.hpp"

namespace {

constexpr int kT = 256;            // threads per workgroup
constexpr int kStatChunk = 4096;   // elements per workgroup of the vector statistics
constexpr int kErrRows = 16;       // rows per workgroup of the error pass
// 4 columns x 64 stripe groups per fold workgroup (6.4 us a fold of 393
// x 768 partial sums with 8 x 32; 2 x 128 slower again).
#ifndef RK_DIAG_FOLD_COLS
#define RK_DIAG_FOLD_COLS 4
#endif
constexpr int kFoldCols = RK_DIAG_FOLD_COLS;        // columns per workgroup of the column fold
constexpr int kFoldGroups = 256 / kFoldCols;        // stripe groups per column of the column fold
static_assert(kFoldCols * kFoldGroups == 256, "fold workgroup shape");

#define DG __attribute__((address_space(1)))
template <typename T> __device__ __forceinline__ const DG T *gp(const T *q) { return (const DG T *)q; }
template <typename T> __device__ __forceinline__ DG T *gp(T *q) { return (DG T *)q; }

// Wave-level sum in a fixed butterfly order (every lane gets the same bits).
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

// Scale of a vector from its fold partials: 1 / sqrt(sum_q parts[2 q]) in
// a fixed order (lanes stride over the partials, then the butterfly), 0 for
// a zero vector; every wave that calls it gets the same bits.
__device__ __forceinline__ double inv_norm(const double *__restrict__ parts, int64_t nparts)
{
    const int lane = threadIdx.x & 63;
    double s = 0.0;
    for (int64_t q = lane; q < nparts; q += 64) s += gp(parts)[2 * q];
    s = wave_sum(s);
    return s > 0.0 ? 1.0 / sqrt(s) : 0.0;
}

// t where c holds, else +0.  A bitwise mask rather than a select: a select
// between a loaded value and 0 is compiled into a branch around the load.
__device__ __forceinline__ float keep_if(bool c, float t)
{
    return __uint_as_float(__float_as_uint(t) & (c ? 0xffffffffu : 0u));
}
__device__ __forceinline__ double keep_if(bool c, double t)
{
    return __longlong_as_double(__double_as_longlong(t) & (c ? ~0ll : 0ll));
}

// out[i] = sum_j xi[i, j] * (w ? w[j] * scale : 1) with scale = inv_norm of
// w's fold partials: one wave per row, lanes stride over the columns, fp64
// accumulation.
__global__ __launch_bounds__(kT) void row_reduce_kernel(const float *__restrict__ xi, int64_t m,
                                                        int64_t n, const double *__restrict__ w,
                                                        const double *__restrict__ wparts,
                                                        int64_t nwparts, double *__restrict__ out)
{
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (kT / 64) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= m) return;
    const double scale = w ? inv_norm(wparts, nwparts) : 1.0;
    const DG float *xr = gp(xi) + row * n;
    double s = 0.0;
    // Eight loads in flight per lane; additions in column order.
    for (int64_t j0 = lane; j0 < n; j0 += 64 * 8) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t j = j0 + 64 * u;
            const int64_t jc = j < n ? j : n - 1;         // in the row; masked below
            v[u] = keep_if(j < n, static_cast<double>(xr[jc]) * (w ? gp(w)[jc] : 1.0));
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    s = wave_sum(s);
    if (lane == 0) gp(out)[row] = w ? s * scale : s;
}

// One pass over xi for n <= 64 * NC, reading xi once: a workgroup takes
// kPowRows rows, each of its kPowWaves waves an equal share in order.  Lane
// l holds columns l, l + 64, ... of a row in registers; the wave forms the row's
// weighted sum s_i = sum_j xi[i, j] w_j (lanes in column order, then the
// butterfly) and adds xi[i, j] times a row weight to its column
// accumulators, rows in order.  The waves' column sums are added in wave
// order into the workgroup's row of part (folded by col_fold_kernel), and
// the per-lane scalar sums into the workgroup's pair of spart.  MODE:
//   kPassSums      w = 1: writes R_i = s_i; column weight 1, so part holds
//                  partial column sums of xi (C)
//   kPassPower     w = v / |v| (scale from v's fold partials): u_i = s_i;
//                  column weight u_i (xi^T u)
//   kPassPowerErr  kPassPower, plus spart = (sum xi^2, sum (xi - xi~)^2)
//                  with xi~_ij = R_i C_j / (1^T R + eps) (0 if that is 0)
//   kPassNorm      kPassPower, plus spart[0] = sum u_i^2
// Shape of the one-pass kernels, measured on the 50257 x 768 report (30
// iterations): 8 waves of 32 rows each (256 rows per workgroup), which
// halves the column partial sums of 4 waves of 32 rows: 1.085-1.089
// against 1.118-1.150 ms (8 waves of 24 rows: 1.52 ms).  With 4 waves,
// 32 rows per wave beat 16 and 64 (1.19 against 1.57 and 1.34 ms).  The
// load of row i + 1 is issued before row i is reduced (more rows ahead
// measured slower: 2 rows 1.19-1.21 ms, 3 rows 1.25, 4 rows 1.30, against
// 1.19 ms, with 4 waves).
#ifndef RK_DIAG_POW_ROWS
#define RK_DIAG_POW_ROWS 256
#endif
#ifndef RK_DIAG_POW_RING
#define RK_DIAG_POW_RING 1
#endif
#ifndef RK_DIAG_POW_WAVES
#define RK_DIAG_POW_WAVES 8
#endif
constexpr int kPowRows = RK_DIAG_POW_ROWS;   // rows per workgroup
constexpr int kPowRing = RK_DIAG_POW_RING;   // rows loaded ahead per wave
constexpr int kPowWaves = RK_DIAG_POW_WAVES; // waves per workgroup
constexpr int kPowThreads = 64 * kPowWaves;
static_assert(kPowRows % kPowWaves == 0, "whole rows per wave");
static_assert(kErrRows <= kPowRows, "the error partials hold one pair per one-pass workgroup");
enum : int { kPassSums = 0, kPassPower = 1, kPassPowerErr = 2, kPassNorm = 3 };

template <int NC, int MODE>
__global__ __launch_bounds__(kPowThreads) void onepass_kernel(
    const float *__restrict__ xi, int64_t m, int64_t n, const double *__restrict__ v,
    const double *__restrict__ vparts, int64_t nvparts, const double *__restrict__ r,
    const double *__restrict__ c, const double *__restrict__ stats_r, double eps,
    double *__restrict__ rout, double *__restrict__ part, double *__restrict__ spart)
{
    constexpr bool kWeighted = MODE != kPassSums;
    constexpr bool kErr = MODE == kPassPowerErr;
    __shared__ double l[kPowWaves][64 * NC];
    __shared__ double ls[kPowWaves][2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const double scale = kWeighted ? inv_norm(vparts, nvparts) : 1.0;
    // Every load below is unconditional, its address clamped into the
    // tensor and its value masked afterwards: loads inside branches make
    // the compiler wait for all outstanding loads before each use, which
    // would empty the ring of row loads at every row.
    double wv[NC], cv[NC], acc[NC];
    int jc[NC];                         // column, clamped into the row
#pragma unroll
    for (int k = 0; k < NC; ++k) {
        const int j = lane + 64 * k;
        jc[k] = j < n ? j : static_cast<int>(n - 1);
        wv[k] = kWeighted ? keep_if(j < n, gp(v)[jc[k]] * scale) : 1.0;
        cv[k] = kErr ? keep_if(j < n, gp(c)[jc[k]]) : 0.0;
        acc[k] = 0.0;
    }
    double inv = 0.0;
    if (kErr) {
        const double denom = gp(stats_r)[1] + eps;
        inv = denom == 0.0 ? 0.0 : 1.0 / denom;
    }
    const int64_t r0 = static_cast<int64_t>(blockIdx.x) * kPowRows + wave * (kPowRows / kPowWaves);
    const int64_t r1 = r0 + kPowRows / kPowWaves < m ? r0 + kPowRows / kPowWaves : m;
    const int64_t rlast = r1 - 1;       // a row of xi (m >= 1), the wave's last if it has rows
    auto load_row = [&](int64_t row, float (&dst)[NC], double &rr) {
        const int64_t rc = row < r1 ? row : rlast;
#pragma unroll
        for (int k = 0; k < NC; ++k)
            dst[k] = keep_if(lane + 64 * k < n && row < r1, gp(xi)[rc * n + jc[k]]);
        if (kErr) rr = keep_if(row < r1, gp(r)[rc] * inv);
    };
    // A ring of kPowRing rows per wave: the loads of row i + kPowRing go out
    // before row i is reduced, so the butterflies overlap the loads.  The
    // ring is refilled unconditionally (rows past the wave's last are
    // clamped and masked), so every wait is for exactly one row.
    float ring[kPowRing][NC];
    double rring[kPowRing] = {};        // row factors (error pass only)
#pragma unroll
    for (int q = 0; q < kPowRing; ++q) load_row(r0 + q, ring[q], rring[q]);
    double sa = 0.0, sb = 0.0;
    for (int64_t i0 = r0; i0 < r1; i0 += kPowRing) {
#pragma unroll
        for (int q = 0; q < kPowRing; ++q) {
            const int64_t i = i0 + q;
            float a[NC];
#pragma unroll
            for (int k = 0; k < NC; ++k) a[k] = ring[q][k];
            const double ri = rring[q];
            load_row(i + kPowRing, ring[q], rring[q]);
            double su = 0.0;
#pragma unroll
            for (int k = 0; k < NC; ++k)
                su += kWeighted ? static_cast<double>(a[k]) * wv[k] : static_cast<double>(a[k]);
            su = wave_sum(su);
            if (i < r1) {
                if (MODE == kPassSums && lane == 0) gp(rout)[i] = su;
#pragma unroll
                for (int k = 0; k < NC; ++k)
                    acc[k] += kWeighted ? static_cast<double>(a[k]) * su : static_cast<double>(a[k]);
                if (kErr) {
#pragma unroll
                    for (int k = 0; k < NC; ++k) {
                        const double x = a[k];
                        const double e = x - ri * cv[k];
                        sa += x * x;
                        sb += e * e;
                    }
                }
                if (MODE == kPassNorm && lane == 0) sa += su * su;
            }
        }
    }
#pragma unroll
    for (int k = 0; k < NC; ++k) l[wave][lane + 64 * k] = acc[k];
    if (kErr || MODE == kPassNorm) {
        sa = wave_sum(sa);
        sb = wave_sum(sb);
        if (lane == 0) {
            ls[wave][0] = sa;
            ls[wave][1] = sb;
        }
    }
    __syncthreads();
    for (int64_t j = threadIdx.x; j < n; j += kPowThreads) {
        double s = l[0][j];
#pragma unroll
        for (int w = 1; w < kPowWaves; ++w) s += l[w][j];
        gp(part)[static_cast<int64_t>(blockIdx.x) * n + j] = s;
    }
    if ((kErr || MODE == kPassNorm) && threadIdx.x == 0) {
        double a = ls[0][0], b = ls[0][1];
#pragma unroll
        for (int w = 1; w < kPowWaves; ++w) {
            a += ls[w][0];
            b += ls[w][1];
        }
        gp(spart)[2 * blockIdx.x] = a;
        gp(spart)[2 * blockIdx.x + 1] = b;
    }
}

// part[s, j] = sum over rows i of stripe s of xi[i, j] * (w ? w[i] : 1).
__global__ __launch_bounds__(kT) void col_partial_kernel(const float *__restrict__ xi, int64_t m,
                                                         int64_t n, int64_t stripe,
                                                         const double *__restrict__ w,
                                                         double *__restrict__ part)
{
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kT + threadIdx.x;
    const int64_t s = blockIdx.y;
    if (j >= n) return;
    const int64_t i0 = s * stripe;
    const int64_t i1 = i0 + stripe < m ? i0 + stripe : m;
    double acc = 0.0;
    // Sixteen rows in flight per thread; additions in row order.
    for (int64_t ib = i0; ib < i1; ib += 16) {
        double v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int64_t i = ib + u;
            const int64_t ic = i < i1 ? i : i1 - 1;       // in the stripe; masked below
            v[u] = keep_if(i < i1, static_cast<double>(gp(xi)[ic * n + j]) * (w ? gp(w)[ic] : 1.0));
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += v[u];
    }
    gp(part)[s * n + j] = acc;
}

// out[j] = sum_s part[s, j]: a workgroup takes kFoldCols columns, its
// kFoldGroups thread groups sum consecutive ranges of stripes in stripe
// order (16 loads in flight, addresses clamped and values masked) and are
// added in group order.  The workgroup also writes parts[2 b] = sum of
// out[j]^2 and parts[2 b + 1] = sum of out[j] over its columns (in column
// order), the partials inv_norm and the statistics use.
__global__ __launch_bounds__(kT) void col_fold_kernel(const double *__restrict__ part, int64_t n,
                                                      int64_t nstripes, double *__restrict__ out,
                                                      double *__restrict__ parts)
{
    __shared__ double l[kT];
    const int c = threadIdx.x % kFoldCols, g = threadIdx.x / kFoldCols;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kFoldCols + c;
    const int64_t jc = j < n ? j : n - 1;
    const int64_t per = (nstripes + kFoldGroups - 1) / kFoldGroups;
    const int64_t s0 = g * per < nstripes ? g * per : nstripes;
    const int64_t s1 = s0 + per < nstripes ? s0 + per : nstripes;
    double acc = 0.0;
    for (int64_t b = s0; b < s1; b += 16) {
        double v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int64_t s = b + u < s1 ? b + u : s1 - 1;
            v[u] = keep_if(b + u < s1 && j < n, gp(part)[s * n + jc]);
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += v[u];
    }
    l[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x < kFoldCols) {
        double v = l[threadIdx.x];
        for (int gg = 1; gg < kFoldGroups; ++gg) v += l[gg * kFoldCols + threadIdx.x];
        l[threadIdx.x] = v;
        if (j < n) gp(out)[j] = v;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double q2 = 0.0, q1 = 0.0;
        for (int cc = 0; cc < kFoldCols; ++cc) {
            const int64_t jj = static_cast<int64_t>(blockIdx.x) * kFoldCols + cc;
            if (jj >= n) break;
            q2 += l[cc] * l[cc];
            q1 += l[cc];
        }
        gp(parts)[2 * blockIdx.x] = q2;
        gp(parts)[2 * blockIdx.x + 1] = q1;
    }
}

// Workgroup b: part[2 b] = sum of v[k]^2 and part[2 b + 1] = sum of v[k]
// over its chunk of kStatChunk elements (fixed order).
__global__ __launch_bounds__(kT) void vec_stats_kernel(const double *__restrict__ v, int64_t k,
                                                       double *__restrict__ part)
{
    __shared__ double l2[kT / 64], l1[kT / 64];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kStatChunk;
    double s2 = 0.0, s1 = 0.0;
#pragma unroll
    for (int u = 0; u < kStatChunk / kT; ++u) {
        const int64_t i = base + u * kT + threadIdx.x;
        const double x = i < k ? gp(v)[i] : 0.0;
        s2 += x * x;
        s1 += x;
    }
    s2 = wave_sum(s2);
    s1 = wave_sum(s1);
    if ((threadIdx.x & 63) == 0) {
        l2[threadIdx.x >> 6] = s2;
        l1[threadIdx.x >> 6] = s1;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int q = 0; q < kT / 64; ++q) {
            a += l2[q];
            b += l1[q];
        }
        gp(part)[2 * blockIdx.x] = a;
        gp(part)[2 * blockIdx.x + 1] = b;
    }
}

// res = the chunk statistics folded in chunk order.
__global__ void stats_fold_kernel(const double *__restrict__ part, int64_t nchunks,
                                  double *__restrict__ res)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int64_t q = 0; q < nchunks; ++q) {
            a += gp(part)[2 * q];
            b += gp(part)[2 * q + 1];
        }
        gp(res)[0] = a;
        gp(res)[1] = b;
    }
}

// Per workgroup of kErrRows rows: sum xi^2 and sum (xi - R_i C_j / (S + eps))^2
// with S = stats_r[1] (the sum of R) and xi~ = 0 when S + eps == 0.  A
// thread takes columns j = t, t + 256, ...; for each it loads the column's
// kErrRows entries together (rows clamped into the tensor and masked) and
// adds them in row order.
__global__ __launch_bounds__(kT) void err_partial_kernel(const float *__restrict__ xi, int64_t m,
                                                         int64_t n, const double *__restrict__ r,
                                                         const double *__restrict__ c,
                                                         const double *__restrict__ stats_r,
                                                         double eps, double *__restrict__ part)
{
    __shared__ double la[kT / 64], lb[kT / 64];
    const double denom = gp(stats_r)[1] + eps;
    const double inv = denom == 0.0 ? 0.0 : 1.0 / denom;
    const int64_t i0 = static_cast<int64_t>(blockIdx.x) * kErrRows;
    const int64_t i1 = i0 + kErrRows < m ? i0 + kErrRows : m;
    double ri[kErrRows];
    int64_t ic[kErrRows];
#pragma unroll
    for (int u = 0; u < kErrRows; ++u) {
        ic[u] = i0 + u < i1 ? i0 + u : i1 - 1;
        ri[u] = keep_if(i0 + u < i1, gp(r)[ic[u]] * inv);
    }
    double sa = 0.0, sb = 0.0;
    for (int64_t j = threadIdx.x; j < n; j += kT) {
        const double cj = gp(c)[j];
        float v[kErrRows];
#pragma unroll
        for (int u = 0; u < kErrRows; ++u) v[u] = keep_if(i0 + u < i1, gp(xi)[ic[u] * n + j]);
#pragma unroll
        for (int u = 0; u < kErrRows; ++u) {
            const double x = v[u];
            const double e = x - ri[u] * cj;
            sa += x * x;
            sb += e * e;
        }
    }
    sa = wave_sum(sa);
    sb = wave_sum(sb);
    if ((threadIdx.x & 63) == 0) {
        la[threadIdx.x >> 6] = sa;
        lb[threadIdx.x >> 6] = sb;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int q = 0; q < kT / 64; ++q) {
            a += la[q];
            b += lb[q];
        }
        gp(part)[2 * blockIdx.x] = a;
        gp(part)[2 * blockIdx.x + 1] = b;
    }
}

// res[0] = sum of part[2 k], res[1] = sum of part[2 k + 1]: thread t sums
// k = t, t + 256, ... in order, then the threads are combined in a fixed
// order (butterfly in each wave, waves in order).
__global__ __launch_bounds__(kT) void err_fold_kernel(const double *__restrict__ part, int64_t nblk,
                                                      double *__restrict__ res)
{
    __shared__ double la[kT / 64], lb[kT / 64];
    double a = 0.0, b = 0.0;
    for (int64_t q = threadIdx.x; q < nblk; q += kT) {
        a += gp(part)[2 * q];
        b += gp(part)[2 * q + 1];
    }
    a = wave_sum(a);
    b = wave_sum(b);
    if ((threadIdx.x & 63) == 0) {
        la[threadIdx.x >> 6] = a;
        lb[threadIdx.x >> 6] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double x = la[0], y = lb[0];
        for (int w = 1; w < kT / 64; ++w) {
            x += la[w];
            y += lb[w];
        }
        gp(res)[0] = x;
        gp(res)[1] = y;
    }
}

struct DevBuf {
    void *p = nullptr;
    ~DevBuf()
    {
        if (p) (void)hipFree(p);
    }
};

// Workspace of one report, in doubles, and the launch geometry it implies.
struct ReportShape {
    int64_t stripe, nstripes, ncb, nerr, nfold, nstat, nblk, nparts, words;
    int nc;   // registers per lane of the one-pass power iteration (0: two passes)
};

ReportShape report_shape(int64_t m, int64_t n)
{
    ReportShape s;
    // Stripe height: the largest power of two in [16, 1024] that still gives
    // the column pass about eight workgroups per compute unit, raised if the
    // stripe count would pass the grid's y limit.
    s.ncb = (n + kT - 1) / kT;
    s.stripe = 1024;
    while (s.stripe > 16 && s.ncb * ((m + s.stripe - 1) / s.stripe) < 2048) s.stripe >>= 1;
    while ((m + s.stripe - 1) / s.stripe > 65535) s.stripe <<= 1;
    s.nstripes = (m + s.stripe - 1) / s.stripe;
    s.nerr = (m + kErrRows - 1) / kErrRows;
    s.nfold = (n + kFoldCols - 1) / kFoldCols;
    const int64_t mk = m > n ? m : n;
    s.nstat = (mk + kStatChunk - 1) / kStatChunk;
    // n <= 1024: xi's rows fit the registers of a wave, and every pass over
    // xi is one onepass_kernel launch
    s.nc = n <= 256 ? 4 : n <= 512 ? 8 : n <= 768 ? 12 : n <= 1024 ? 16 : 0;
    s.nblk = (m + kPowRows - 1) / kPowRows;
    s.nparts = s.nc ? s.nblk : s.nstripes;
    // r m, c n, u m, v n, column partials nparts*n, error partials 2*nerr,
    // fold partials 2*nfold (C) and 2*nfold (v), statistics partials
    // 2*nstat, results 2 (R), 2 (u), 2 (errors)
    s.words = m + n + m + n + s.nparts * n + 2 * s.nerr + 4 * s.nfold + 2 * s.nstat + 6;
    return s;
}

rikfad_status check_report_args(const float *xi, int64_t m, int64_t n, double eps_stab,
                                int32_t power_iters, const rikfad_friction_stats *out)
{
    if (!xi || !out || m < 1 || n < 1 || m >= (int64_t(1) << 31) || n >= (int64_t(1) << 31) ||
        power_iters < 1 || power_iters > 10000 || !(eps_stab >= 0.0) || !std::isfinite(eps_stab)) {
        rk::set_last_error("friction_report: NULL pointer, m or n outside [1, 2^31), "
                           "power_iters outside [1, 10000] or eps_stab negative / not finite");
        return RIKFAD_EINVAL;
    }
    if (reinterpret_cast<uintptr_t>(xi) % 4 != 0) {
        rk::set_last_error("friction_report: xi is not 4-byte aligned");
        return RIKFAD_EALIGN;
    }
    return RIKFAD_OK;
}

template <int MODE, typename... Args>
void launch_onepass(int nc, dim3 grid, hipStream_t st, Args... args)
{
    if (nc == 4)
        hipLaunchKernelGGL((onepass_kernel<4, MODE>), grid, dim3(kPowThreads), 0, st, args...);
    else if (nc == 8)
        hipLaunchKernelGGL((onepass_kernel<8, MODE>), grid, dim3(kPowThreads), 0, st, args...);
    else if (nc == 12)
        hipLaunchKernelGGL((onepass_kernel<12, MODE>), grid, dim3(kPowThreads), 0, st, args...);
    else
        hipLaunchKernelGGL((onepass_kernel<16, MODE>), grid, dim3(kPowThreads), 0, st, args...);
}

// The report itself on a workspace of sh.words doubles at buf (device
// memory).  Every word of the workspace that a kernel reads was written
// earlier in the same call, so its previous contents do not matter.
rikfad_status report_on(const float *xi, int64_t m, int64_t n, double eps_stab,
                        int32_t power_iters, hipStream_t st, const ReportShape &sh, double *buf,
                        rikfad_friction_stats *out)
{
    const int64_t stripe = sh.stripe, nstripes = sh.nstripes, nerr = sh.nerr;
    const int64_t nfold = sh.nfold, nblk = sh.nblk, nparts = sh.nparts;
    const int nc = sh.nc;
    double *r = buf, *c = r + m, *u = c + n, *v = u + m;
    double *cpart = v + n, *epart = cpart + nparts * n, *cfold = epart + 2 * nerr;
    double *vfold = cfold + 2 * nfold, *spart = vfold + 2 * nfold;
    double *stats_r = spart + 2 * sh.nstat, *stats_u = stats_r + 2, *err = stats_u + 2;
    const dim3 rows_grid(static_cast<uint32_t>((m + kT / 64 - 1) / (kT / 64)));
    const dim3 cols_grid(static_cast<uint32_t>(sh.ncb), static_cast<uint32_t>(nstripes));
    const dim3 fold_grid(static_cast<uint32_t>(nfold));
    auto stats = [&](const double *vec, int64_t k, double *res) {
        const int64_t nch = (k + kStatChunk - 1) / kStatChunk;
        hipLaunchKernelGGL(vec_stats_kernel, dim3(static_cast<uint32_t>(nch)), dim3(kT), 0, st,
                           vec, k, spart);
        hipLaunchKernelGGL(stats_fold_kernel, dim3(1), dim3(1), 0, st, spart, nch, res);
    };

    if (nc) {
        // n <= 1024: iters + 2 passes over xi.  The first forms R = xi 1 and
        // C = xi^T 1; the first power iteration (from v = C / |C|) also sums
        // |xi|_F^2 and |xi - xi~|_F^2; the last pass forms |xi v| for the
        // final unit vector v.
        const dim3 grid(static_cast<uint32_t>(nblk));
        launch_onepass<kPassSums>(nc, grid, st, xi, m, n, nullptr, nullptr, 0, nullptr, nullptr,
                                  nullptr, 0.0, r, cpart, nullptr);
        hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nblk, c, cfold);
        stats(r, m, stats_r);
        const double *vin = c, *vin_fold = cfold;
        for (int it = 0; it < power_iters; ++it) {
            if (it == 0) {
                launch_onepass<kPassPowerErr>(nc, grid, st, xi, m, n, vin, vin_fold, nfold, r, c,
                                              stats_r, eps_stab, nullptr, cpart, epart);
                hipLaunchKernelGGL(err_fold_kernel, dim3(1), dim3(kT), 0, st, epart, nblk, err);
            } else {
                launch_onepass<kPassPower>(nc, grid, st, xi, m, n, vin, vin_fold, nfold, nullptr,
                                           nullptr, nullptr, 0.0, nullptr, cpart, nullptr);
            }
            hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nblk, v,
                               vfold);
            vin = v;
            vin_fold = vfold;
        }
        launch_onepass<kPassNorm>(nc, grid, st, xi, m, n, vin, vin_fold, nfold, nullptr, nullptr,
                                  nullptr, 0.0, nullptr, cpart, epart);
        hipLaunchKernelGGL(err_fold_kernel, dim3(1), dim3(kT), 0, st, epart, nblk, stats_u);
    } else {
        // Shadow factors R = xi 1, C = xi^T 1 and the sum of R.
        hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, nullptr,
                           nullptr, int64_t(0), r);
        hipLaunchKernelGGL(col_partial_kernel, cols_grid, dim3(kT), 0, st, xi, m, n, stripe,
                           nullptr, cpart);
        hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nstripes, c,
                           cfold);
        stats(r, m, stats_r);
        // |xi|_F^2 and |xi - xi~|_F^2
        hipLaunchKernelGGL(err_partial_kernel, dim3(static_cast<uint32_t>(nerr)), dim3(kT), 0, st,
                           xi, m, n, r, c, stats_r, eps_stab, epart);
        hipLaunchKernelGGL(err_fold_kernel, dim3(1), dim3(kT), 0, st, epart, nerr, err);
        // Power iteration on xi^T xi from v = C / |C|: u = xi v / |v|,
        // v <- xi^T u; each row pass normalises its input from the fold
        // partials of the last column pass.
        const double *vin = c, *vin_fold = cfold;
        for (int it = 0; it < power_iters; ++it) {
            hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, vin,
                               vin_fold, nfold, u);
            hipLaunchKernelGGL(col_partial_kernel, cols_grid, dim3(kT), 0, st, xi, m, n, stripe,
                               u, cpart);
            hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nstripes,
                               v, vfold);
            vin = v;
            vin_fold = vfold;
        }
        // sigma_1 = |xi v| for the final unit vector v.
        hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, vin,
                           vin_fold, nfold, u);
        stats(u, m, stats_u);
    }
    // stats_r, stats_u and err are adjacent: one copy brings all three back
    // (host[] keeps the order R, errors, u).
    hipError_t e = hipGetLastError();
    double res[6];
    if (e == hipSuccess) e = hipMemcpyAsync(res, stats_r, sizeof(res), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    const double host[6] = {res[0], res[1], res[4], res[5], res[2], res[3]};
    if (e != hipSuccess) {
        rk::set_last_error((std::string("friction_report: ") + hipGetErrorString(e)).c_str());
        return RIKFAD_EHIP;
    }
    const double fro2 = host[2], err2 = host[3], sigma1_sq = host[4];
    out->xi_fro2 = fro2;
    out->err_fro2 = err2;
    out->sum_r = host[1];
    out->sigma1 = std::sqrt(sigma1_sq);
    out->rel_err = fro2 > 0.0 ? std::sqrt(err2 / fro2) : 0.0;
    const double ratio = fro2 > 0.0 ? sigma1_sq / fro2 : 1.0;
    out->eckart_young_floor = std::sqrt(ratio < 1.0 ? 1.0 - ratio : 0.0);
    out->stable_rank = sigma1_sq > 0.0 ? fro2 / sigma1_sq : 0.0;
    out->power_iters = power_iters;
    out->reserved = 0;
    return RIKFAD_OK;
}

// ------------------------------------------------ report without allocation
//
// A file-scope device array is the workspace of rikfad_friction_report_noalloc.
// Each device holds its own copy at its own address, which host code must
// obtain with hipGetSymbolAddress (the array's name in host code is only a
// stand-in for the symbol, not a device address).  The address is looked up
// once per device, with that device current, on the first call there.
constexpr int64_t kScratchWords = int64_t(1) << 21;    // 16 MiB of doubles

}  // namespace

static __device__ __align__(256) double scratch[kScratchWords];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double *g_scratch_ptr[kMaxDevices] = {};

rikfad_status scratch_of_current_device(double **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        rk::set_last_error((std::string("friction_report_noalloc: hipGetDevice: ") +
                            hipGetErrorString(e)).c_str());
        return RIKFAD_EHIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        rk::set_last_error("friction_report_noalloc: device index beyond 63");
        return RIKFAD_EINVAL;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            rk::set_last_error((std::string("friction_report_noalloc: hipGetSymbolAddress: ") +
                                hipGetErrorString(e)).c_str());
            return RIKFAD_EHIP;
        }
        g_scratch_ptr[dev] = static_cast<double *>(p);
    }
    *out = g_scratch_ptr[dev];
    return RIKFAD_OK;
}

}  // namespace

extern "C" rikfad_status rikfad_friction_report(const float *xi, int64_t m, int64_t n,
                                                double eps_stab, int32_t power_iters,
                                                void *stream_, rikfad_friction_stats *out)
{
    rikfad_status s = check_report_args(xi, m, n, eps_stab, power_iters, out);
    if (s != RIKFAD_OK) return s;
    const ReportShape sh = report_shape(m, n);
    DevBuf buf;
    if (hipMalloc(&buf.p, sizeof(double) * static_cast<size_t>(sh.words)) != hipSuccess) {
        rk::set_last_error("friction_report: hipMalloc of the workspace failed");
        return RIKFAD_ENOMEM;
    }
    return report_on(xi, m, n, eps_stab, power_iters, static_cast<hipStream_t>(stream_), sh,
                     static_cast<double *>(buf.p), out);
}

extern "C" int64_t rikfad_friction_report_noalloc_max_bytes(void)
{
    return kScratchWords * static_cast<int64_t>(sizeof(double));
}

extern "C" int64_t rikfad_friction_report_workspace_bytes(int64_t m, int64_t n)
{
    if (m < 1 || n < 1 || m >= (int64_t(1) << 31) || n >= (int64_t(1) << 31)) return -1;
    return report_shape(m, n).words * static_cast<int64_t>(sizeof(double));
}

extern "C" rikfad_status rikfad_friction_report_noalloc(const float *xi, int64_t m, int64_t n,
                                                        double eps_stab, int32_t power_iters,
                                                        void *stream_,
                                                        rikfad_friction_stats *out)
{
    rikfad_status s = check_report_args(xi, m, n, eps_stab, power_iters, out);
    if (s != RIKFAD_OK) return s;
    const ReportShape sh = report_shape(m, n);
    if (sh.words > kScratchWords) {
        rk::set_last_error(("friction_report_noalloc: an " + std::to_string(m) + " x " +
                            std::to_string(n) + " tensor needs " +
                            std::to_string(sh.words * 8) + " bytes of workspace, more than the " +
                            std::to_string(kScratchWords * 8) + "-byte static scratch")
                               .c_str());
        return RIKFAD_EINVAL;
    }
    double *ws = nullptr;
    if ((s = scratch_of_current_device(&ws)) != RIKFAD_OK) return s;
    return report_on(xi, m, n, eps_stab, power_iters, static_cast<hipStream_t>(stream_), sh, ws,
                     out);
}
