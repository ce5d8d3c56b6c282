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
// so the leading singular vectors are non-negative), normalised on the GPU.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cmath>

#include "../../include/rikfad.h"

namespace {

constexpr int kT = 256;            // threads per workgroup
constexpr int kStatChunk = 4096;   // elements per workgroup of the vector statistics
constexpr int kErrRows = 16;       // rows per workgroup of the error pass

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

// out[i] = sum_j xi[i, j] * (w ? w[j] * (*wscale) : 1): one wave per row,
// lanes stride over the columns, fp64 accumulation.
__global__ __launch_bounds__(kT) void row_reduce_kernel(const float *__restrict__ xi, int64_t m,
                                                        int64_t n, const double *__restrict__ w,
                                                        const double *__restrict__ wscale,
                                                        double *__restrict__ out)
{
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (kT / 64) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= m) return;
    const DG float *xr = gp(xi) + row * n;
    double s = 0.0;
    // Eight loads in flight per lane; additions in column order.
    for (int64_t j0 = lane; j0 < n; j0 += 64 * 8) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t j = j0 + 64 * u;
            v[u] = j < n ? static_cast<double>(xr[j]) * (w ? gp(w)[j] : 1.0) : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) s += v[u];
    }
    s = wave_sum(s);
    if (lane == 0) gp(out)[row] = w ? s * gp(wscale)[0] : s;
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
            v[u] = i < i1 ? static_cast<double>(gp(xi)[i * n + j]) * (w ? gp(w)[i] : 1.0) : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += v[u];
    }
    gp(part)[s * n + j] = acc;
}

// out[j] = (sum_s part[s, j]) * (wscale ? *wscale : 1), stripes in order.
__global__ __launch_bounds__(kT) void col_fold_kernel(const double *__restrict__ part, int64_t n,
                                                      int64_t nstripes,
                                                      const double *__restrict__ wscale,
                                                      double *__restrict__ out)
{
    const int64_t j = static_cast<int64_t>(blockIdx.x) * kT + threadIdx.x;
    if (j >= n) return;
    double acc = 0.0;
    for (int64_t s0 = 0; s0 < nstripes; s0 += 16) {
        double v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = s0 + u < nstripes ? gp(part)[(s0 + u) * n + j] : 0.0;
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += v[u];
    }
    gp(out)[j] = wscale ? acc * gp(wscale)[0] : acc;
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

// res = the chunk statistics folded in chunk order; scale = 1 / sqrt(res[0])
// (0 for a zero vector) when scale is given.
__global__ void stats_fold_kernel(const double *__restrict__ part, int64_t nchunks,
                                  double *__restrict__ res, double *__restrict__ scale)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int64_t q = 0; q < nchunks; ++q) {
            a += gp(part)[2 * q];
            b += gp(part)[2 * q + 1];
        }
        gp(res)[0] = a;
        gp(res)[1] = b;
        if (scale) gp(scale)[0] = a > 0.0 ? 1.0 / sqrt(a) : 0.0;
    }
}

// Per workgroup of kErrRows rows: sum xi^2 and sum (xi - R_i C_j / (S + eps))^2
// with S = stats_r[1] (the sum of R) and xi~ = 0 when S + eps == 0.
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
    double sa = 0.0, sb = 0.0;
    for (int64_t i = i0; i < i1; ++i) {
        const double ri = gp(r)[i] * inv;
        for (int64_t j = threadIdx.x; j < n; j += kT) {
            const double v = gp(xi)[i * n + j];
            const double d = v - ri * gp(c)[j];
            sa += v * v;
            sb += d * d;
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

// res[0] = sum of part[2 k], res[1] = sum of part[2 k + 1], in k order.
__global__ void err_fold_kernel(const double *__restrict__ part, int64_t nblk,
                                double *__restrict__ res)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double a = 0.0, b = 0.0;
        for (int64_t q = 0; q < nblk; ++q) {
            a += gp(part)[2 * q];
            b += gp(part)[2 * q + 1];
        }
        gp(res)[0] = a;
        gp(res)[1] = b;
    }
}

struct DevBuf {
    void *p = nullptr;
    ~DevBuf()
    {
        if (p) (void)hipFree(p);
    }
};

}  // namespace

extern "C" rikfad_status rikfad_friction_report(const float *xi, int64_t m, int64_t n,
                                                double eps_stab, int32_t power_iters,
                                                void *stream_, rikfad_friction_stats *out)
{
    if (!xi || !out || m < 1 || n < 1 || m >= (int64_t(1) << 31) || n >= (int64_t(1) << 31) ||
        power_iters < 1 || power_iters > 10000 || !(eps_stab >= 0.0) || !std::isfinite(eps_stab))
        return RIKFAD_EINVAL;
    if (reinterpret_cast<uintptr_t>(xi) % 4 != 0) return RIKFAD_EALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream_);
    // Stripe height: the largest power of two in [16, 1024] that still gives
    // the column pass about eight workgroups per compute unit, raised if the
    // stripe count would pass the grid's y limit.
    const int64_t ncb = (n + kT - 1) / kT;
    int64_t stripe = 1024;
    while (stripe > 16 && ncb * ((m + stripe - 1) / stripe) < 2048) stripe >>= 1;
    while ((m + stripe - 1) / stripe > 65535) stripe <<= 1;
    const int64_t nstripes = (m + stripe - 1) / stripe;
    const int64_t nerr = (m + kErrRows - 1) / kErrRows;
    const int64_t mk = m > n ? m : n;
    const int64_t nstat = (mk + kStatChunk - 1) / kStatChunk;
    // workspace (doubles): r m, c n, u m, v n, colpart nstripes*n, errpart 2*nerr,
    // statpart 2*nstat, stats 2 (r), 2 (v), 2 (u), 2 (err), scale 1
    const int64_t words = m + n + m + n + nstripes * n + 2 * nerr + 2 * nstat + 9;
    DevBuf buf;
    if (hipMalloc(&buf.p, sizeof(double) * static_cast<size_t>(words)) != hipSuccess)
        return RIKFAD_ENOMEM;
    double *r = static_cast<double *>(buf.p), *c = r + m, *u = c + n, *v = u + m;
    double *cpart = v + n, *epart = cpart + nstripes * n, *spart = epart + 2 * nerr;
    double *stats_r = spart + 2 * nstat, *stats_v = stats_r + 2, *stats_u = stats_v + 2;
    double *err = stats_u + 2, *scale_v = err + 2;
    const dim3 rows_grid(static_cast<uint32_t>((m + kT / 64 - 1) / (kT / 64)));
    const dim3 cols_grid(static_cast<uint32_t>(ncb), static_cast<uint32_t>(nstripes));
    const dim3 fold_grid(static_cast<uint32_t>((n + kT - 1) / kT));
    auto stats = [&](const double *vec, int64_t k, double *res, double *scale) {
        const int64_t nc = (k + kStatChunk - 1) / kStatChunk;
        hipLaunchKernelGGL(vec_stats_kernel, dim3(static_cast<uint32_t>(nc)), dim3(kT), 0, st, vec,
                           k, spart);
        hipLaunchKernelGGL(stats_fold_kernel, dim3(1), dim3(1), 0, st, spart, nc, res, scale);
    };

    // Shadow factors R = xi 1, C = xi^T 1 and their totals.
    hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, nullptr, nullptr, r);
    hipLaunchKernelGGL(col_partial_kernel, cols_grid, dim3(kT), 0, st, xi, m, n, stripe, nullptr,
                       cpart);
    hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nstripes, nullptr, c);
    stats(r, m, stats_r, nullptr);
    // |xi|_F^2 and |xi - xi~|_F^2
    hipLaunchKernelGGL(err_partial_kernel, dim3(static_cast<uint32_t>(nerr)), dim3(kT), 0, st, xi,
                       m, n, r, c, stats_r, eps_stab, epart);
    hipLaunchKernelGGL(err_fold_kernel, dim3(1), dim3(1), 0, st, epart, nerr, err);
    // Power iteration on xi^T xi from v = C / |C|: u = xi v, v <- xi^T u / |xi^T u|.
    stats(c, n, stats_v, scale_v);
    const double *vin = c;
    for (int it = 0; it < power_iters; ++it) {
        hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, vin, scale_v, u);
        hipLaunchKernelGGL(col_partial_kernel, cols_grid, dim3(kT), 0, st, xi, m, n, stripe, u,
                           cpart);
        hipLaunchKernelGGL(col_fold_kernel, fold_grid, dim3(kT), 0, st, cpart, n, nstripes,
                           nullptr, v);
        stats(v, n, stats_v, scale_v);
        vin = v;
    }
    // sigma_1 = |xi v| for the final unit vector v.
    hipLaunchKernelGGL(row_reduce_kernel, rows_grid, dim3(kT), 0, st, xi, m, n, vin, scale_v, u);
    stats(u, m, stats_u, nullptr);
    if (hipGetLastError() != hipSuccess) return RIKFAD_EHIP;
    double host[6];
    if (hipMemcpyAsync(host, stats_r, sizeof(double) * 2, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipMemcpyAsync(host + 2, err, sizeof(double) * 2, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipMemcpyAsync(host + 4, stats_u, sizeof(double) * 2, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
        return RIKFAD_EHIP;
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
