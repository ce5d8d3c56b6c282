// kernels.hip -- gfx950 kernels of the R-iKFAD optimiser step.
//
// Step of Section 2 ("Splitting Discretization") / App. A (Table of
// analytical sub-step updates), in the deferred form: the second friction
// half-kick of step n and the first of step n+1 use the same factors
// (R_{n+1}, C_{n+1}), so one streaming pass per step applies both with a
// single exponential per element:
//
//   E     = exp(-(h/2) R_i C_j / (1^T R + eps))     rank-1 friction, eq. (xi_def)
//   P_n   = d (Q .* E)          pending C.4 + D of the previous step (Q = its P^(1))
//   P^(B) = P_n - h g                                 B
//   X'    = X + h P^(B)                               A
//   P^(1) = P^(B) .* E                                C.1, stored in p
//   row / column partial sums of [P^(1)]^2            C.2 / C.3, stage 1
//
// followed by a small finalisation pass (C.2 / C.3 stage 2 and 1^T R).
// The step is HBM-bound (about half a flop per byte), so there is no MFMA:
// the kernels are organised around coalesced 128-bit loads, register
// accumulation of column sums, wavefront shuffles for row sums, and a
// fixed-order combine through LDS.  No atomics: every sum has a fixed order,
// so results are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"
#include "layout.hpp"

namespace rk {

// All tensors live in global memory.  The pointers arrive through tables,
// so the compiler cannot prove their address space; casting them to the
// global address space selects global_load/global_store instead of flat
// accesses.
#define RK_GLOBAL __attribute__((address_space(1)))

template <typename T>
__device__ __forceinline__ const RK_GLOBAL T *gmem(const T *q)
{
    return (const RK_GLOBAL T *)q;
}
template <typename T>
__device__ __forceinline__ RK_GLOBAL T *gmem(T *q)
{
    return (RK_GLOBAL T *)q;
}

// Native clang vectors (the HIP float4 class cannot bind to an
// address-space-qualified reference).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ bf16

__device__ __forceinline__ float bf16_to_f32(uint16_t b)
{
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even; NaN stays a (quiet) NaN, overflow -> inf.
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// ------------------------------------------------------- vector accesses
// Io<T, V>: V consecutive elements of storage type T as fp32 registers.

template <typename T, int V> struct Io;

template <> struct Io<float, 4> {
    static __device__ __forceinline__ void load(const float *q, float (&o)[4])
    {
        const f32x4 v = *gmem(reinterpret_cast<const f32x4 *>(q));
        o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
    }
    static __device__ __forceinline__ void store(float *q, const float (&o)[4])
    {
        *gmem(reinterpret_cast<f32x4 *>(q)) = f32x4{o[0], o[1], o[2], o[3]};
    }
};

template <> struct Io<float, 8> {
    static __device__ __forceinline__ void load(const float *q, float (&o)[8])
    {
        const f32x4 a = gmem(reinterpret_cast<const f32x4 *>(q))[0];
        const f32x4 b = gmem(reinterpret_cast<const f32x4 *>(q))[1];
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
        o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
    static __device__ __forceinline__ void store(float *q, const float (&o)[8])
    {
        gmem(reinterpret_cast<f32x4 *>(q))[0] = f32x4{o[0], o[1], o[2], o[3]};
        gmem(reinterpret_cast<f32x4 *>(q))[1] = f32x4{o[4], o[5], o[6], o[7]};
    }
};

template <> struct Io<float, 1> {
    static __device__ __forceinline__ void load(const float *q, float (&o)[1]) { o[0] = *gmem(q); }
    static __device__ __forceinline__ void store(float *q, const float (&o)[1]) { *gmem(q) = o[0]; }
};

template <> struct Io<uint16_t, 8> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[8])
    {
        const u32x4 v = *gmem(reinterpret_cast<const u32x4 *>(q));
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __uint_as_float(w[i] << 16);
            o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    static __device__ __forceinline__ void store(uint16_t *q, const float (&o)[8])
    {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = static_cast<uint32_t>(f32_to_bf16(o[2 * i])) |
                   (static_cast<uint32_t>(f32_to_bf16(o[2 * i + 1])) << 16);
        *gmem(reinterpret_cast<u32x4 *>(q)) = u32x4{w[0], w[1], w[2], w[3]};
    }
};

template <> struct Io<uint16_t, 4> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[4])
    {
        const u32x2 v = *gmem(reinterpret_cast<const u32x2 *>(q));
        o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
        o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
    }
    static __device__ __forceinline__ void store(uint16_t *q, const float (&o)[4])
    {
        const uint32_t a = static_cast<uint32_t>(f32_to_bf16(o[0])) |
                           (static_cast<uint32_t>(f32_to_bf16(o[1])) << 16);
        const uint32_t b = static_cast<uint32_t>(f32_to_bf16(o[2])) |
                           (static_cast<uint32_t>(f32_to_bf16(o[3])) << 16);
        *gmem(reinterpret_cast<u32x2 *>(q)) = u32x2{a, b};
    }
};

template <> struct Io<uint16_t, 1> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[1]) { o[0] = bf16_to_f32(*gmem(q)); }
    static __device__ __forceinline__ void store(uint16_t *q, const float (&o)[1]) { *gmem(q) = f32_to_bf16(o[0]); }
};

// ---------------------------------------------------------- reductions

// Sum of the partial sums of R written by the finalisation pass.  Every
// wave of every workgroup of a tensor evaluates the same expression in the
// same order, so all of them obtain the same bits.
__device__ __forceinline__ float sum_r(const float *__restrict__ part, int count)
{
    const int lane = threadIdx.x & (kWave - 1);
    float s = 0.f;
    for (int i = lane; i < count; i += kWave) s += gmem(part)[i];
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) s += __shfl_xor(s, o);
    return s;
}

// kh * R_i / (1^T R + eps), or 0 where the denominator vanishes (the
// eps_stab = 0 convention at 1^T R = 0).  exp2(this * C_j) is the half-kick.
__device__ __forceinline__ float row_rate(float kh, float r_i, float denom)
{
    return denom == 0.f ? 0.f : kh * (r_i / denom);
}

// ------------------------------------------------ streaming pass (matrix)
//
// A tile is kStripeRows rows x one column block.  Each wave walks
// kRowsPerWave consecutive rows; a row of the block is covered by L lanes
// (L = 64 for wide blocks; narrow blocks put 64/L rows in one load), each
// lane owning V consecutive columns.  Column sums accumulate in the lane's
// registers while it walks down the rows; row sums are reduced across the
// L lanes of a row with xor shuffles and parked in lane (row - first row).

template <typename XT, int V>
__device__ void stream_matrix(const TensorDesc &td, const XT *__restrict__ g,
                              const Tile &tile, float *__restrict__ ws,
                              const Coeffs &k, int pending, float *lds)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int llog = tile.lanes_log2;
    const int L = 1 << llog;
    const int G = kWave >> llog;                  // rows per load
    const int seg = lane >> llog;
    const int sl = lane & (L - 1);
    const int64_t n = td.n;
    const int ccol = sl * V;
    const bool colok = ccol < tile.ncols;
    const int64_t col = tile.col0 + ccol;

    float cv[V];
#pragma unroll
    for (int i = 0; i < V; ++i) cv[i] = colok ? gmem(td.c)[col + i] : 0.f;

    const float denom = sum_r(ws + td.chunk, td.nchunk) + k.eps;
    const int64_t r0 = tile.start + static_cast<int64_t>(wave) * kRowsPerWave;
    const int nr = max(0, min(kRowsPerWave, static_cast<int>(tile.start + tile.count - r0)));
    const float myrate = lane < nr ? row_rate(k.kh, gmem(td.r)[r0 + lane], denom) : 0.f;

    XT *__restrict__ x = static_cast<XT *>(td.x);
    float *__restrict__ p = td.p;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
    float myrow = 0.f;

    const int nld = (nr + G - 1) >> (6 - llog);
    for (int ld = 0; ld < nld; ++ld) {
        const int rl = ld * G + seg;
        const bool ok = colok && rl < nr;
        const float rate = __shfl(myrate, rl & (kWave - 1));
        const int64_t off = (r0 + rl) * n + col;
        float xv[V], gv[V], qv[V];
        if (ok) {
            Io<XT, V>::load(x + off, xv);
            Io<XT, V>::load(g + off, gv);
            Io<float, V>::load(p + off, qv);
        } else {
#pragma unroll
            for (int i = 0; i < V; ++i) xv[i] = gv[i] = qv[i] = 0.f;
        }
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const float e = exp2f(rate * cv[i]);
            const float pn = pending ? k.d * (qv[i] * e) : qv[i];
            const float pb = pn - k.h * gv[i];
            xv[i] = xv[i] + k.h * pb;
            const float p1 = pb * e;
            qv[i] = p1;
            const float s = ok ? p1 * p1 : 0.f;
            acc[i] += s;
            rs += s;
        }
        if (ok) {
            Io<XT, V>::store(x + off, xv);
            Io<float, V>::store(p + off, qv);
        }
        for (int o = 1; o < L; o <<= 1) rs += __shfl_xor(rs, o);
        const float v = __shfl(rs, ((lane - ld * G) & (G - 1)) << llog);
        if (lane >= ld * G && lane < ld * G + G) myrow = v;
    }

    // Lanes l and l ^ o (o >= L) own the same columns: fold them, then fold
    // the four waves through LDS in wave order.
    for (int o = L; o < kWave; o <<= 1) {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += __shfl_xor(acc[i], o);
    }
    if (seg == 0 && colok) {
#pragma unroll
        for (int i = 0; i < V; ++i) lds[wave * kWave * V + ccol + i] = acc[i];
    }
    __syncthreads();
    float *colpart = ws + td.colpart + static_cast<int64_t>(tile.stripe) * n + tile.col0;
    for (int j = threadIdx.x; j < tile.ncols; j += kThreads) {
        const float s = ((lds[j] + lds[kWave * V + j]) + lds[2 * kWave * V + j]) +
                        lds[3 * kWave * V + j];
        gmem(colpart)[j] = s;
    }
    if (lane < nr) gmem(ws)[td.rowpart + static_cast<int64_t>(tile.cb) * td.m + r0 + lane] = myrow;
}

// ------------------------------------------- element-wise iKFAD (vectors)
//
// Each entry carries its own friction xi: half-kick with xi_n, exact
// friction update driven by P^(1), half-kick with xi_{n+1}, then D.

template <typename XT, int V>
__device__ __forceinline__ void ikfad_elems(XT *__restrict__ x, const XT *__restrict__ g,
                                            float *__restrict__ p, float *__restrict__ xi,
                                            const Coeffs &k)
{
    float xv[V], gv[V], pv[V], fv[V];
    Io<XT, V>::load(x, xv);
    Io<XT, V>::load(g, gv);
    Io<float, V>::load(p, pv);
    Io<float, V>::load(xi, fv);
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const float pb = pv[i] - k.h * gv[i];
        xv[i] = xv[i] + k.h * pb;
        const float p1 = pb * exp2f(k.kh * fv[i]);
        fv[i] = k.a * fv[i] + k.kappa * (p1 * p1);
        pv[i] = k.d * (p1 * exp2f(k.kh * fv[i]));
    }
    Io<XT, V>::store(x, xv);
    Io<float, V>::store(p, pv);
    Io<float, V>::store(xi, fv);
}

template <typename XT, int V>
__device__ void elementwise_range(XT *__restrict__ x, const XT *__restrict__ g,
                                  float *__restrict__ p, float *__restrict__ xi,
                                  int64_t start, int count, const Coeffs &k)
{
    const int full = count - count % V;
    for (int e = threadIdx.x * V; e < full; e += kThreads * V) {
        const int64_t o = start + e;
        ikfad_elems<XT, V>(x + o, g + o, p + o, xi + o, k);
    }
    for (int e = full + threadIdx.x; e < count; e += kThreads) {
        const int64_t o = start + e;
        ikfad_elems<XT, 1>(x + o, g + o, p + o, xi + o, k);
    }
}

template <typename XT>
__device__ void elementwise_tile(const TensorDesc &td, const void *g, const Tile &tile,
                                 const Coeffs &k)
{
    XT *x = static_cast<XT *>(td.x);
    const XT *gg = static_cast<const XT *>(g);
    if (tile.vec == 8)
        elementwise_range<XT, 8>(x, gg, td.p, td.xi, tile.start, tile.count, k);
    else if (tile.vec == 4)
        elementwise_range<XT, 4>(x, gg, td.p, td.xi, tile.start, tile.count, k);
    else
        elementwise_range<XT, 1>(x, gg, td.p, td.xi, tile.start, tile.count, k);
}

// ------------------------------------------------------------- kernels

__global__ __launch_bounds__(kThreads) void rikfad_stream_kernel(
    const TensorDesc *__restrict__ tensors, const void *const *__restrict__ grads,
    const Tile *__restrict__ tiles, float *__restrict__ ws, Coeffs k, int pending)
{
    __shared__ float lds[kWaves * kWave * 8];
    const Tile tile = tiles[blockIdx.x];
    const TensorDesc td = tensors[tile.tensor];
    const void *g = grads[tile.tensor];
    if (tile.kind == KIND_VECTOR) {
        if (tile.dtype == DT_F32) elementwise_tile<float>(td, g, tile, k);
        else elementwise_tile<uint16_t>(td, g, tile, k);
        return;
    }
    if (tile.dtype == DT_F32) {
        const float *gf = static_cast<const float *>(g);
        if (tile.vec == 4) stream_matrix<float, 4>(td, gf, tile, ws, k, pending, lds);
        else stream_matrix<float, 1>(td, gf, tile, ws, k, pending, lds);
    } else {
        const uint16_t *gb = static_cast<const uint16_t *>(g);
        if (tile.vec == 8) stream_matrix<uint16_t, 8>(td, gb, tile, ws, k, pending, lds);
        else if (tile.vec == 4) stream_matrix<uint16_t, 4>(td, gb, tile, ws, k, pending, lds);
        else stream_matrix<uint16_t, 1>(td, gb, tile, ws, k, pending, lds);
    }
}

// Finalisation (C.2 / C.3 stage 2).  Row items: thread t owns row start+t,
// sums its column-block partials in block order, updates R, and the
// workgroup writes the fixed-order sum of its 256 new R values.  Column
// items: 64 columns x 4 groups of row stripes, folded in group order.
// init_only recomputes the partial sums of R from R as it stands.
__global__ __launch_bounds__(kThreads) void rikfad_finalize_kernel(
    const TensorDesc *__restrict__ tensors, const FinItem *__restrict__ items,
    float *__restrict__ ws, Coeffs k, int *__restrict__ flag, int init_only)
{
    __shared__ float lds[kThreads];
    const FinItem it = items[blockIdx.x];
    const TensorDesc td = tensors[it.tensor];
    if (it.kind == FIN_ROWS) {
        const int t = threadIdx.x;
        float rv = 0.f;
        if (t < it.count) {
            const int64_t i = static_cast<int64_t>(it.start) + t;
            rv = gmem(td.r)[i];
            if (!init_only) {
                const float *rp = ws + td.rowpart + i;
                float s = 0.f;
                for (int cb = 0; cb < td.ncb; ++cb) s += gmem(rp)[static_cast<int64_t>(cb) * td.m];
                rv = k.a * rv + k.kappa * s;
                gmem(td.r)[i] = rv;
            }
            if (!isfinite(rv)) *gmem(flag) = 1;
        }
        float v = rv;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) v += __shfl_xor(v, o);
        if ((threadIdx.x & (kWave - 1)) == 0) lds[threadIdx.x >> 6] = v;
        __syncthreads();
        if (threadIdx.x == 0) {
            const float s = ((lds[0] + lds[1]) + lds[2]) + lds[3];
            gmem(ws)[td.chunk + it.chunk] = s;
            if (!isfinite(s)) *gmem(flag) = 1;
        }
    } else {
        const int j = threadIdx.x & (kWave - 1);
        const int grp = threadIdx.x >> 6;
        const int per = (td.nrs + kWaves - 1) / kWaves;
        const int s0 = grp * per;
        const int s1 = min(td.nrs, s0 + per);
        float s = 0.f;
        if (j < it.count) {
            const float *cp = ws + td.colpart + it.start + j;
            for (int st = s0; st < s1; ++st) s += gmem(cp)[static_cast<int64_t>(st) * td.n];
        }
        lds[threadIdx.x] = s;
        __syncthreads();
        if (grp == 0 && j < it.count) {
            const float cs = ((lds[j] + lds[kWave + j]) + lds[2 * kWave + j]) + lds[3 * kWave + j];
            const int64_t jj = static_cast<int64_t>(it.start) + j;
            const float cvn = k.a * gmem(td.c)[jj] + k.kappa * cs;
            gmem(td.c)[jj] = cvn;
            if (!isfinite(cvn)) *gmem(flag) = 1;
        }
    }
}

// Second half-kick + D on stored P^(1): p <- d (p .* exp(-(h/2) xi~)) with
// the current factors (App. A Table rows C.4 and D).
template <int V>
__device__ void apply_matrix(const TensorDesc &td, const Tile &tile, const float *__restrict__ ws,
                             const Coeffs &k)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int llog = tile.lanes_log2;
    const int L = 1 << llog;
    const int G = kWave >> llog;
    const int seg = lane >> llog;
    const int sl = lane & (L - 1);
    const int64_t n = td.n;
    const int ccol = sl * V;
    const bool colok = ccol < tile.ncols;
    const int64_t col = tile.col0 + ccol;
    float cv[V];
#pragma unroll
    for (int i = 0; i < V; ++i) cv[i] = colok ? gmem(td.c)[col + i] : 0.f;
    const float denom = sum_r(ws + td.chunk, td.nchunk) + k.eps;
    const int64_t r0 = tile.start + static_cast<int64_t>(wave) * kRowsPerWave;
    const int nr = max(0, min(kRowsPerWave, static_cast<int>(tile.start + tile.count - r0)));
    const float myrate = lane < nr ? row_rate(k.kh, gmem(td.r)[r0 + lane], denom) : 0.f;
    float *__restrict__ p = td.p;
    const int nld = (nr + G - 1) >> (6 - llog);
    for (int ld = 0; ld < nld; ++ld) {
        const int rl = ld * G + seg;
        const float rate = __shfl(myrate, rl & (kWave - 1));
        if (colok && rl < nr) {
            const int64_t off = (r0 + rl) * n + col;
            float qv[V];
            Io<float, V>::load(p + off, qv);
#pragma unroll
            for (int i = 0; i < V; ++i) qv[i] = k.d * (qv[i] * exp2f(rate * cv[i]));
            Io<float, V>::store(p + off, qv);
        }
    }
}

__global__ __launch_bounds__(kThreads) void rikfad_apply_kernel(
    const TensorDesc *__restrict__ tensors, const Tile *__restrict__ tiles,
    const float *__restrict__ ws, Coeffs k)
{
    const Tile tile = tiles[blockIdx.x];
    const TensorDesc td = tensors[tile.tensor];
    if (tile.kind != KIND_MATRIX) return;
    if (tile.vec == 8) apply_matrix<8>(td, tile, ws, k);
    else if (tile.vec == 4) apply_matrix<4>(td, tile, ws, k);
    else apply_matrix<1>(td, tile, ws, k);
}

// Full-tensor iKFAD: every tile is an element range with its own friction.
__global__ __launch_bounds__(kThreads) void ikfad_kernel(
    const TensorDesc *__restrict__ tensors, const void *const *__restrict__ grads,
    const Tile *__restrict__ tiles, Coeffs k)
{
    const Tile tile = tiles[blockIdx.x];
    const TensorDesc td = tensors[tile.tensor];
    const void *g = grads[tile.tensor];
    if (tile.dtype == DT_F32) elementwise_tile<float>(td, g, tile, k);
    else elementwise_tile<uint16_t>(td, g, tile, k);
}

// ------------------------------------------------------------- probes

__global__ __launch_bounds__(kThreads) void probe_stream_kernel(
    const float4 *__restrict__ a, const float4 *__restrict__ b, const float4 *__restrict__ c,
    float4 *__restrict__ d, float4 *__restrict__ e, int64_t n4)
{
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n4;
         i += static_cast<int64_t>(gridDim.x) * kThreads) {
        const float4 va = a[i], vb = b[i], vc = c[i];
        d[i] = make_float4(va.x + vb.x, va.y + vb.y, va.z + vb.z, va.w + vb.w);
        e[i] = make_float4(va.x * vc.x, va.y * vc.y, va.z * vc.z, va.w * vc.w);
    }
}

__global__ __launch_bounds__(kThreads) void probe_copy_kernel(
    const uint4 *__restrict__ s, uint4 *__restrict__ d, int64_t n16)
{
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n16;
         i += static_cast<int64_t>(gridDim.x) * kThreads)
        d[i] = s[i];
}

// ------------------------------------------------------------- launchers

hipError_t launch_stream(const TensorDesc *tensors, const void *const *grads, const Tile *tiles,
                         int64_t ntiles, float *ws, const Coeffs &k, int pending,
                         hipStream_t stream)
{
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(rikfad_stream_kernel, dim3(static_cast<uint32_t>(ntiles)), dim3(kThreads),
                       0, stream, tensors, grads, tiles, ws, k, pending);
    return hipGetLastError();
}

hipError_t launch_finalize(const TensorDesc *tensors, const FinItem *items, int64_t nitems,
                           float *ws, const Coeffs &k, int *flag, int init_only,
                           hipStream_t stream)
{
    if (nitems <= 0) return hipSuccess;
    hipLaunchKernelGGL(rikfad_finalize_kernel, dim3(static_cast<uint32_t>(nitems)),
                       dim3(kThreads), 0, stream, tensors, items, ws, k, flag, init_only);
    return hipGetLastError();
}

hipError_t launch_apply(const TensorDesc *tensors, const Tile *tiles, int64_t ntiles,
                        const float *ws, const Coeffs &k, hipStream_t stream)
{
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(rikfad_apply_kernel, dim3(static_cast<uint32_t>(ntiles)), dim3(kThreads),
                       0, stream, tensors, tiles, ws, k);
    return hipGetLastError();
}

hipError_t launch_ikfad(const TensorDesc *tensors, const void *const *grads, const Tile *tiles,
                        int64_t ntiles, const Coeffs &k, hipStream_t stream)
{
    if (ntiles <= 0) return hipSuccess;
    hipLaunchKernelGGL(ikfad_kernel, dim3(static_cast<uint32_t>(ntiles)), dim3(kThreads), 0,
                       stream, tensors, grads, tiles, k);
    return hipGetLastError();
}

static uint32_t probe_grid(int64_t units)
{
    const int64_t want = (units + kThreads - 1) / kThreads;
    const int64_t cap = 256 * 32;     // 32 workgroups per CU on 256 CUs
    return static_cast<uint32_t>(want < 1 ? 1 : (want < cap ? want : cap));
}

hipError_t launch_probe_stream(const float *a, const float *b, const float *c, float *d,
                               float *e, int64_t nfloat, hipStream_t stream)
{
    const int64_t n4 = nfloat / 4;
    if (n4 <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_stream_kernel, dim3(probe_grid(n4)), dim3(kThreads), 0, stream,
                       reinterpret_cast<const float4 *>(a), reinterpret_cast<const float4 *>(b),
                       reinterpret_cast<const float4 *>(c), reinterpret_cast<float4 *>(d),
                       reinterpret_cast<float4 *>(e), n4);
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void *s, void *d, int64_t nbytes, hipStream_t stream)
{
    const int64_t n16 = nbytes / 16;
    if (n16 <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_copy_kernel, dim3(probe_grid(n16)), dim3(kThreads), 0, stream,
                       static_cast<const uint4 *>(s), static_cast<uint4 *>(d), n16);
    return hipGetLastError();
}

}  // namespace rk
