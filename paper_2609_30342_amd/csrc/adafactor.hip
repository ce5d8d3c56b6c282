// adafactor.hip -- gfx950 kernels of the Adafactor-m step.
//
// Adafactor-m is the paper's baseline (Section 2, Methodology, left-hand
// system; discrete schedule of Section 3 and App. "Hyperparameters"): a full
// first moment M and the factored second moment of the gradient, R (row
// sums) and C (column sums) of an exponential average of G^2 + eps1,
// acting in the position equation.  Step t with b = 1 - t^decay_rate:
//
//   pass 1  row / column partial sums of G^2 + eps1            reads g
//   fin     R <- b R + (1-b) rowsum, C <- b C + (1-b) colsum,
//           partial sums of R (the R-iKFAD finalisation kernel)
//   pass 2  tile sums of U^2, U = G / sqrt(R C^T / 1^T R)      reads g
//   scale   s = h [max(eps2, RMS(X))] / max(1, RMS(U) / d)     per tensor
//   pass 3  M <- beta1 M + (1 - beta1) s U,  X <- X - M         reads g, x, M; writes x, M
//
// The clipping divisor needs RMS(U) over the whole tensor with the new
// factors before any element can move, so the gradient is streamed three
// times (R-iKFAD's factors damp the momentum instead, and its step needs
// one pass).  Vectors keep an unfactored second moment v and finish their
// U^2 sums in pass 1.  The passes use R-iKFAD's tile tables and partial-sum
// layout; every sum has a fixed order, so results are reproducible bit for
// bit.  HBM-bound like the R-iKFAD step: no MFMA.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "adafactor.hpp"
#include "device.hpp"
#include "launch.hpp"
#include "layout.hpp"

namespace rk {
namespace {

// Row loads per wave issued together in the two read passes (statistics,
// RMS); half as many when the statistics pass also reads x.  With the read
// passes' 16-row waves and 1 KB row loads (fp32, or bf16 at 8 elements per
// lane), 4 measured as fast as 8 for fp32 and faster for bf16 (statistics
// pass 5.2 against 4.2 TB/s), and 16 slower for both.
#ifndef RK_ADA_READ_BATCH
#define RK_ADA_READ_BATCH 4
#endif
constexpr int kReadBatch = RK_ADA_READ_BATCH;
static_assert(kReadBatch >= 1 && kReadBatch <= 32, "read batch");

// Lane geometry of a matrix tile (see the R-iKFAD streaming pass): wave w
// walks rows r0 .. r0 + nr - 1; each row of the block is covered by L
// lanes owning V consecutive columns, G = 64 / L rows per load.
struct Lanes {
    int lane, llog, L, G, seg, nr, nld;
    bool colok;
    int64_t col, lcol, r0;
    int64_t r_any;     // a row of the tile this wave may read: r0, or the tile's first row
};

template <int V>
__device__ __forceinline__ Lanes lanes_of(const Tile &tile)
{
    Lanes t;
    t.lane = threadIdx.x & (kWave - 1);
    t.llog = tile.lanes_log2;
    t.L = 1 << t.llog;
    t.G = kWave >> t.llog;
    t.seg = t.lane >> t.llog;
    const int ccol = (t.lane & (t.L - 1)) * V;
    t.colok = ccol < tile.ncols;
    t.col = tile.col0 + ccol;
    t.lcol = t.colok ? t.col : tile.col0;   // lanes past the block read its first column
    t.r0 = tile.start + static_cast<int64_t>(threadIdx.x >> 6) * tile.rpw;
    t.nr = max(0, min(tile.rpw, static_cast<int>(tile.start + tile.count - t.r0)));
    t.nld = (t.nr + t.G - 1) >> (6 - t.llog);
    t.r_any = t.nr > 0 ? t.r0 : tile.start;
    return t;
}

// Element offset of row rl of a load; rows outside the wave read a row of
// the tile (its own first row, or the tile's if the wave has none), so the
// load is always in bounds, and are masked by the caller.
__device__ __forceinline__ int64_t row_off(const Lanes &t, int rl, int64_t n)
{
    return (t.colok && rl < t.nr ? t.r0 + rl : t.r_any) * n + t.lcol;
}

// v where keep, else +0, by a bitwise mask: a select on a loaded value can
// be compiled into a branch around the load, and a load under a branch
// makes the wave wait for every load it has in flight.
__device__ __forceinline__ float masked(float v, bool keep)
{
    return __uint_as_float(__float_as_uint(v) & (keep ? 0xffffffffu : 0u));
}

// Row sums of the statistics pass, kRowChunk row loads at a time.  a[u] is
// this lane's share of the row of load c0 + u (row (c0 + u) * G + seg); the
// L lanes of a row are combined pairwise by lane bit 0, 1, 2, ... -- the
// xor-butterfly tree, so every sum has the same bits as a butterfly per row
// -- but each exchange hands over half of the loads a lane holds and keeps
// the other half (lanes with the bit set keep the upper half).  After
// log2(kRowChunk) exchanges a lane holds one load's sum, which the last
// exchanges complete; about kRowChunk + log2(L) shuffles per chunk instead
// of log2(L) + 1 per row, none of them between two row loads.  Lane t then
// fetches the sum of row t from a lane that holds it.  Chunks of 8 loads
// (two per 16-row wave) measured faster than 16, which need more registers.
#ifndef RK_ADA_ROW_CHUNK_LOG2
#define RK_ADA_ROW_CHUNK_LOG2 3
#endif
constexpr int kRowChunkLog2 = RK_ADA_ROW_CHUNK_LOG2;
constexpr int kRowChunk = 1 << kRowChunkLog2;

__device__ __forceinline__ void park_rows(float (&a)[kRowChunk], int c0, const Lanes &t,
                                          float &myrow)
{
#pragma unroll
    for (int s = 0; s < kRowChunkLog2; ++s) {
        const int o = 1 << s;
        if (o < t.L) {
            const bool up = (t.lane & o) != 0;
            constexpr int h0 = kRowChunk >> 1;
#pragma unroll
            for (int i = 0; i < (h0 >> s); ++i) {
                const int h = h0 >> s;
                // The empty asm keeps the lane-dependent choice a choice of
                // registers (otherwise it is folded into a choice of address,
                // which sends a[] to scratch memory).
                float lo = a[i], hi = a[i + h];
                asm("" : "+v"(lo), "+v"(hi));
                const float give = up ? lo : hi;
                const float keep = up ? hi : lo;
                a[i] = keep + __shfl_xor(give, o);
            }
        }
    }
    for (int o = kRowChunk; o < t.L; o <<= 1) a[0] += __shfl_xor(a[0], o);
    // The halving exchanges done: j = min(log2 L, log2 kRowChunk); a lane
    // keeps a[0 .. m), m = kRowChunk >> j, the loads whose top j bits
    // (most significant first) equal its lane bits 0 .. j-1.
    const int j = t.llog < kRowChunkLog2 ? t.llog : kRowChunkLog2;
    const int m = kRowChunk >> j;
    const int rl = t.lane;                       // the row this lane stores
    const int ld = rl >> (6 - t.llog);
    const int u = ld - c0;
    const int seg = rl & (t.G - 1);
    int sl = 0;
    for (int b = 0; b < j; ++b) sl |= ((u >> (kRowChunkLog2 - 1 - b)) & 1) << b;
    const int src = (seg << t.llog) | sl;
    const int i = u & (m - 1);
    float v = __shfl(a[0], src);
#pragma unroll
    for (int q = 1; q < kRowChunk; ++q) {
        if (q < m) {
            const float w = __shfl(a[q], src);
            if (i == q) v = w;
        }
    }
    if (u >= 0 && u < kRowChunk) myrow = v;
}

// Workgroup sums of a and b in a fixed order (xor butterfly inside each
// wave, then the waves in order); valid in thread 0.
template <int NW>
__device__ __forceinline__ void block_sum2(float &a, float &b, float *red)
{
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        a += __shfl_xor(a, o);
        b += __shfl_xor(b, o);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        red[2 * wave] = a;
        red[2 * wave + 1] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = red[0];
        b = red[1];
#pragma unroll
        for (int w = 1; w < NW; ++w) {
            a += red[2 * w];
            b += red[2 * w + 1];
        }
    }
}

// 1 / sqrt(R_i / 1^T R) and 1 / sqrt(C_j); 0 where the factor is 0, so that
// U = G * row_factor * col_factor is 0 where the estimate R C^T / 1^T R is.
__device__ __forceinline__ float row_factor(float r, float inv_s)
{
    return r > 0.f ? rsqrtf(r * inv_s) : 0.f;
}
__device__ __forceinline__ float col_factor(float c) { return c > 0.f ? rsqrtf(c) : 0.f; }

// Per-row factors of a matrix tile: lane t holds row r0 + t's, columns in fc.
template <int V>
__device__ __forceinline__ float tile_factors(const TensorDesc &td, const Lanes &t,
                                              const float *__restrict__ ws, float (&fc)[V])
{
#pragma unroll
    for (int i = 0; i < V; ++i) fc[i] = t.colok ? col_factor(gmem(td.c)[t.col + i]) : 0.f;
    const float s = sum_r(ws + td.chunk, td.nchunk);
    const float inv_s = s > 0.f ? 1.f / s : 0.f;
    return t.lane < t.nr ? row_factor(gmem(td.r)[t.r0 + t.lane], inv_s) : 0.f;
}

// The same factors for the read passes, with every load issued at once:
// columns from the clamped column lcol, the partial sums of R in batches of
// kChunkLoads per lane (summed in the order of sum_r: lane, lane + 64, ...,
// then the butterfly), and R from a clamped row.  Identical values.
constexpr int kChunkLoads = 8;

template <int V>
__device__ __forceinline__ float read_factors(const TensorDesc &td, const Lanes &t,
                                              const float *__restrict__ ws, float (&fc)[V])
{
    float cv[V];
#pragma unroll
    for (int i = 0; i < V; ++i) cv[i] = gmem(td.c)[t.lcol + i];
    const int nch = td.nchunk;
    const RK_GLOBAL float *part = gmem(ws) + td.chunk;
    const bool rowok = t.lane < t.nr;
    const float rv = gmem(td.r)[rowok ? t.r0 + t.lane : t.r_any];
    float s = 0.f;
    for (int i0 = 0; i0 < nch; i0 += kWave * kChunkLoads) {
        float v[kChunkLoads];
#pragma unroll
        for (int u = 0; u < kChunkLoads; ++u) {
            const int idx = i0 + u * kWave + t.lane;
            v[u] = part[idx < nch ? idx : nch - 1];
        }
#pragma unroll
        for (int u = 0; u < kChunkLoads; ++u) s += masked(v[u], i0 + u * kWave + t.lane < nch);
    }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) s += __shfl_xor(s, o);
    const float inv_s = s > 0.f ? 1.f / s : 0.f;
#pragma unroll
    for (int i = 0; i < V; ++i) fc[i] = t.colok ? col_factor(cv[i]) : 0.f;
    return rowok ? row_factor(rv, inv_s) : 0.f;
}

// Runs op.run<W>(offset) over the elements [start, start + count) of a
// vector tile, W = the tile's access width, then the scalar tail.
template <int W, typename Op>
__device__ __forceinline__ void flat_walk(int64_t start, int count, Op &op)
{
    const int full = count - count % W;
    for (int e = threadIdx.x * W; e < full; e += kStreamThreads * W) op.template run<W>(start + e);
    for (int e = full + threadIdx.x; e < count; e += kStreamThreads) op.template run<1>(start + e);
}

template <typename Op>
__device__ __forceinline__ void flat_tile(const Tile &tile, Op &op)
{
    if (tile.vec == 8)
        flat_walk<8>(tile.start, tile.count, op);
    else if (tile.vec == 4)
        flat_walk<4>(tile.start, tile.count, op);
    else
        flat_walk<1>(tile.start, tile.count, op);
}

// ---------------------------------------------------------------- pass 1

template <typename XT, int V, bool X2>
__device__ void stats_matrix(const TensorDesc &td, const XT *__restrict__ g, const Tile &tile,
                             float *__restrict__ ws, const AdaCoeffs &k, float *lds, float &x2)
{
    // Batches of B row loads, all issued before the first is summed.  The
    // loads are unconditional (rows past the wave's last are clamped into
    // the tensor and masked), so the compiler waits for each row exactly.
    // The row sums of a chunk of kRowChunk loads are completed together
    // after its last batch.
    constexpr int B = X2 ? (kReadBatch + 1) / 2 : kReadBatch;
    static_assert(kRowChunk % B == 0, "whole batches per row chunk");
    const Lanes t = lanes_of<V>(tile);
    const XT *__restrict__ x = static_cast<const XT *>(td.x);
    const int64_t n = td.n;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
    float myrow = 0.f;
    for (int c0 = 0; c0 < t.nld; c0 += kRowChunk) {
        float a[kRowChunk];
#pragma unroll
        for (int u = 0; u < kRowChunk; ++u) a[u] = 0.f;
#pragma unroll
        for (int b0 = 0; b0 < kRowChunk; b0 += B) {
            if (c0 + b0 < t.nld) {
                typename Raw<XT, V>::type gr[B], xr[B];
#pragma unroll
                for (int u = 0; u < B; ++u) {
                    const int64_t off = row_off(t, (c0 + b0 + u) * t.G + t.seg, n);
                    gr[u] = Raw<XT, V>::load(g + off);
                    if (X2) xr[u] = Raw<XT, V>::load(x + off);
                }
#pragma unroll
                for (int u = 0; u < B; ++u) {
                    const bool ok = t.colok && (c0 + b0 + u) * t.G + t.seg < t.nr;
                    float gv[V];
                    Raw<XT, V>::unpack(gr[u], gv);
                    float rs = 0.f;
#pragma unroll
                    for (int i = 0; i < V; ++i) {
                        const float q = ok ? gv[i] * gv[i] + k.eps1 : 0.f;
                        acc[i] += q;
                        rs += q;
                    }
                    a[b0 + u] = rs;
                    if (X2) {
                        float xv[V];
                        Raw<XT, V>::unpack(xr[u], xv);
#pragma unroll
                        for (int i = 0; i < V; ++i) x2 += ok ? xv[i] * xv[i] : 0.f;
                    }
                }
            }
        }
        park_rows(a, c0, t, myrow);
    }
    store_partials<V>(td, tile, ws, acc, myrow, t.nr, t.r0, lds);
}

// Unfactored second moment: v <- b v + (1-b)(G^2 + eps1); sums of U^2 with
// U = G / sqrt(v), and of X^2 when X2.
template <typename XT, bool X2>
struct StatsVec {
    const XT *g;
    const XT *x;
    float *v;
    AdaCoeffs k;
    float u2, x2;

    template <int W>
    __device__ __forceinline__ void run(int64_t o)
    {
        float gv[W], vv[W];
        Io<XT, W>::load(g + o, gv);
        Io<float, W>::load(v + o, vv);
#pragma unroll
        for (int i = 0; i < W; ++i) {
            vv[i] = k.b * vv[i] + k.omb * (gv[i] * gv[i] + k.eps1);
            const float u = vv[i] > 0.f ? gv[i] * rsqrtf(vv[i]) : 0.f;
            u2 += u * u;
        }
        Io<float, W>::store(v + o, vv);
        if (X2) {
            float xv[W];
            Io<XT, W>::load(x + o, xv);
#pragma unroll
            for (int i = 0; i < W; ++i) x2 += xv[i] * xv[i];
        }
    }
};

template <typename XT, int V, bool X2>
__global__ __launch_bounds__(kStreamThreads) void adafm_stats_kernel(
    const TensorDesc *__restrict__ tensors, const void *const *__restrict__ grads,
    const Tile *__restrict__ tiles, int64_t tile0, float *__restrict__ ws,
    float *__restrict__ tilepart, AdaCoeffs k)
{
    __shared__ float lds[kStreamWaves * kWave * V];
    __shared__ float red[2 * kStreamWaves];
    const int64_t ti = tile0 + blockIdx.x;
    const Tile tile = tiles[ti];
    const TensorDesc td = tensors[tile.tensor];
    const XT *g = static_cast<const XT *>(grads[tile.tensor]);
    float u2 = 0.f, x2 = 0.f;
    if (tile.kind == KIND_VECTOR) {
        StatsVec<XT, X2> op{g, static_cast<const XT *>(td.x), td.xi, k, 0.f, 0.f};
        flat_tile(tile, op);
        u2 = op.u2;
        x2 = op.x2;
    } else if (V > 1 && tile.vec == 1) {
        stats_matrix<XT, 1, X2>(td, g, tile, ws, k, lds, x2);
    } else {
        stats_matrix<XT, V, X2>(td, g, tile, ws, k, lds, x2);
    }
    block_sum2<kStreamWaves>(u2, x2, red);
    if (threadIdx.x == 0) {
        gmem(tilepart)[2 * ti] = u2;
        gmem(tilepart)[2 * ti + 1] = x2;
    }
}

// ---------------------------------------------------------------- pass 2

// Sum of U^2 over one matrix tile (this lane's share), in batches of row
// loads as in the statistics pass.  The first batch goes out before the
// factor loads, so their round trips overlap.
template <typename XT, int V>
__device__ float rms_matrix(const TensorDesc &td, const XT *__restrict__ g, const Tile &tile,
                            const float *__restrict__ ws)
{
    constexpr int B = kReadBatch;
    const Lanes t = lanes_of<V>(tile);
    typename Raw<XT, V>::type gr[B];
    float u2 = 0.f;
    auto issue = [&](int ld0) {
#pragma unroll
        for (int u = 0; u < B; ++u)
            gr[u] = Raw<XT, V>::load(g + row_off(t, (ld0 + u) * t.G + t.seg, td.n));
    };
    issue(0);
    float fc[V];
    const float myfr = read_factors<V>(td, t, ws, fc);
    auto sum = [&](int ld0) {
        // u2 + uu * uu stays a product and a sum (never fused), in every
        // row alike, so the sum does not depend on code placement.
#pragma clang fp contract(off)
#pragma unroll
        for (int u = 0; u < B; ++u) {
            const int rl = (ld0 + u) * t.G + t.seg;
            const bool ok = t.colok && rl < t.nr;
            const float fr = __shfl(myfr, rl & (kWave - 1));
            float gv[V];
            Raw<XT, V>::unpack(gr[u], gv);
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const float uu = (gv[i] * fr) * fc[i];
                u2 += ok ? uu * uu : 0.f;
            }
        }
    };
    sum(0);
    for (int ld0 = B; ld0 < t.nld; ld0 += B) {
        issue(ld0);
        sum(ld0);
    }
    return u2;
}

template <typename XT, int V>
__global__ __launch_bounds__(kStreamThreads) void adafm_rms_kernel(
    const TensorDesc *__restrict__ tensors, const void *const *__restrict__ grads,
    const Tile *__restrict__ tiles, int64_t tile0, const float *__restrict__ ws,
    float *__restrict__ tilepart)
{
    __shared__ float red[2 * kStreamWaves];
    const int64_t ti = tile0 + blockIdx.x;
    const Tile tile = tiles[ti];
    if (tile.kind == KIND_VECTOR) return;   // vector sums are complete after pass 1
    const TensorDesc td = tensors[tile.tensor];
    const XT *__restrict__ g = static_cast<const XT *>(grads[tile.tensor]);
    float u2 = V > 1 && tile.vec == 1 ? rms_matrix<XT, 1>(td, g, tile, ws)
                                      : rms_matrix<XT, V>(td, g, tile, ws);
    float zero = 0.f;
    block_sum2<kStreamWaves>(u2, zero, red);
    if (threadIdx.x == 0) gmem(tilepart)[2 * ti] = u2;
}

// ----------------------------------------------------------------- scale

__global__ __launch_bounds__(kThreads) void adafm_scale_kernel(
    const TensorRange *__restrict__ ranges, const float *__restrict__ tilepart,
    float *__restrict__ scales, AdaCoeffs k)
{
    __shared__ float red[2 * (kThreads / kWave)];
    const TensorRange rg = ranges[blockIdx.x];
    float u2 = 0.f, x2 = 0.f;
    for (int64_t q = threadIdx.x; q < rg.ntile; q += kThreads) {
        u2 += gmem(tilepart)[2 * (rg.tile0 + q)];
        x2 += gmem(tilepart)[2 * (rg.tile0 + q) + 1];
    }
    block_sum2<kThreads / kWave>(u2, x2, red);
    if (threadIdx.x == 0) {
        const double el = static_cast<double>(rg.elems);
        const double rms_u = sqrt(static_cast<double>(u2) / el);
        const double rms_x = sqrt(static_cast<double>(x2) / el);
        double step = k.h;
        if (k.scale) step *= rms_x > k.eps2 ? rms_x : static_cast<double>(k.eps2);
        const double div = (k.clip > 0.f && rms_u / k.clip > 1.0) ? rms_u / k.clip : 1.0;
        gmem(scales)[blockIdx.x] = static_cast<float>(step / div);
    }
}

// ---------------------------------------------------------------- pass 3

// Row loads in flight per wave in pass 3 (g, x, M per slot), as in the
// R-iKFAD streaming pass: the factors are read first, then the load of
// row-load ld + B goes out as soon as row-load ld has been consumed.
template <typename XT> struct UpdateRing { static constexpr int value = kRingF32; };
template <> struct UpdateRing<uint16_t> { static constexpr int value = kRingBF16; };

template <typename XT, int V>
__device__ void update_matrix(const TensorDesc &td, const XT *__restrict__ g, const Tile &tile,
                              const float *__restrict__ ws, float s, const AdaCoeffs &k)
{
    constexpr int B = UpdateRing<XT>::value;
    const Lanes t = lanes_of<V>(tile);
    XT *__restrict__ x = static_cast<XT *>(td.x);
    float *__restrict__ mom = td.p;
    const int64_t n = td.n;
    typename Raw<XT, V>::type gr[B], xr[B];
    float mv[B][V];
    float fc[V];
    const float myfr = tile_factors<V>(td, t, ws, fc);
    if (t.nld > 0) {
#pragma unroll
        for (int u = 0; u < B; ++u) {
            const int64_t off = row_off(t, u * t.G + t.seg, n);
            gr[u] = Raw<XT, V>::load(g + off);
            xr[u] = Raw<XT, V>::load(x + off);
            Io<float, V>::load(mom + off, mv[u]);
        }
    }
    for (int ld0 = 0; ld0 < t.nld; ld0 += B) {
#pragma unroll
        for (int u = 0; u < B; ++u) {
            const int ld = ld0 + u;
            const int rl = ld * t.G + t.seg;
            const float fr = __shfl(myfr, rl & (kWave - 1));
            float gv[V], xv[V];
            Raw<XT, V>::unpack(gr[u], gv);
            Raw<XT, V>::unpack(xr[u], xv);
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const float uu = (gv[i] * fr) * fc[i];
                mv[u][i] = k.beta1 * mv[u][i] + k.omb1 * (s * uu);
                xv[i] = xv[i] - mv[u][i];
            }
            if (t.colok && rl < t.nr) {
                const int64_t off = (t.r0 + rl) * n + t.col;
                Io<XT, V>::store(x + off, xv);
                Io<float, V>::store(mom + off, mv[u]);
            }
            if (ld + B < t.nld) {
                const int64_t off = row_off(t, (ld + B) * t.G + t.seg, n);
                gr[u] = Raw<XT, V>::load(g + off);
                xr[u] = Raw<XT, V>::load(x + off);
                Io<float, V>::load(mom + off, mv[u]);
            }
        }
    }
}

template <typename XT>
struct UpdateVec {
    const XT *g;
    XT *x;
    float *mom;
    const float *v;
    float s;
    AdaCoeffs k;

    template <int W>
    __device__ __forceinline__ void run(int64_t o)
    {
        float gv[W], xv[W], mv[W], vv[W];
        Io<XT, W>::load(g + o, gv);
        Io<XT, W>::load(x + o, xv);
        Io<float, W>::load(mom + o, mv);
        Io<float, W>::load(v + o, vv);
#pragma unroll
        for (int i = 0; i < W; ++i) {
            const float uu = vv[i] > 0.f ? gv[i] * rsqrtf(vv[i]) : 0.f;
            mv[i] = k.beta1 * mv[i] + k.omb1 * (s * uu);
            xv[i] = xv[i] - mv[i];
        }
        Io<XT, W>::store(x + o, xv);
        Io<float, W>::store(mom + o, mv);
    }
};

template <typename XT, int V>
__global__ __launch_bounds__(kStreamThreads) void adafm_update_kernel(
    const TensorDesc *__restrict__ tensors, const void *const *__restrict__ grads,
    const Tile *__restrict__ tiles, int64_t tile0, const float *__restrict__ ws,
    const float *__restrict__ scales, AdaCoeffs k)
{
    const Tile tile = tiles[tile0 + blockIdx.x];
    const TensorDesc td = tensors[tile.tensor];
    const XT *g = static_cast<const XT *>(grads[tile.tensor]);
    const float s = gmem(scales)[tile.tensor];
    if (tile.kind == KIND_VECTOR) {
        UpdateVec<XT> op{g, static_cast<XT *>(td.x), td.p, td.xi, s, k};
        flat_tile(tile, op);
        return;
    }
    if (V > 1 && tile.vec == 1) update_matrix<XT, 1>(td, g, tile, ws, s, k);
    else update_matrix<XT, V>(td, g, tile, ws, s, k);
}

// Kernel instantiation for a tile group's (storage type, width); a wide
// one also serves the group's one-column tiles.  nullptr for a combination
// the planner does not produce.
template <typename F, typename Pick>
F pick(const TileGroup &gr, Pick p)
{
    if (gr.dtype == DT_F32) return gr.vec == 4 ? p.template get<float, 4>()
                                : gr.vec == 1 ? p.template get<float, 1>() : nullptr;
    return gr.vec == 4 ? p.template get<uint16_t, 4>()
         : gr.vec == 1 ? p.template get<uint16_t, 1>() : nullptr;
}

typedef void (*StatsFn)(const TensorDesc *, const void *const *, const Tile *, int64_t, float *,
                        float *, AdaCoeffs);
typedef void (*RmsFn)(const TensorDesc *, const void *const *, const Tile *, int64_t,
                      const float *, float *);
typedef void (*UpdateFn)(const TensorDesc *, const void *const *, const Tile *, int64_t,
                         const float *, const float *, AdaCoeffs);

template <bool X2> struct PickStats {
    template <typename XT, int V> StatsFn get() const { return adafm_stats_kernel<XT, V, X2>; }
};
struct PickRms {
    template <typename XT, int V> RmsFn get() const { return adafm_rms_kernel<XT, V>; }
};
struct PickUpdate {
    template <typename XT, int V> UpdateFn get() const { return adafm_update_kernel<XT, V>; }
};

}  // namespace

hipError_t launch_adafm_stats(const TensorDesc *tensors, const void *const *grads,
                              const Tile *tiles, const TileGroup *groups, int ngroups, float *ws,
                              float *tilepart, const AdaCoeffs &k, bool x2, hipStream_t stream,
                              hipEvent_t start, hipEvent_t stop)
{
    const int last = last_group(groups, ngroups);
    for (int q = 0; q < ngroups; ++q) {
        const TileGroup &gr = groups[q];
        if (gr.count <= 0) continue;
        const StatsFn fn = x2 ? pick<StatsFn>(gr, PickStats<true>())
                              : pick<StatsFn>(gr, PickStats<false>());
        if (!fn) return hipErrorInvalidValue;
        hipEvent_t a = start, b = q == last ? stop : nullptr;
        start = nullptr;
        const hipError_t e = launch(fn, dim3(static_cast<uint32_t>(gr.count)),
                                    dim3(kStreamThreads), stream, a, b, tensors, grads, tiles,
                                    gr.begin, ws, tilepart, k);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_adafm_rms(const TensorDesc *tensors, const void *const *grads,
                            const Tile *tiles, const TileGroup *groups, int ngroups,
                            const float *ws, float *tilepart, hipStream_t stream,
                            hipEvent_t start, hipEvent_t stop)
{
    const int last = last_group(groups, ngroups);
    for (int q = 0; q < ngroups; ++q) {
        const TileGroup &gr = groups[q];
        if (gr.count <= 0) continue;
        const RmsFn fn = pick<RmsFn>(gr, PickRms());
        if (!fn) return hipErrorInvalidValue;
        hipEvent_t a = start, b = q == last ? stop : nullptr;
        start = nullptr;
        const hipError_t e = launch(fn, dim3(static_cast<uint32_t>(gr.count)),
                                    dim3(kStreamThreads), stream, a, b, tensors, grads, tiles,
                                    gr.begin, ws, tilepart);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_adafm_scale(const TensorRange *ranges, int64_t ntensors, const float *tilepart,
                              float *scales, const AdaCoeffs &k, hipStream_t stream,
                              hipEvent_t start, hipEvent_t stop)
{
    if (ntensors <= 0) return hipSuccess;
    return launch(adafm_scale_kernel, dim3(static_cast<uint32_t>(ntensors)), dim3(kThreads),
                  stream, start, stop, ranges, tilepart, scales, k);
}

hipError_t launch_adafm_update(const TensorDesc *tensors, const void *const *grads,
                               const Tile *tiles, const TileGroup *groups, int ngroups,
                               const float *ws, const float *scales, const AdaCoeffs &k,
                               hipStream_t stream, hipEvent_t start, hipEvent_t stop)
{
    const int last = last_group(groups, ngroups);
    for (int q = 0; q < ngroups; ++q) {
        const TileGroup &gr = groups[q];
        if (gr.count <= 0) continue;
        const UpdateFn fn = pick<UpdateFn>(gr, PickUpdate());
        if (!fn) return hipErrorInvalidValue;
        hipEvent_t a = start, b = q == last ? stop : nullptr;
        start = nullptr;
        const hipError_t e = launch(fn, dim3(static_cast<uint32_t>(gr.count)),
                                    dim3(kStreamThreads), stream, a, b, tensors, grads, tiles,
                                    gr.begin, ws, scales, k);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace rk
