// device.hpp -- device-side helpers shared by the gfx950 kernels: global
// address-space casts, non-temporal streaming accesses, bf16 conversion,
// vectorised row accesses and the fixed-order sum of the partial sums of R.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Streams are read and written exactly once per step: the accesses carry
// the non-temporal hint so they do not displace the small, reused data
// (factors, partial sums, tables) from the caches.
template <typename T>
__device__ __forceinline__ T ldg(const T *q)
{
    return __builtin_nontemporal_load(gmem(q));
}

template <typename T>
__device__ __forceinline__ void stg(T *q, T v)
{
    __builtin_nontemporal_store(v, gmem(q));
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
        const f32x4 v = ldg(reinterpret_cast<const f32x4 *>(q));
        o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
    }
    static __device__ __forceinline__ void store(float *q, const float (&o)[4])
    {
        stg(reinterpret_cast<f32x4 *>(q), f32x4{o[0], o[1], o[2], o[3]});
    }
};

template <> struct Io<float, 8> {
    static __device__ __forceinline__ void load(const float *q, float (&o)[8])
    {
        const f32x4 a = ldg(reinterpret_cast<const f32x4 *>(q));
        const f32x4 b = ldg(reinterpret_cast<const f32x4 *>(q) + 1);
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
        o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
    static __device__ __forceinline__ void store(float *q, const float (&o)[8])
    {
        stg(reinterpret_cast<f32x4 *>(q), f32x4{o[0], o[1], o[2], o[3]});
        stg(reinterpret_cast<f32x4 *>(q) + 1, f32x4{o[4], o[5], o[6], o[7]});
    }
};

template <> struct Io<float, 1> {
    static __device__ __forceinline__ void load(const float *q, float (&o)[1]) { o[0] = ldg(q); }
    static __device__ __forceinline__ void store(float *q, const float (&o)[1]) { stg(q, o[0]); }
};

template <> struct Io<uint16_t, 8> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[8])
    {
        const u32x4 v = ldg(reinterpret_cast<const u32x4 *>(q));
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
        stg(reinterpret_cast<u32x4 *>(q), u32x4{w[0], w[1], w[2], w[3]});
    }
};

template <> struct Io<uint16_t, 4> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[4])
    {
        const u32x2 v = ldg(reinterpret_cast<const u32x2 *>(q));
        o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
        o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
    }
    static __device__ __forceinline__ void store(uint16_t *q, const float (&o)[4])
    {
        const uint32_t a = static_cast<uint32_t>(f32_to_bf16(o[0])) |
                           (static_cast<uint32_t>(f32_to_bf16(o[1])) << 16);
        const uint32_t b = static_cast<uint32_t>(f32_to_bf16(o[2])) |
                           (static_cast<uint32_t>(f32_to_bf16(o[3])) << 16);
        stg(reinterpret_cast<u32x2 *>(q), u32x2{a, b});
    }
};

template <> struct Io<uint16_t, 1> {
    static __device__ __forceinline__ void load(const uint16_t *q, float (&o)[1]) { o[0] = bf16_to_f32(ldg(q)); }
    static __device__ __forceinline__ void store(uint16_t *q, const float (&o)[1]) { stg(q, f32_to_bf16(o[0])); }
};

// Raw<T, V>: the V elements of one lane access as loaded (packed bf16 stays
// packed in registers until it is used).
template <typename T, int V> struct Raw;

template <> struct Raw<float, 4> {
    typedef f32x4 type;
    static __device__ __forceinline__ type load(const float *q)
    {
        return ldg(reinterpret_cast<const f32x4 *>(q));
    }
    static __device__ __forceinline__ void unpack(const type &v, float (&o)[4])
    {
        o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
    }
};

template <> struct Raw<float, 1> {
    typedef float type;
    static __device__ __forceinline__ type load(const float *q) { return ldg(q); }
    static __device__ __forceinline__ void unpack(const type &v, float (&o)[1]) { o[0] = v; }
};

template <> struct Raw<uint16_t, 4> {
    typedef u32x2 type;
    static __device__ __forceinline__ type load(const uint16_t *q)
    {
        return ldg(reinterpret_cast<const u32x2 *>(q));
    }
    static __device__ __forceinline__ void unpack(const type &v, float (&o)[4])
    {
        o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
        o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
    }
};

template <> struct Raw<uint16_t, 1> {
    typedef uint16_t type;
    static __device__ __forceinline__ type load(const uint16_t *q) { return ldg(q); }
    static __device__ __forceinline__ void unpack(const type &v, float (&o)[1])
    {
        o[0] = bf16_to_f32(v);
    }
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

// v - h g and d v with the split coefficients (h = h + h_lo, d = 1 + dm1):
// each product is added by a fused multiply-add, so the coefficients'
// fp32 rounding does not accumulate over steps.
__device__ __forceinline__ float kick(float v, float g, const Coeffs &k)
{
    return __builtin_fmaf(-k.h_lo, g, __builtin_fmaf(-k.h, g, v));
}
__device__ __forceinline__ float damp(float v, const Coeffs &k)
{
    return __builtin_fmaf(v, k.dm1, v);
}

// Stage 1 of the row and column sums of a matrix tile, after each wave has
// walked its rows.  acc[V]: this lane's column sums; myrow: in lane t, the
// sum of the wave's row r0 + t (t < nr).  Lanes l and l ^ o (o >= L) own the
// same columns and are folded first, then the waves through LDS in wave
// order; the tile writes its column partials (stripe `stripe` of colpart) and
// each wave its row partials (row `cb` of rowpart).  Every thread of the
// workgroup must call this (it synchronises the workgroup).
template <int V>
__device__ __forceinline__ void store_partials(const TensorDesc &td, const Tile &tile,
                                               float *__restrict__ ws, float (&acc)[V],
                                               float myrow, int nr, int64_t r0, float *lds)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int L = 1 << tile.lanes_log2;
    const int ccol = (lane & (L - 1)) * V;
    for (int o = L; o < kWave; o <<= 1) {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += __shfl_xor(acc[i], o);
    }
    if (lane < L && ccol < tile.ncols) {
#pragma unroll
        for (int i = 0; i < V; ++i) lds[wave * kWave * V + ccol + i] = acc[i];
    }
    __syncthreads();
    float *colpart = ws + td.colpart;
    for (int j = threadIdx.x; j < tile.ncols; j += kStreamWaves * kWave) {
        float sum = lds[j];
#pragma unroll
        for (int w = 1; w < kStreamWaves; ++w) sum += lds[w * kWave * V + j];
        gmem(colpart)[colpart_index(tile.col0 + j, tile.stripe, td.nrs)] = sum;
    }
    if (lane < nr) gmem(ws)[td.rowpart + static_cast<int64_t>(tile.cb) * pad4(td.m) + r0 + lane] = myrow;
}

}  // namespace rk
