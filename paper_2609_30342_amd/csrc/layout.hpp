// layout.hpp -- tables shared by the host planner and the gfx950 kernels.
//
// The step runs over a flat table of workgroup tiles covering every tensor
// of a context (one launch for all tensors), and a table of finalisation
// items that turn per-tile partial sums into the new friction factors.
#pragma once
#include <stdint.h>

namespace rk {

// The streaming tile's shape and the ring depths can be overridden at build
// time (-DRK_...) to measure alternatives; the defaults are the fastest
// measured on MI355X.
#ifndef RK_STREAM_WAVES
#define RK_STREAM_WAVES 8
#endif
constexpr int kWave = 64;                       // CDNA wavefront
constexpr int kThreads = 256;                   // workgroup of the small kernels
constexpr int kThreadsLog2 = 8;
constexpr int kStreamWaves = RK_STREAM_WAVES;   // waves per streaming workgroup
constexpr int kStreamThreads = kWave * kStreamWaves;
#ifndef RK_RING_F32
#define RK_RING_F32 3
#endif
#ifndef RK_RING_BF16
#define RK_RING_BF16 2
#endif
#ifndef RK_BLOCK_LANES
#define RK_BLOCK_LANES 64
#endif
#ifndef RK_ROWS_PER_WAVE
#define RK_ROWS_PER_WAVE 4
#endif
constexpr int kRingF32 = RK_RING_F32;           // row loads in flight per wave (fp32)
constexpr int kRingBF16 = RK_RING_BF16;         // the same for bf16 x/g
constexpr int kMaxRowsPerWave = 64;             // lane t keeps row t's partial sum
constexpr int kBlockLanes = RK_BLOCK_LANES;     // lanes per row of a full column block
constexpr int kRowsPerWave = RK_ROWS_PER_WAVE;  // rows per wave of a matrix tile
constexpr int kChunkRows = kThreads;            // rows per partial sum of R
constexpr int kSmallSetTiles = 256;             // compute units of the chip
constexpr int kVecIters = 4;                    // vector tile = kThreads*vec*kVecIters
static_assert(kStreamWaves >= 1 && kStreamWaves <= 16, "a workgroup holds at most 16 waves");
static_assert(kRingF32 >= 1 && kRingBF16 >= 1, "a ring holds at least one row load");
static_assert(kRowsPerWave >= 1 && kRowsPerWave <= kMaxRowsPerWave, "rows per wave");
static_assert(kBlockLanes >= 1 && kBlockLanes <= kWave && (kBlockLanes & (kBlockLanes - 1)) == 0,
              "a column block is a power of two of lanes, at most one wave");

enum : int32_t { DT_F32 = 0, DT_BF16 = 1 };
enum : int32_t { KIND_MATRIX = 0, KIND_VECTOR = 1 };
enum : int32_t { FIN_ROWS = 0, FIN_COLS = 1 };

// Finalisation workgroups: 256 threads, or 1024 for sets with a matrix of
// more than 512 row stripes (about 16K rows), whose column items need more
// stripe lanes than 256 threads hold at 16 columns each.  Every thread of
// the finalisation handles 4 rows or 4 columns with 16-byte accesses to the
// partial sums.
#ifndef RK_FIN_LARGE_LOG2
#define RK_FIN_LARGE_LOG2 10
#endif
constexpr int kFinSmallLog2 = 8;
constexpr int kFinLargeLog2 = RK_FIN_LARGE_LOG2;
#ifndef RK_FIN_LOADS
#define RK_FIN_LOADS 8
#endif
#ifndef RK_FIN_ROW_LOADS
#define RK_FIN_ROW_LOADS 4
#endif
constexpr int kFinLoads = RK_FIN_LOADS;         // 16-byte column partial loads in flight per thread
constexpr int kFinRowLoads = RK_FIN_ROW_LOADS;  // the same for row partials (row items)
static_assert(kFinLargeLog2 >= kFinSmallLog2 && kFinLargeLog2 <= 10, "finalisation workgroup");

// Row partials are [ncb][pad4(m)]: each block's row sums padded to a
// multiple of 4 floats, so that the finalisation reads 4 rows' partial sums
// with one 16-byte access (the padding is never written or used).  Column
// partials are kept in groups of 16 columns, each group holding all of its
// stripes one after the other ([ceil(n/16)][nrs][16], 64-byte rows): a
// finalisation item then reads each group's stripes as one contiguous run.
constexpr int64_t pad4(int64_t v) { return (v + 3) & ~int64_t(3); }
constexpr int kColGroup = 16;
constexpr int64_t colpart_index(int64_t j, int64_t stripe, int64_t nrs)
{
    return (j >> 4) * (nrs << 4) + (stripe << 4) + (j & 15);
}
constexpr int64_t colpart_floats(int64_t n, int64_t nrs) { return ((n + 15) >> 4) * (nrs << 4); }

// One parameter tensor.  Offsets are in floats into the context workspace.
struct TensorDesc {
    void *x;           // m*n of dtype
    float *p;          // m*n momentum
    float *r;          // m row factor (matrix)
    float *c;          // n column factor (matrix)
    float *xi;         // m*n element-wise friction (vector / full iKFAD)
    int64_t m, n;
    int64_t rowpart;   // [ncb][pad4(m)] row partial sums of [P^(1)]^2
    int64_t colpart;   // [ceil(n/16)][nrs][16] column partial sums of [P^(1)]^2
    int64_t chunk;     // [nchunk] partial sums of R
    int32_t nchunk, ncb, nrs, dtype;
    int32_t kind, vec;
};

// One workgroup of the streaming pass.
struct Tile {
    int64_t start;     // matrix: first row; vector: first element
    int32_t tensor;
    int32_t count;     // matrix: rows (<= kStreamWaves * rpw); vector: elements
    int32_t col0;      // matrix: first column of the block
    int32_t ncols;     // matrix: columns of the block (multiple of vec)
    int32_t stripe;    // matrix: row-stripe index (row of the column partials)
    int32_t cb;        // matrix: column-block index (row of the row partials)
    int32_t lanes_log2;// matrix: log2 of lanes per row (rows per load = 64 >> it)
    int32_t kind;
    int32_t vec;       // elements per lane access: 1, 4 or 8
    int32_t dtype;
    int32_t rpw;       // matrix: rows per wave (<= kMaxRowsPerWave)
    int32_t pad;
};

// A contiguous range of the tile table served by one launch of the
// streaming kernel: the matrix tiles of one storage type (4-wide ones
// first, then one-column ones, which the 4-wide instantiation also serves),
// then that type's vector tiles.  vec (4, or 1 when the type has no 4-wide
// matrix tile) selects the kernel instantiation.
struct TileGroup {
    int32_t dtype;
    int32_t vec;
    int64_t begin;
    int64_t count;
};

// One workgroup of the finalisation pass (one launch), T threads.
//   FIN_ROWS  4T rows, 4 per thread: R update and one partial sum of R per
//             256 rows (one wave).  start is a multiple of 4T.
//   FIN_COLS  4T / S columns, all row stripes: C update.  Thread t takes
//             columns 4(t mod 4) .. +3 of group t / 4S (16 columns each)
//             and stripe lane (t / 4) mod S, S = 2^lanes_log2 the smallest
//             power of two that leaves each thread at most kFinLoads
//             stripes, capped so that an item keeps at least one group.
//             start is a multiple of 16.
// An item carries what it needs of its tensor, so that a workgroup's first
// load is its only descriptor load.
struct FinItem {
    float *f;          // R (FIN_ROWS) or C (FIN_COLS) of the tensor
    int64_t len;       // m (FIN_ROWS) or n (FIN_COLS)
    int64_t part;      // workspace offset of the tensor's row / column partials
    int64_t chunk;     // FIN_ROWS: workspace offset of the first partial sum of R it writes
    int32_t tensor;
    int32_t kind;
    int32_t start;     // first row / column
    int32_t count;     // rows / columns
    int32_t nparts;    // FIN_ROWS: column blocks (ncb); FIN_COLS: row stripes (nrs)
    int32_t lanes_log2;// FIN_COLS: log2 of the stripe lanes S
};

// Step coefficients, computed in fp64 on the host and rounded once.
// h and e^{-gamma h} enter every step of a momentum that can carry the
// same value for many steps, so their fp32 rounding errors would add up
// (about 2e-8 relative per step for d at gamma h = 1e-4, amplified where a
// momentum is a cancelling sum of many kicks).  The kernels therefore apply
// h as h_hi + h_lo and d as 1 + dm1, each with fused multiply-adds.
struct Coeffs {
    float h;           // step size (h_hi: h rounded to fp32)
    float h_lo;        // h - h_hi
    float kh;          // -(h/2) log2(e): exp(-(h/2) v) = exp2(kh v)
    float a;           // e^{-alpha h}
    float kappa;       // (1 - e^{-alpha h}) / (mu alpha)
    float d;           // e^{-gamma h}
    float dm1;         // e^{-gamma h} - 1, from expm1
    float eps;         // eps_stab
};

// Adafactor-m step coefficients (fp64 on the host, rounded once).
struct AdaCoeffs {
    float b;           // beta2_t = 1 - t^decay_rate
    float omb;         // 1 - beta2_t
    float eps1;        // added to G^2
    float beta1;       // first-moment decay
    float omb1;        // 1 - beta1
    float h;           // step size
    float eps2;        // floor of RMS(X) in the parameter scale
    float clip;        // update clipping threshold (<= 0: off)
    int32_t scale;     // parameter scaling on
    int32_t pad;
};

// Tiles of one tensor in the tile table (they are contiguous).
struct TensorRange {
    int64_t tile0;
    int64_t ntile;
    int64_t elems;
};

}  // namespace rk
