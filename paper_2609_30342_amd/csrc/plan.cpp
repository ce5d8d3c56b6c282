// plan.cpp -- validation, tile tables and workspace layout (host only).
#include "plan.hpp"

#include <cmath>
#include <cstdint>
#include <initializer_list>

namespace rk {

namespace {

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int esize(int32_t dt) { return dt == DT_BF16 ? 2 : 4; }

constexpr int64_t kMaxDim = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxElems = (int64_t(1) << 62) - 1;

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// 128-bit path when rows stay 16-byte aligned, else narrower accesses.
// bf16 matrices take 4 elements per lane (64-bit x and g accesses).
int32_t matrix_vec(const rikfad_tensor &t)
{
    if (t.dtype == RIKFAD_FP32)
        return (t.n % 4 == 0 && aligned(t.x, 16) && aligned(t.g, 16) && aligned(t.p, 16)) ? 4 : 1;
    if (t.n % 4 == 0 && aligned(t.x, 8) && aligned(t.g, 8) && aligned(t.p, 16)) return 4;
    return 1;
}

int32_t flat_vec(int32_t dtype, const void *x, const void *g, const void *p, const void *xi)
{
    if (dtype == RIKFAD_FP32)
        return (aligned(x, 16) && aligned(g, 16) && aligned(p, 16) && aligned(xi, 16)) ? 4 : 1;
    if (aligned(x, 16) && aligned(g, 16) && aligned(p, 16) && aligned(xi, 16)) return 8;
    if (aligned(x, 8) && aligned(g, 8) && aligned(p, 16) && aligned(xi, 16)) return 4;
    return 1;
}

rikfad_status check_common(int64_t i, const void *x, const void *g, const void *p, int64_t m,
                           int64_t n, int32_t dtype, int32_t reserved, std::string &err)
{
    const std::string who = "tensor " + std::to_string(i) + ": ";
    if (reserved != 0) { err = who + "reserved field must be 0"; return RIKFAD_EINVAL; }
    if (dtype != RIKFAD_FP32 && dtype != RIKFAD_BF16) {
        err = who + "unsupported dtype " + std::to_string(dtype);
        return RIKFAD_EDTYPE;
    }
    if (m < 1 || n < 1) { err = who + "zero-size tensor (m and n must be >= 1)"; return RIKFAD_EINVAL; }
    if (m > kMaxDim || n > kMaxDim || m > kMaxElems / n) {
        err = who + "too large (m, n < 2^31 and m*n < 2^62 required)";
        return RIKFAD_EINVAL;
    }
    if (!x || !g || !p) { err = who + "x, g and p must be non-NULL"; return RIKFAD_EINVAL; }
    if (!aligned(x, esize(dtype)) || !aligned(g, esize(dtype)) || !aligned(p, 4)) {
        err = who + "pointer not aligned to its element size";
        return RIKFAD_EALIGN;
    }
    return RIKFAD_OK;
}

void add_flat_tiles(Plan &pl, int32_t tensor, int64_t k, int32_t dtype, int32_t vec)
{
    const int64_t per = int64_t(kThreads) * vec * kVecIters;
    for (int64_t s = 0; s < k; s += per) {
        Tile t{};
        t.start = s;
        t.tensor = tensor;
        t.count = static_cast<int32_t>(k - s < per ? k - s : per);
        t.kind = KIND_VECTOR;
        t.vec = vec;
        t.dtype = dtype;
        pl.tiles.push_back(t);
    }
}

}  // namespace

rikfad_status check_hparams(const rikfad_hparams *hp, std::string &err)
{
    if (!hp) { err = "hparams is NULL"; return RIKFAD_EINVAL; }
    if (!(std::isfinite(hp->h) && std::isfinite(hp->gamma) && std::isfinite(hp->alpha) &&
          std::isfinite(hp->mu) && std::isfinite(hp->eps_stab))) {
        err = "hyperparameters must be finite";
        return RIKFAD_EINVAL;
    }
    if (!(hp->h > 0) || !(hp->mu > 0) || hp->alpha < 0 || hp->gamma < 0 || hp->eps_stab < 0) {
        err = "need h > 0, mu > 0, alpha >= 0, gamma >= 0, eps_stab >= 0";
        return RIKFAD_EINVAL;
    }
    const Coeffs k = make_coeffs(*hp);
    if (!(std::isfinite(k.h) && std::isfinite(k.kh) && std::isfinite(k.kappa) &&
          std::isfinite(k.eps))) {
        err = "hyperparameters give step coefficients outside the fp32 range";
        return RIKFAD_EINVAL;
    }
    return RIKFAD_OK;
}

// App. A Table rows C and D: e^{-alpha h}, (1 - e^{-alpha h})/(mu alpha)
// evaluated as -expm1(-alpha h)/(mu alpha) (alpha = 0: its limit h/mu),
// e^{-gamma h} (also as expm1(-gamma h)); h as an fp32 pair; and
// -(h/2) log2(e) so that the half-kick is one exp2.  All in fp64, each
// rounded once to fp32.
Coeffs make_coeffs(const rikfad_hparams &hp)
{
    const double ah = hp.alpha * hp.h;
    Coeffs k;
    k.h = static_cast<float>(hp.h);
    k.h_lo = static_cast<float>(hp.h - static_cast<double>(k.h));
    k.kh = static_cast<float>(-0.5 * hp.h * 1.44269504088896340736);
    k.a = static_cast<float>(std::exp(-ah));
    k.kappa = static_cast<float>(hp.alpha > 0 ? -std::expm1(-ah) / (hp.mu * hp.alpha)
                                              : hp.h / hp.mu);
    k.d = static_cast<float>(std::exp(-hp.gamma * hp.h));
    k.dm1 = static_cast<float>(std::expm1(-hp.gamma * hp.h));
    k.eps = static_cast<float>(hp.eps_stab);
    return k;
}

bool grad_fits(const void *g, int32_t dtype, int32_t vec)
{
    if (!g) return false;
    return aligned(g, static_cast<uintptr_t>(esize(dtype)) * static_cast<uintptr_t>(vec));
}

// Column blocks of a matrix: kBlockLanes lanes x vec columns each; a narrow
// last block uses the smallest power-of-two lane count that covers it.
// Tiles are kStreamWaves waves x rpw rows, rpw = base rows per wave, grown
// for narrow blocks so that every tile has about the same number of
// accesses.  Returns rpw.
namespace {
struct Block { int32_t col0, ncols, llog; };

int matrix_blocks(int64_t n, int32_t vec, int base, std::vector<Block> &blocks)
{
    blocks.clear();
    int blog = 0;
    while ((1 << blog) < kBlockLanes) ++blog;
    const int64_t lanes = n / vec;
    const int64_t full = lanes >> blog, rem = lanes & ((int64_t(1) << blog) - 1);
    for (int64_t b = 0; b < full; ++b)
        blocks.push_back({static_cast<int32_t>((b << blog) * vec),
                          static_cast<int32_t>((int64_t(1) << blog) * vec), blog});
    if (rem > 0) {
        int llog = 0;
        while ((int64_t(1) << llog) < rem) ++llog;
        blocks.push_back({static_cast<int32_t>((full << blog) * vec),
                          static_cast<int32_t>(rem * vec), llog});
    }
    const int lead_llog = blocks.front().llog;
    int rpw = base << (blog - (lead_llog < blog ? lead_llog : blog));
    return rpw > kMaxRowsPerWave ? kMaxRowsPerWave : rpw;
}
}  // namespace

rikfad_status plan_rikfad(const rikfad_tensor *t, int64_t count, Plan &pl, std::string &err,
                          int rows_per_wave)
{
    if (count < 0 || (count > 0 && !t)) {
        err = "tensor list is NULL or count < 0";
        return RIKFAD_EINVAL;
    }
    pl = Plan{};
    for (int64_t i = 0; i < count; ++i) {
        const rikfad_tensor &T = t[i];
        rikfad_status s = check_common(i, T.x, T.g, T.p, T.m, T.n, T.dtype, T.reserved, err);
        if (s != RIKFAD_OK) return s;
        const bool vec = (T.m == 1 || T.n == 1);
        float *xi = (T.m == 1) ? T.c : T.r;
        if (vec ? !xi : (!T.r || !T.c)) {
            err = "tensor " + std::to_string(i) +
                  (vec ? ": vector friction (c when m == 1, else r) is NULL"
                       : ": factors r and c must be non-NULL");
            return RIKFAD_EINVAL;
        }
        if ((T.r && !aligned(T.r, 4)) || (T.c && !aligned(T.c, 4))) {
            err = "tensor " + std::to_string(i) + ": factor pointer not 4-byte aligned";
            return RIKFAD_EALIGN;
        }
    }

    // A set with fewer matrix tiles than the chip has compute units leaves
    // most of it idle, and its step lasts as long as one tile's chain of
    // dependent row loads: halving the rows per wave doubles the tiles and
    // shortens that chain.  Sets that fill the chip keep the full rows per
    // wave, which streams at a higher rate.
    int rpw_base = rows_per_wave > 0 ? rows_per_wave : kRowsPerWave;
    if (rows_per_wave <= 0) {
        int64_t ntiles = 0;
        std::vector<Block> blocks;
        for (int64_t i = 0; i < count; ++i) {
            const rikfad_tensor &T = t[i];
            if (T.m == 1 || T.n == 1) continue;
            const int rpw = matrix_blocks(T.n, matrix_vec(T), kRowsPerWave, blocks);
            ntiles += static_cast<int64_t>(blocks.size()) *
                      ceil_div(T.m, int64_t(kStreamWaves) * rpw);
        }
        if (ntiles < kSmallSetTiles && kRowsPerWave > 1) rpw_base = kRowsPerWave / 2;
    }

    if (rpw_base > kMaxRowsPerWave) {
        err = "rows per wave above " + std::to_string(kMaxRowsPerWave);
        return RIKFAD_EINVAL;
    }

    int64_t ws = 0;
    pl.tensors.resize(static_cast<size_t>(count));
    pl.grads.resize(static_cast<size_t>(count));
    // Matrix tiles by class (fp32 v4, fp32 v1, bf16 v4, bf16 v1); vector
    // tiles by dtype.
    constexpr int kClasses = 4;
    const int32_t class_dtype[kClasses] = {DT_F32, DT_F32, DT_BF16, DT_BF16};
    const int32_t class_vec[kClasses] = {4, 1, 4, 1};
    std::vector<Tile> mat_tiles[kClasses];
    std::vector<Tile> vec_tiles[2];
    std::vector<FinItem> col_items;
    for (int64_t i = 0; i < count; ++i) {
        const rikfad_tensor &T = t[i];
        TensorDesc &d = pl.tensors[static_cast<size_t>(i)];
        d = TensorDesc{};
        d.x = T.x;
        d.p = T.p;
        d.r = T.r;
        d.c = T.c;
        d.m = T.m;
        d.n = T.n;
        d.dtype = T.dtype;
        pl.grads[static_cast<size_t>(i)] = T.g;
        const int64_t mn = T.m * T.n;
        const int64_t eb = esize(T.dtype);
        pl.elements += mn;
        pl.ikfad_state_bytes += 8 * mn;
        if (T.m == 1 || T.n == 1) {
            d.kind = KIND_VECTOR;
            d.xi = (T.m == 1) ? T.c : T.r;
            d.vec = flat_vec(T.dtype, T.x, T.g, T.p, d.xi);
            pl.vectors += 1;
            pl.state_bytes += 8 * mn;
            pl.min_bytes += mn * (3 * eb + 16);        // read x g p xi, write x p xi
            pl.stream_min_bytes += mn * (3 * eb + 16);
            Plan tmp;
            add_flat_tiles(tmp, static_cast<int32_t>(i), mn, T.dtype, d.vec);
            std::vector<Tile> &vt = vec_tiles[T.dtype == DT_F32 ? 0 : 1];
            vt.insert(vt.end(), tmp.tiles.begin(), tmp.tiles.end());
            continue;
        }
        d.kind = KIND_MATRIX;
        d.vec = matrix_vec(T);
        pl.matrices += 1;
        pl.state_bytes += 4 * mn + 4 * (T.m + T.n);
        pl.min_bytes += mn * (3 * eb + 8) + 8 * (T.m + T.n);   // x g p in, x p out; R C
        pl.stream_min_bytes += mn * (3 * eb + 8) + 4 * (T.m + T.n); // R, C read only

        std::vector<Block> blocks;
        const int rpw = matrix_blocks(T.n, d.vec, rpw_base, blocks);
        const int64_t stripe_rows = int64_t(kStreamWaves) * rpw;
        d.ncb = static_cast<int32_t>(blocks.size());
        d.nrs = static_cast<int32_t>(ceil_div(T.m, stripe_rows));
        d.nchunk = static_cast<int32_t>(ceil_div(T.m, kChunkRows));
        d.rowpart = ws;
        ws += round_up(pad4(T.m) * d.ncb, 64);
        d.colpart = ws;
        ws += round_up(colpart_floats(T.n, d.nrs), 64);
        d.chunk = ws;
        ws += round_up(d.nchunk, 64);

        int cls = 0;
        while (!(class_dtype[cls] == T.dtype && class_vec[cls] == d.vec)) ++cls;
        // Workgroups go to the 8 XCDs round-robin (launch index mod 8).  When
        // a matrix's last column block is narrow, the tiles of a stripe carry
        // unequal work, and in stripe-by-stripe order with 2 blocks every
        // narrow tile would land on the odd XCDs.  In runs of 8 stripes such
        // a matrix is therefore ordered block by block, so that all blocks of
        // one stripe lie 8 apart and run on the same XCD.
        const bool group8 = blocks.back().llog < blocks.front().llog;
        std::vector<std::pair<int32_t, int32_t>> order;     // (stripe, block)
        for (int32_t s0 = 0; s0 < d.nrs; s0 += 8) {
            const int32_t k = d.nrs - s0 < 8 ? d.nrs - s0 : 8;
            if (group8 && k == 8) {
                for (int32_t b = 0; b < d.ncb; ++b)
                    for (int32_t q = 0; q < 8; ++q) order.push_back({s0 + q, b});
            } else {
                for (int32_t q = 0; q < k; ++q)
                    for (int32_t b = 0; b < d.ncb; ++b) order.push_back({s0 + q, b});
            }
        }
        for (const std::pair<int32_t, int32_t> &sb : order) {
            const int32_t s = sb.first, b = sb.second;
            Tile tl{};
            tl.start = int64_t(s) * stripe_rows;
            tl.tensor = static_cast<int32_t>(i);
            tl.count = static_cast<int32_t>(
                T.m - tl.start < stripe_rows ? T.m - tl.start : stripe_rows);
            tl.col0 = blocks[static_cast<size_t>(b)].col0;
            tl.ncols = blocks[static_cast<size_t>(b)].ncols;
            tl.stripe = s;
            tl.cb = b;
            tl.lanes_log2 = blocks[static_cast<size_t>(b)].llog;
            tl.kind = KIND_MATRIX;
            tl.vec = d.vec;
            tl.dtype = T.dtype;
            tl.rpw = rpw;
            mat_tiles[cls].push_back(tl);
        }
    }
    // Finalisation items (layout.hpp), sized for the set's workgroup: 1024
    // threads when some matrix has more stripes than 256 threads cover at
    // 16 columns per item and kFinLoads stripes per thread.
    for (const TensorDesc &d : pl.tensors)
        if (d.kind == KIND_MATRIX && d.nrs > (int64_t(kFinLoads) << (kFinSmallLog2 - 2)))
            pl.fin_log2 = kFinLargeLog2;
    const int64_t fin_threads = int64_t(1) << pl.fin_log2;
    const int max_slog = pl.fin_log2 - 2;
    for (int64_t i = 0; i < count; ++i) {
        const TensorDesc &d = pl.tensors[static_cast<size_t>(i)];
        if (d.kind != KIND_MATRIX) continue;
        // Row items: 4 rows per thread, one partial sum of R per 256 rows.
        const int64_t rows = 4 * fin_threads;
        for (int64_t r0 = 0; r0 < d.m; r0 += rows)
            pl.fin.push_back({d.r, d.m, d.rowpart, d.chunk + r0 / kChunkRows,
                              static_cast<int32_t>(i), FIN_ROWS, static_cast<int32_t>(r0),
                              static_cast<int32_t>(d.m - r0 < rows ? d.m - r0 : rows), d.ncb, 0});
        // Column items: S stripe lanes x fin_threads / S threads of 4 columns.
        int slog = 0;
        while (slog < max_slog && (int64_t(kFinLoads) << slog) < d.nrs) ++slog;
        const int64_t cols = 4 * (fin_threads >> slog);
        for (int64_t j0 = 0; j0 < d.n; j0 += cols)
            col_items.push_back({d.c, d.n, d.colpart, 0, static_cast<int32_t>(i), FIN_COLS,
                                 static_cast<int32_t>(j0),
                                 static_cast<int32_t>(d.n - j0 < cols ? d.n - j0 : cols), d.nrs,
                                 slog});
    }
    // One launch per storage type: its 4-wide matrix tiles, then its
    // one-column matrix tiles (served by the same launch), then its vector
    // tiles; the group's width selects the kernel instantiation.
    auto add_group = [&](int32_t dtype, int32_t vec, std::initializer_list<int> classes,
                         bool vectors) {
        TileGroup gr{dtype, vec, static_cast<int64_t>(pl.tiles.size()), 0};
        for (int cls : classes) {
            pl.tiles.insert(pl.tiles.end(), mat_tiles[cls].begin(), mat_tiles[cls].end());
            pl.matrix_tiles += static_cast<int64_t>(mat_tiles[cls].size());
        }
        if (vectors) {
            const std::vector<Tile> &vt = vec_tiles[dtype == DT_F32 ? 0 : 1];
            pl.tiles.insert(pl.tiles.end(), vt.begin(), vt.end());
        }
        gr.count = static_cast<int64_t>(pl.tiles.size()) - gr.begin;
        if (gr.count > 0) pl.groups.push_back(gr);
    };
    add_group(DT_F32, mat_tiles[0].empty() ? 1 : 4, {0, 1}, true);
    add_group(DT_BF16, mat_tiles[2].empty() ? 1 : 4, {2, 3}, true);
    pl.row_items = static_cast<int64_t>(pl.fin.size());
    pl.fin.insert(pl.fin.end(), col_items.begin(), col_items.end());
    pl.ws_floats = ws;
    if (pl.tiles.size() > static_cast<size_t>(INT32_MAX) || pl.fin.size() > static_cast<size_t>(INT32_MAX)) {
        err = "parameter set needs more than 2^31 workgroups";
        return RIKFAD_EINVAL;
    }
    return RIKFAD_OK;
}

rikfad_status plan_ikfad(const ikfad_tensor *t, int64_t count, Plan &pl, std::string &err)
{
    if (count < 0 || (count > 0 && !t)) {
        err = "tensor list is NULL or count < 0";
        return RIKFAD_EINVAL;
    }
    pl = Plan{};
    pl.tensors.resize(static_cast<size_t>(count));
    pl.grads.resize(static_cast<size_t>(count));
    for (int64_t i = 0; i < count; ++i) {
        const ikfad_tensor &T = t[i];
        rikfad_status s = check_common(i, T.x, T.g, T.p, T.m, T.n, T.dtype, T.reserved, err);
        if (s != RIKFAD_OK) return s;
        if (!T.xi) { err = "tensor " + std::to_string(i) + ": xi is NULL"; return RIKFAD_EINVAL; }
        if (!aligned(T.xi, 4)) {
            err = "tensor " + std::to_string(i) + ": xi not 4-byte aligned";
            return RIKFAD_EALIGN;
        }
        TensorDesc &d = pl.tensors[static_cast<size_t>(i)];
        d = TensorDesc{};
        d.x = T.x;
        d.p = T.p;
        d.xi = T.xi;
        d.m = T.m;
        d.n = T.n;
        d.dtype = T.dtype;
        d.kind = KIND_VECTOR;
        d.vec = flat_vec(T.dtype, T.x, T.g, T.p, T.xi);
        pl.grads[static_cast<size_t>(i)] = T.g;
        const int64_t mn = T.m * T.n;
        pl.elements += mn;
        pl.vectors += 1;
        pl.state_bytes += 8 * mn;
        pl.ikfad_state_bytes += 8 * mn;
        pl.min_bytes += mn * (3 * esize(T.dtype) + 16);
        pl.stream_min_bytes += mn * (3 * esize(T.dtype) + 16);
        add_flat_tiles(pl, static_cast<int32_t>(i), mn, T.dtype, d.vec);
    }
    if (pl.tiles.size() > static_cast<size_t>(INT32_MAX)) {
        err = "parameter set needs more than 2^31 workgroups";
        return RIKFAD_EINVAL;
    }
    return RIKFAD_OK;
}

}  // namespace rk
