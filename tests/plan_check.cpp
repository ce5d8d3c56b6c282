// plan_check.cpp -- host-side check of the tile and finalisation tables.
//
// Builds random parameter lists, plans them with the library's own planner
// and replays, on the CPU, the index arithmetic the gfx950 kernels perform
// for every workgroup, wave and lane: every load and store address must lie
// inside its buffer, every matrix and vector element must be updated
// exactly once, every partial sum written exactly once and read only where
// it was written, and the workspace regions must not overlap.  Built with
// -fsanitize=address,undefined by the test that runs it.
#include <cstdint>
#include <cstdio>
#include <random>
#include <string>
#include <vector>

#include "../paper_2609_30342_amd/csrc/plan.hpp"

using namespace rk;

static int failures = 0;
#define CHECK(cond, ...)                                            \
    do {                                                            \
        if (!(cond)) {                                              \
            if (failures < 20) {                                    \
                std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
                std::fprintf(stderr, __VA_ARGS__);                  \
                std::fprintf(stderr, "\n");                         \
            }                                                       \
            ++failures;                                             \
        }                                                           \
    } while (0)

struct Marks {
    std::vector<uint8_t> v;
    void init(int64_t n) { v.assign(static_cast<size_t>(n), 0); }
    void hit(int64_t i, const char *what)
    {
        CHECK(i >= 0 && i < static_cast<int64_t>(v.size()), "%s index %lld out of [0,%zu)", what,
              (long long)i, v.size());
        if (i >= 0 && i < static_cast<int64_t>(v.size())) {
            CHECK(v[static_cast<size_t>(i)] == 0, "%s index %lld written twice", what, (long long)i);
            v[static_cast<size_t>(i)] = 1;
        }
    }
    bool all() const
    {
        for (uint8_t b : v)
            if (!b) return false;
        return true;
    }
    // every entry of rows of `stride` entries whose column is below `used`
    // (the padding at the end of each row is never written)
    bool all_rows(int64_t stride, int64_t used) const
    {
        for (size_t i = 0; i < v.size(); ++i)
            if (static_cast<int64_t>(i) % stride < used && !v[i]) return false;
        return true;
    }
};

static int ring_depth(int32_t dtype) { return dtype == DT_F32 ? kRingF32 : kRingBF16; }

// Replays rikfad_stream_kernel's matrix-tile indexing.
static void check_matrix_tile(const Plan &pl, const Tile &tl, std::vector<Marks> &elems,
                              std::vector<Marks> &rowp, std::vector<Marks> &colp)
{
    const TensorDesc &td = pl.tensors[static_cast<size_t>(tl.tensor)];
    const int64_t m = td.m, n = td.n, mn = m * n;
    const int V = tl.vec, llog = tl.lanes_log2, L = 1 << llog, G = kWave >> llog;
    const int B = ring_depth(tl.dtype);
    CHECK(tl.rpw >= 1 && tl.rpw <= kMaxRowsPerWave, "rpw %d", tl.rpw);
    CHECK(tl.ncols % V == 0 && tl.ncols <= L * V, "ncols %d L %d V %d", tl.ncols, L, V);
    CHECK(tl.col0 % V == 0 && tl.col0 + tl.ncols <= n, "col range");
    CHECK(tl.count <= kStreamWaves * tl.rpw && tl.start + tl.count <= m, "row range");
    for (int wave = 0; wave < kStreamWaves; ++wave) {
        const int64_t r0 = tl.start + int64_t(wave) * tl.rpw;
        int nr = static_cast<int>(tl.start + tl.count - r0);
        nr = nr < 0 ? 0 : (nr > tl.rpw ? tl.rpw : nr);
        const int nld = (nr + G - 1) >> (6 - llog);
        for (int lane = 0; lane < kWave; ++lane) {
            const int seg = lane >> llog, sl = lane & (L - 1), ccol = sl * V;
            const bool colok = ccol < tl.ncols;
            const int64_t col = tl.col0 + ccol;
            const int64_t lcol = colok ? col : tl.col0;
            auto check_load = [&](int rl) {
                const bool ok = colok && rl < nr;
                const int64_t off = ok ? (r0 + rl) * n + lcol : r0 * n + lcol;
                CHECK(off >= 0 && off + V <= mn && off % V == 0, "load off %lld mn %lld",
                      (long long)off, (long long)mn);
            };
            if (nr > 0)
                for (int u = 0; u < B; ++u) check_load(u * G + seg);
            if (colok) CHECK(col + V <= n, "c load");
            if (lane < nr) CHECK(r0 + lane < m, "r load");
            for (int ld0 = 0; ld0 < nld; ld0 += B) {
                for (int u = 0; u < B; ++u) {
                    const int ld = ld0 + u, rl = ld * G + seg;
                    if (colok && rl < nr) {
                        for (int i = 0; i < V; ++i)
                            elems[static_cast<size_t>(tl.tensor)].hit((r0 + rl) * n + col + i,
                                                                      "element");
                    }
                    if (ld + B < nld) check_load((ld + B) * G + seg);
                }
            }
            if (lane < nr)
                rowp[static_cast<size_t>(tl.tensor)].hit(int64_t(tl.cb) * pad4(m) + r0 + lane,
                                                         "rowpart");
        }
    }
    for (int j = 0; j < tl.ncols; ++j)
        colp[static_cast<size_t>(tl.tensor)].hit(colpart_index(tl.col0 + j, tl.stripe, td.nrs),
                                                 "colpart");
}

static void check_vector_tile(const Plan &pl, const Tile &tl, std::vector<Marks> &elems)
{
    const TensorDesc &td = pl.tensors[static_cast<size_t>(tl.tensor)];
    const int64_t k = td.m * td.n;
    CHECK(tl.start % tl.vec == 0 && tl.start + tl.count <= k, "vector tile range");
    for (int64_t e = 0; e < tl.count; ++e)
        elems[static_cast<size_t>(tl.tensor)].hit(tl.start + e, "vector element");
}

static void check_plan(const Plan &pl, int64_t count)
{
    // 1024-thread finalisation exactly when some matrix has more row
    // stripes than 64 stripe lanes of kFinLoads loads cover
    bool tall = false;
    for (const TensorDesc &td : pl.tensors)
        tall = tall || (td.kind == KIND_MATRIX && td.nrs > kFinLoads * 64);
    CHECK(pl.fin_log2 == (tall ? kFinLargeLog2 : kFinSmallLog2), "finalisation workgroup size");
    std::vector<Marks> elems(static_cast<size_t>(count)), rowp(static_cast<size_t>(count)),
        colp(static_cast<size_t>(count)), chunks(static_cast<size_t>(count)),
        cols(static_cast<size_t>(count)), rows(static_cast<size_t>(count));
    // workspace regions
    std::vector<std::pair<int64_t, int64_t>> regions;
    for (int64_t i = 0; i < count; ++i) {
        const TensorDesc &td = pl.tensors[static_cast<size_t>(i)];
        elems[static_cast<size_t>(i)].init(td.m * td.n);
        if (td.kind == KIND_MATRIX) {
            rowp[static_cast<size_t>(i)].init(int64_t(td.ncb) * pad4(td.m));
            colp[static_cast<size_t>(i)].init(colpart_floats(td.n, td.nrs));
            chunks[static_cast<size_t>(i)].init(td.nchunk);
            cols[static_cast<size_t>(i)].init(td.n);
            rows[static_cast<size_t>(i)].init(td.m);
            CHECK(td.rowpart % 4 == 0 && td.colpart % 4 == 0, "partials not 16-byte aligned");
            regions.push_back({td.rowpart, int64_t(td.ncb) * pad4(td.m)});
            regions.push_back({td.colpart, colpart_floats(td.n, td.nrs)});
            regions.push_back({td.chunk, td.nchunk});
        }
    }
    for (size_t a = 0; a < regions.size(); ++a) {
        CHECK(regions[a].first >= 0 && regions[a].first + regions[a].second <= pl.ws_floats,
              "workspace region outside");
        for (size_t b = a + 1; b < regions.size(); ++b) {
            const bool disjoint = regions[a].first + regions[a].second <= regions[b].first ||
                                  regions[b].first + regions[b].second <= regions[a].first;
            CHECK(disjoint || regions[a].second == 0 || regions[b].second == 0, "regions overlap");
        }
    }
    // groups partition the tile table, one group per storage type; a
    // group's matrix tiles are its own width or one-column (served by the
    // same instantiation), and a one-column group holds no wider tile.
    int64_t covered = 0;
    int ngroups[2] = {0, 0};
    for (const TileGroup &g : pl.groups) {
        CHECK(g.begin == covered, "groups not contiguous");
        CHECK(g.count > 0, "empty group");
        const int dt = g.dtype == DT_F32 ? 0 : 1;
        CHECK(g.vec == 4 || g.vec == 1, "group width %d", g.vec);
        CHECK(ngroups[dt] == 0, "two groups of one storage type");
        ++ngroups[dt];
        covered += g.count;
        for (int64_t t = g.begin; t < g.begin + g.count; ++t) {
            const Tile &tl = pl.tiles[static_cast<size_t>(t)];
            CHECK(tl.dtype == g.dtype, "tile dtype vs group");
            if (tl.kind == KIND_MATRIX) CHECK(tl.vec == g.vec || tl.vec == 1, "tile vec vs group");
        }
    }
    CHECK(covered == static_cast<int64_t>(pl.tiles.size()), "groups do not cover tiles");
    for (const Tile &tl : pl.tiles) {
        if (tl.kind == KIND_MATRIX) check_matrix_tile(pl, tl, elems, rowp, colp);
        else check_vector_tile(pl, tl, elems);
    }
    // finalisation items: replays rikfad_finalize_kernel's indexing (4 rows
    // or 4 columns per thread, 16-byte partial-sum reads)
    const int T = 1 << pl.fin_log2;
    const int64_t nfin = static_cast<int64_t>(pl.fin.size());
    for (int64_t q = 0; q < nfin; ++q) {
        const FinItem &it = pl.fin[static_cast<size_t>(q)];
        const TensorDesc &td = pl.tensors[static_cast<size_t>(it.tensor)];
        CHECK(td.kind == KIND_MATRIX, "finalisation item on a vector");
        if (it.kind == FIN_ROWS) {
            CHECK(q < pl.row_items, "row item after the row range");
            CHECK(it.count >= 1 && it.count <= 4 * T, "row item count");
            CHECK(it.start % (4 * T) == 0 && it.chunk == td.chunk + it.start / kChunkRows,
                  "row item alignment");
            CHECK(it.f == td.r && it.len == td.m && it.part == td.rowpart && it.nparts == td.ncb,
                  "row item descriptor");
            const int64_t mp = pad4(td.m);
            for (int t = 0; t < T; ++t) {
                const int t0 = 4 * t;
                if (t0 >= it.count) continue;
                const int nv = it.count - t0 < 4 ? it.count - t0 : 4;
                const int64_t i0 = int64_t(it.start) + t0;
                for (int cb0 = 0; cb0 < td.ncb; cb0 += kFinRowLoads)
                    for (int u = 0; u < kFinRowLoads; ++u) {
                        const int cb = cb0 + u < td.ncb ? cb0 + u : td.ncb - 1;
                        const int64_t off = int64_t(cb) * mp + i0;
                        CHECK(off % 4 == 0 && off + 4 <= int64_t(td.ncb) * mp, "rowpart read");
                        if (cb0 + u < td.ncb)
                            for (int j = 0; j < nv; ++j)
                                CHECK(rowp[static_cast<size_t>(it.tensor)]
                                          .v[static_cast<size_t>(off + j)] == 1,
                                      "rowpart read before written");
                    }
                for (int j = 0; j < nv; ++j)
                    rows[static_cast<size_t>(it.tensor)].hit(i0 + j, "row item row");
            }
            for (int w = 0; w < T / kWave; ++w)
                if (w * kChunkRows < it.count)
                    chunks[static_cast<size_t>(it.tensor)].hit(it.chunk - td.chunk + w, "chunk");
        } else {
            // thread t: columns 4(t mod 4) .. + 3 of group t / 4S, stripe
            // lane (t / 4) mod S; every stripe of every column read once,
            // each column updated once (by lane 0), and stripe lanes enough
            // for at most kFinLoads stripes per thread unless that would
            // leave less than one group per item.
            CHECK(it.kind == FIN_COLS && q >= pl.row_items, "column item placement");
            CHECK(it.f == td.c && it.len == td.n && it.part == td.colpart && it.nparts == td.nrs,
                  "column item descriptor");
            const int slog = it.lanes_log2, max_slog = pl.fin_log2 - 2;
            CHECK(slog >= 0 && slog <= max_slog, "stripe lanes log2 %d", slog);
            const int S = 1 << slog, ncol = 4 * (T >> slog);
            CHECK(it.count >= 1 && it.count <= ncol && it.start % kColGroup == 0,
                  "column item count %d cols %d start %d", it.count, ncol, it.start);
            CHECK((int64_t(kFinLoads) << slog) >= td.nrs || slog == max_slog,
                  "stripe lanes too few for %d stripes", td.nrs);
            CHECK(slog == 0 || (int64_t(kFinLoads) << (slog - 1)) < td.nrs,
                  "stripe lanes more than needed for %d stripes", td.nrs);
            // the LDS fold past 16 stripe lanes: slots wave * 4 + c4 of the
            // group's S / 16 waves, all inside the workgroup
            if (S > kWave / 4) CHECK(T % (4 * S) == 0, "a group spans whole waves");
            const int64_t csize = colpart_floats(td.n, td.nrs);
            std::vector<int> seen(static_cast<size_t>(td.nrs) * static_cast<size_t>(ncol), 0);
            for (int t = 0; t < T; ++t) {
                const int c4 = t & 3, lane = (t >> 2) & (S - 1), g = t >> (2 + slog);
                const int c0 = 16 * g + 4 * c4;
                if (c0 >= it.count) continue;
                const int64_t j0 = int64_t(it.start) + c0;
                const int64_t base = colpart_index(j0, 0, td.nrs);
                for (int s0 = lane; s0 < td.nrs; s0 += S * kFinLoads)
                    for (int u = 0; u < kFinLoads; ++u) {
                        const int st = s0 + u * S;
                        const int stc = st < td.nrs ? st : td.nrs - 1;
                        const int64_t off = base + int64_t(stc) * kColGroup;
                        CHECK(off % 4 == 0 && off + 4 <= csize, "colpart read");
                        if (st >= td.nrs) continue;
                        for (int j = 0; j < 4 && c0 + j < it.count; ++j) {
                            CHECK(off + j == colpart_index(j0 + j, st, td.nrs), "colpart layout");
                            CHECK(colp[static_cast<size_t>(it.tensor)]
                                      .v[static_cast<size_t>(off + j)] == 1,
                                  "colpart read before written");
                            seen[static_cast<size_t>(st) * ncol + c0 + j] += 1;
                        }
                    }
                if (lane == 0)
                    for (int j = 0; j < 4 && c0 + j < it.count; ++j)
                        cols[static_cast<size_t>(it.tensor)].hit(j0 + j, "column item column");
            }
            for (int st = 0; st < td.nrs; ++st)
                for (int c = 0; c < it.count; ++c)
                    CHECK(seen[static_cast<size_t>(st) * ncol + c] == 1,
                          "stripe %d column %d read %d times", st, c,
                          seen[static_cast<size_t>(st) * ncol + c]);
        }
    }
    for (int64_t i = 0; i < count; ++i) {
        const TensorDesc &td = pl.tensors[static_cast<size_t>(i)];
        CHECK(elems[static_cast<size_t>(i)].all(), "tensor %lld (%lldx%lld) not fully covered",
              (long long)i, (long long)td.m, (long long)td.n);
        if (td.kind == KIND_MATRIX) {
            CHECK(rowp[static_cast<size_t>(i)].all_rows(pad4(td.m), td.m), "row partials incomplete");
            bool cols_done = true;
            for (int64_t st = 0; st < td.nrs; ++st)
                for (int64_t j = 0; j < td.n; ++j)
                    cols_done = cols_done && colp[static_cast<size_t>(i)]
                                                 .v[static_cast<size_t>(colpart_index(j, st, td.nrs))];
            CHECK(cols_done, "column partials incomplete");
            CHECK(chunks[static_cast<size_t>(i)].all(), "chunks incomplete");
            CHECK(rows[static_cast<size_t>(i)].all(), "row items incomplete");
            CHECK(cols[static_cast<size_t>(i)].all(), "column items incomplete");
        }
    }
}

// Rows per wave of every matrix tile of a one-tensor fp32 set m x n.
static int single_rpw(int64_t m, int64_t n, int64_t *ntiles)
{
    const uintptr_t base = uintptr_t(1) << 40;
    rikfad_tensor t{};
    t.x = reinterpret_cast<void *>(base);
    t.g = reinterpret_cast<const void *>(base + (uintptr_t(1) << 36));
    t.p = reinterpret_cast<float *>(base + (uintptr_t(2) << 36));
    t.r = reinterpret_cast<float *>(base + (uintptr_t(3) << 36));
    t.c = reinterpret_cast<float *>(base + (uintptr_t(4) << 36));
    t.m = m;
    t.n = n;
    t.dtype = RIKFAD_FP32;
    Plan pl;
    std::string err;
    if (plan_rikfad(&t, 1, pl, err) != RIKFAD_OK || pl.tiles.empty()) return -1;
    int rpw = pl.tiles[0].rpw;
    for (const Tile &tl : pl.tiles) if (tl.rpw != rpw) return -2;
    *ntiles = static_cast<int64_t>(pl.tiles.size());
    return rpw;
}

int main(int argc, char **argv)
{
    // A set with fewer tiles than compute units at the full rows per wave
    // takes half of it; a set that fills the chip keeps it.
    int64_t nt = 0;
    CHECK(single_rpw(256, 512, &nt) == kRowsPerWave / 2 && nt == 32,
          "256x512 set: rpw %d, %lld tiles", single_rpw(256, 512, &nt), (long long)nt);
    CHECK(single_rpw(768, 3072, &nt) == kRowsPerWave && nt == 288,
          "768x3072 set: rpw %d, %lld tiles", single_rpw(768, 3072, &nt), (long long)nt);
    CHECK(single_rpw(1024, 2048, &nt) == kRowsPerWave && nt == 256,
          "1024x2048 set (256 tiles): rpw %d", single_rpw(1024, 2048, &nt));
    CHECK(single_rpw(992, 2048, &nt) == kRowsPerWave / 2 && nt == 496,
          "992x2048 set (248 tiles at full rpw): rpw %d, %lld tiles", single_rpw(992, 2048, &nt),
          (long long)nt);

    {
        // A matrix whose last column block is narrow (n = 384: 256 + 128
        // columns) is ordered in runs of 8 stripes block by block, so that
        // all tiles of a stripe share their launch position mod 8 (one XCD);
        // 768 columns (three full blocks) keep stripe-by-stripe order.
        for (int64_t n : {384, 768}) {
            const uintptr_t b = uintptr_t(1) << 40;
            rikfad_tensor t{};
            t.x = reinterpret_cast<void *>(b);
            t.g = reinterpret_cast<const void *>(b + (uintptr_t(1) << 36));
            t.p = reinterpret_cast<float *>(b + (uintptr_t(2) << 36));
            t.r = reinterpret_cast<float *>(b + (uintptr_t(3) << 36));
            t.c = reinterpret_cast<float *>(b + (uintptr_t(4) << 36));
            t.m = 2048;
            t.n = n;
            t.dtype = RIKFAD_FP32;
            Plan pl;
            std::string err;
            CHECK(plan_rikfad(&t, 1, pl, err) == RIKFAD_OK, "plan 2048x%lld", (long long)n);
            std::vector<int> residue(static_cast<size_t>(pl.tensors[0].nrs), -1);
            bool same_xcd = true, stripe_major = true;
            for (size_t k = 0; k < pl.tiles.size(); ++k) {
                const Tile &tl = pl.tiles[k];
                int &r = residue[static_cast<size_t>(tl.stripe)];
                if (r < 0) r = static_cast<int>(k % 8);
                same_xcd = same_xcd && r == static_cast<int>(k % 8);
                stripe_major = stripe_major &&
                               static_cast<int64_t>(k) == int64_t(tl.stripe) * pl.tensors[0].ncb + tl.cb;
            }
            if (n == 384) CHECK(same_xcd, "n = 384: a stripe's tiles on different XCDs");
            else CHECK(stripe_major, "n = 768: order changed");
            check_plan(pl, 1);
        }
    }

    const int trials = argc > 1 ? std::atoi(argv[1]) : 300;
    std::mt19937_64 rng(12345);
    const int64_t dims[] = {1, 2, 3, 4, 5, 7, 8, 12, 16, 27, 31, 33, 63, 64, 65, 100, 127, 128,
                            129, 255, 256, 257, 300, 384, 513, 640, 768, 776, 1000, 1024, 1152,
                            1440, 2304, 3072, 4097};
    const int ndims = sizeof(dims) / sizeof(dims[0]);
    const uintptr_t base = uintptr_t(1) << 40;
    int planned = 0, rejected = 0;
    for (int trial = 0; trial < trials; ++trial) {
        const int count = static_cast<int>(rng() % 9);
        std::vector<rikfad_tensor> ts(static_cast<size_t>(count));
        bool expect_align_error = false;
        for (int i = 0; i < count; ++i) {
            rikfad_tensor &t = ts[static_cast<size_t>(i)];
            t.m = dims[rng() % ndims];
            t.n = dims[rng() % ndims];
            if (rng() % 40 == 0) t.m = 50257;
            t.dtype = (rng() % 2) ? RIKFAD_BF16 : RIKFAD_FP32;
            t.reserved = 0;
            const uintptr_t slot = base + (uintptr_t(i) << 34);
            const int es = t.dtype == RIKFAD_BF16 ? 2 : 4;
            // mostly aligned buffers, sometimes element-aligned views
            const uintptr_t offx = (rng() % 5 == 0) ? uintptr_t(es) * (rng() % 4) : 0;
            const uintptr_t offg = (rng() % 5 == 0) ? uintptr_t(es) * (rng() % 4) : 0;
            const uintptr_t offp = (rng() % 7 == 0) ? 4 * (rng() % 4) : 0;
            t.x = reinterpret_cast<void *>(slot + offx);
            t.g = reinterpret_cast<const void *>(slot + (uintptr_t(1) << 32) + offg);
            t.p = reinterpret_cast<float *>(slot + (uintptr_t(2) << 32) + offp);
            t.r = reinterpret_cast<float *>(slot + (uintptr_t(3) << 32));
            t.c = reinterpret_cast<float *>(slot + (uintptr_t(3) << 32) + (uintptr_t(1) << 31));
            if (rng() % 50 == 0) {      // a misaligned pointer must be rejected
                t.p = reinterpret_cast<float *>(reinterpret_cast<uintptr_t>(t.p) + 2);
                expect_align_error = true;
            }
        }
        Plan pl;
        std::string err;
        const rikfad_status s = plan_rikfad(ts.data(), count, pl, err);
        if (expect_align_error) {
            CHECK(s == RIKFAD_EALIGN, "misaligned p accepted (status %d)", s);
            ++rejected;
            continue;
        }
        CHECK(s == RIKFAD_OK, "plan failed: %s", err.c_str());
        if (s != RIKFAD_OK) continue;
        ++planned;
        check_plan(pl, count);
        // the Adafactor-m update pass plans the same set with 3 rows per wave
        Plan pu;
        CHECK(plan_rikfad(ts.data(), count, pu, err, 3) == RIKFAD_OK, "plan (3 rows per wave): %s",
              err.c_str());
        check_plan(pu, count);
        for (const Tile &tl : pu.tiles)
            if (tl.kind == KIND_MATRIX && tl.lanes_log2 == 6)
                CHECK(tl.rpw == 3, "full-width tile with %d rows per wave, not 3", tl.rpw);
        // its read passes plan it with 16 rows per wave (and with the
        // default rows, for sets too small for that)
        for (int rows : {16, 0}) {
            Plan pr;
            CHECK(plan_rikfad(ts.data(), count, pr, err, rows) == RIKFAD_OK,
                  "plan (read passes, %d rows): %s", rows, err.c_str());
            check_plan(pr, count);
        }
    }
    std::printf("plan_check: %d plans checked, %d rejected as expected, %d failures\n", planned,
                rejected, failures);
    return failures == 0 ? 0 : 1;
}
