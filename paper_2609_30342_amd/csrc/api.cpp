// api.cpp -- the extern "C" entry points declared in include/rikfad.h.
//
// Host side of the library: argument validation (before any HIP call),
// device tables, workspace, the deferred half-kick state machine, event
// timing.  All launches go to the caller's stream; nothing here blocks
// except the calls documented as blocking.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/rikfad.h"
#include "adafactor.hpp"
#include "kernels.hpp"
#include "plan.hpp"

namespace {

thread_local std::string g_last_error;

rikfad_status fail(rikfad_status s, const std::string &msg)
{
    g_last_error = msg;
    return s;
}

rikfad_status hip_fail(hipError_t e, const char *what)
{
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return RIKFAD_EHIP;
}

#define HIP_TRY(expr, what)                                   \
    do {                                                      \
        hipError_t e_ = (expr);                               \
        if (e_ != hipSuccess) return hip_fail(e_, what);      \
    } while (0)

// Device copies of the plan tables plus the partial-sum workspace.
struct DeviceTables {
    rk::TensorDesc *tensors = nullptr;
    const void **grads = nullptr;
    rk::Tile *tiles = nullptr;
    rk::FinItem *fin = nullptr;
    float *ws = nullptr;
    int *flag = nullptr;
};

template <typename T>
rikfad_status upload(T **dst, const std::vector<T> &src, const char *what)
{
    if (src.empty()) return RIKFAD_OK;
    const size_t bytes = sizeof(T) * src.size();
    HIP_TRY(hipMalloc(reinterpret_cast<void **>(dst), bytes), what);
    HIP_TRY(hipMemcpy(*dst, src.data(), bytes, hipMemcpyHostToDevice), what);
    return RIKFAD_OK;
}

void free_tables(DeviceTables &d)
{
    if (d.tensors) (void)hipFree(d.tensors);
    if (d.grads) (void)hipFree(const_cast<void **>(d.grads));
    if (d.tiles) (void)hipFree(d.tiles);
    if (d.fin) (void)hipFree(d.fin);
    if (d.ws) (void)hipFree(d.ws);
    if (d.flag) (void)hipFree(d.flag);
    d = DeviceTables{};
}

rikfad_status make_tables(const rk::Plan &pl, DeviceTables &d)
{
    rikfad_status s;
    if ((s = upload(&d.tensors, pl.tensors, "hipMalloc/copy tensor table")) != RIKFAD_OK) return s;
    if ((s = upload(&d.grads, pl.grads, "hipMalloc/copy gradient table")) != RIKFAD_OK) return s;
    if ((s = upload(&d.tiles, pl.tiles, "hipMalloc/copy tile table")) != RIKFAD_OK) return s;
    if ((s = upload(&d.fin, pl.fin, "hipMalloc/copy finalisation table")) != RIKFAD_OK) return s;
    const size_t wsb = sizeof(float) * static_cast<size_t>(pl.ws_floats > 0 ? pl.ws_floats : 1);
    HIP_TRY(hipMalloc(reinterpret_cast<void **>(&d.ws), wsb), "hipMalloc workspace");
    HIP_TRY(hipMemset(d.ws, 0, wsb), "hipMemset workspace");
    HIP_TRY(hipMalloc(reinterpret_cast<void **>(&d.flag), sizeof(int)), "hipMalloc flag");
    HIP_TRY(hipMemset(d.flag, 0, sizeof(int)), "hipMemset flag");
    return RIKFAD_OK;
}

// Gradient-pointer updates go through a small ring of pinned host slots so
// that the asynchronous copy never reads a buffer the host has reused.
struct GradRing {
    static constexpr int kSlots = 4;
    const void **host[kSlots] = {};
    hipEvent_t done[kSlots] = {};
    bool used[kSlots] = {};
    int next = 0;
    size_t count = 0;

    rikfad_status init(size_t n)
    {
        count = n;
        for (int i = 0; i < kSlots; ++i) {
            HIP_TRY(hipHostMalloc(reinterpret_cast<void **>(&host[i]),
                                  sizeof(void *) * (n ? n : 1), hipHostMallocDefault),
                    "hipHostMalloc gradient slots");
            HIP_TRY(hipEventCreateWithFlags(&done[i], hipEventDisableTiming), "hipEventCreate");
        }
        return RIKFAD_OK;
    }
    void release()
    {
        for (int i = 0; i < kSlots; ++i) {
            if (host[i]) (void)hipHostFree(host[i]);
            if (done[i]) (void)hipEventDestroy(done[i]);
            host[i] = nullptr;
            done[i] = nullptr;
        }
    }
    rikfad_status push(const void **dev, const void *const *src, hipStream_t stream)
    {
        const int s = next;
        next = (next + 1) % kSlots;
        if (used[s]) HIP_TRY(hipEventSynchronize(done[s]), "hipEventSynchronize gradient slot");
        std::memcpy(host[s], src, sizeof(void *) * count);
        HIP_TRY(hipMemcpyAsync(dev, host[s], sizeof(void *) * count, hipMemcpyHostToDevice, stream),
                "hipMemcpyAsync gradient table");
        HIP_TRY(hipEventRecord(done[s], stream), "hipEventRecord gradient slot");
        used[s] = true;
        return RIKFAD_OK;
    }
};

// Per-step kernel timing (benchmarks only).  Each timed phase of a step has
// a start and a stop event attached to its first and last kernel dispatch
// (launch.hpp): they carry the kernels' own begin and end times and put no
// packet of their own into the stream, so a timed step runs like an
// untimed one.
struct Timing {
    explicit Timing(int phases) : nph(phases) {}
    int nph;
    bool on = false;
    std::vector<hipEvent_t> ev;     // 2 per phase and step
    std::vector<uint8_t> ran;       // per phase and step: events attached
    int64_t steps = 0;

    // Events of phase ph of the step being enqueued (nullptr when off).
    rikfad_status phase(int ph, hipEvent_t *start, hipEvent_t *stop)
    {
        *start = *stop = nullptr;
        if (!on) return RIKFAD_OK;
        const size_t slot = static_cast<size_t>(steps * nph + ph);
        while (ev.size() < 2 * (slot + 1)) {
            hipEvent_t e;
            HIP_TRY(hipEventCreate(&e), "hipEventCreate timing");
            ev.push_back(e);
        }
        if (ran.size() < static_cast<size_t>((steps + 1) * nph))
            ran.resize(static_cast<size_t>((steps + 1) * nph), 0);
        ran[slot] = 1;
        *start = ev[2 * slot];
        *stop = ev[2 * slot + 1];
        return RIKFAD_OK;
    }
    void end_step()
    {
        if (on) steps += 1;
    }
    void release()
    {
        for (hipEvent_t e : ev) (void)hipEventDestroy(e);
        ev.clear();
        ran.clear();
        steps = 0;
    }
};

}  // namespace

struct rikfad_ctx {
    rk::Plan plan;
    DeviceTables dev;
    GradRing ring;
    Timing timing{3};          // streaming, finalisation, apply
    rikfad_hparams hp{};
    rk::Coeffs k{};
    bool two_pass = false;
    bool pending = false;       // a deferred C.4 + D is owed to the matrices' p
    bool sums_valid = false;    // partial sums of R reflect the current R
    std::vector<const void *> grads_host;
};

constexpr int kUpdateRowsPerWave = 3;   // Adafactor-m update pass (see adafm_ctx)
#ifndef RK_ADA_READ_ROWS
#define RK_ADA_READ_ROWS 16
#endif
// Adafactor-m read passes (statistics, RMS) and their finalisation: rows per
// wave of their tile table.  They only read g, so a taller tile moves more
// bytes per workgroup for the same fixed costs (descriptors, factors, the
// partial sums) and leaves fewer partial sums to finalise: with 16 rows the
// two passes read GPT2-S's gradient at 6.0-6.3 TB/s (fp32) against 5.1-5.7
// with the streaming table's 4.  A set with fewer than kReadMinTiles tiles
// at that height keeps the streaming table's rows, so that it still fills
// the chip.
constexpr int kReadRowsPerWave = RK_ADA_READ_ROWS;
constexpr int64_t kReadMinTiles = 512;

struct adafm_ctx {
    rk::Plan plan;
    DeviceTables dev;
    GradRing ring;
    Timing timing{5};          // statistics, finalisation, RMS pass, scale, update
    adafm_hparams hp{};
    int64_t steps = 0;                      // steps taken
    std::vector<rk::TensorRange> ranges;    // tiles of each tensor
    rk::TensorRange *ranges_dev = nullptr;
    float *tilepart = nullptr;              // 2 per tile: sums of U^2 and X^2
    float *scales = nullptr;                // 1 per tensor
    std::vector<const void *> grads_host;
    int64_t min_bytes = 0, update_bytes = 0;
    // The update pass has no reductions, so it runs over a tile table of its
    // own with fewer rows per wave (3 against 4: 1.5-3% faster on GPT2-S);
    // tensor descriptors, gradients and workspace are the plan's.
    std::vector<rk::TileGroup> upd_groups;
    rk::Tile *upd_tiles = nullptr;
};

struct ikfad_ctx {
    rk::Plan plan;
    DeviceTables dev;
    Timing timing{1};
    rikfad_hparams hp{};
    rk::Coeffs k{};
};

namespace rk {
void set_last_error(const char *msg) { g_last_error = msg; }
}  // namespace rk

extern "C" {

const char *rikfad_status_string(rikfad_status s)
{
    switch (s) {
    case RIKFAD_OK: return "ok";
    case RIKFAD_EINVAL: return "invalid argument";
    case RIKFAD_EALIGN: return "misaligned pointer";
    case RIKFAD_EDTYPE: return "unsupported dtype";
    case RIKFAD_ENOMEM: return "out of memory";
    case RIKFAD_EHIP: return "HIP runtime error";
    case RIKFAD_ESTATE: return "invalid state";
    }
    return "unknown status";
}

const char *rikfad_last_error(void) { return g_last_error.c_str(); }

rikfad_status rikfad_state_bytes(const rikfad_tensor *tensors, int64_t count,
                                 int64_t *rikfad_bytes, int64_t *ikfad_bytes)
{
    if (!rikfad_bytes || !ikfad_bytes) return fail(RIKFAD_EINVAL, "output pointer is NULL");
    rk::Plan pl;
    std::string err;
    rikfad_status s = rk::plan_rikfad(tensors, count, pl, err);
    if (s != RIKFAD_OK) return fail(s, err);
    *rikfad_bytes = pl.state_bytes;
    *ikfad_bytes = pl.ikfad_state_bytes;
    return RIKFAD_OK;
}

rikfad_status rikfad_create(const rikfad_tensor *tensors, int64_t count,
                            const rikfad_hparams *hp, uint32_t flags, rikfad_ctx **out)
{
    if (!out) return fail(RIKFAD_EINVAL, "out is NULL");
    *out = nullptr;
    std::string err;
    if (flags & ~RIKFAD_FLAG_TWO_PASS) return fail(RIKFAD_EINVAL, "unknown flag bits");
    rikfad_status s = rk::check_hparams(hp, err);
    if (s != RIKFAD_OK) return fail(s, err);
    rikfad_ctx *ctx = new (std::nothrow) rikfad_ctx();
    if (!ctx) return fail(RIKFAD_ENOMEM, "host allocation failed");
    s = rk::plan_rikfad(tensors, count, ctx->plan, err);
    if (s != RIKFAD_OK) {
        delete ctx;
        return fail(s, err);
    }
    ctx->hp = *hp;
    ctx->k = rk::make_coeffs(*hp);
    ctx->two_pass = (flags & RIKFAD_FLAG_TWO_PASS) != 0;
    ctx->grads_host = ctx->plan.grads;
    if ((s = make_tables(ctx->plan, ctx->dev)) != RIKFAD_OK ||
        (s = ctx->ring.init(ctx->plan.grads.size())) != RIKFAD_OK) {
        std::string keep = g_last_error;
        free_tables(ctx->dev);
        ctx->ring.release();
        delete ctx;
        g_last_error = keep;
        return s;
    }
    *out = ctx;
    return RIKFAD_OK;
}

static rikfad_status apply_pending(rikfad_ctx *ctx, hipStream_t stream,
                                   hipEvent_t start = nullptr, hipEvent_t stop = nullptr)
{
    if (!ctx->pending) return RIKFAD_OK;
    hipError_t e = rk::launch_apply(ctx->dev.tensors, ctx->dev.tiles, ctx->plan.groups.data(),
                                    static_cast<int>(ctx->plan.groups.size()), ctx->dev.ws,
                                    ctx->k, stream, start, stop);
    if (e != hipSuccess) return hip_fail(e, "launch apply kernel");
    ctx->pending = false;
    return RIKFAD_OK;
}

rikfad_status rikfad_step(rikfad_ctx *ctx, void *stream_)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    hipStream_t stream = static_cast<hipStream_t>(stream_);
    const rk::Plan &pl = ctx->plan;
    if (pl.tiles.empty()) return RIKFAD_OK;
    hipError_t e;
    if (!ctx->sums_valid && pl.row_items > 0) {
        e = rk::launch_finalize(ctx->dev.fin, pl.row_items, pl.fin_log2,
                                ctx->dev.ws, ctx->k, ctx->dev.flag, 1, stream);
        if (e != hipSuccess) return hip_fail(e, "launch finalize kernel (init)");
    }
    ctx->sums_valid = true;
    Timing &tm = ctx->timing;
    hipEvent_t t0, t1;
    rikfad_status s;
    if ((s = tm.phase(0, &t0, &t1)) != RIKFAD_OK) return s;
    e = rk::launch_stream(ctx->dev.tensors, ctx->dev.grads, ctx->dev.tiles, pl.groups.data(),
                          static_cast<int>(pl.groups.size()), ctx->dev.ws, ctx->k,
                          ctx->pending ? 1 : 0, ctx->dev.flag, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch stream kernel");
    ctx->pending = false;
    const int64_t nfin = static_cast<int64_t>(pl.fin.size());
    t0 = t1 = nullptr;
    if (nfin > 0 && (s = tm.phase(1, &t0, &t1)) != RIKFAD_OK) return s;
    e = rk::launch_finalize(ctx->dev.fin, nfin, pl.fin_log2, ctx->dev.ws,
                            ctx->k, ctx->dev.flag, 0, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch finalize kernel");
    ctx->pending = pl.matrix_tiles > 0;
    if (ctx->two_pass && ctx->pending) {
        if ((s = tm.phase(2, &t0, &t1)) != RIKFAD_OK) return s;
        if ((s = apply_pending(ctx, stream, t0, t1)) != RIKFAD_OK) return s;
    }
    tm.end_step();
    return RIKFAD_OK;
}

rikfad_status rikfad_step_grads(rikfad_ctx *ctx, const void *const *grads, void *stream)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    const size_t n = ctx->plan.tensors.size();
    if (n > 0 && !grads) return fail(RIKFAD_EINVAL, "grads is NULL");
    bool changed = false;
    for (size_t i = 0; i < n; ++i) {
        const rk::TensorDesc &d = ctx->plan.tensors[i];
        if (!rk::grad_fits(grads[i], d.dtype, d.vec))
            return fail(grads[i] ? RIKFAD_EALIGN : RIKFAD_EINVAL,
                        "gradient " + std::to_string(i) +
                            " is NULL or breaks the alignment planned at create");
        changed = changed || grads[i] != ctx->grads_host[i];
    }
    if (changed) {
        rikfad_status s = ctx->ring.push(ctx->dev.grads, grads, static_cast<hipStream_t>(stream));
        if (s != RIKFAD_OK) return s;
        for (size_t i = 0; i < n; ++i) ctx->grads_host[i] = grads[i];
    }
    return rikfad_step(ctx, stream);
}

rikfad_status rikfad_set_hparams(rikfad_ctx *ctx, const rikfad_hparams *hp, void *stream)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    std::string err;
    rikfad_status s = rk::check_hparams(hp, err);
    if (s != RIKFAD_OK) return fail(s, err);
    const bool kick_changes = hp->h != ctx->hp.h || hp->gamma != ctx->hp.gamma ||
                              hp->eps_stab != ctx->hp.eps_stab;
    if (ctx->pending && kick_changes &&
        (s = apply_pending(ctx, static_cast<hipStream_t>(stream))) != RIKFAD_OK)
        return s;
    ctx->hp = *hp;
    ctx->k = rk::make_coeffs(*hp);
    return RIKFAD_OK;
}

rikfad_status rikfad_sync_momentum(rikfad_ctx *ctx, void *stream)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    return apply_pending(ctx, static_cast<hipStream_t>(stream));
}

rikfad_status rikfad_state_changed(rikfad_ctx *ctx)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    ctx->pending = false;
    ctx->sums_valid = false;
    return RIKFAD_OK;
}

rikfad_status rikfad_query(const rikfad_ctx *ctx, rikfad_info *out)
{
    if (!ctx || !out) return fail(RIKFAD_EINVAL, "ctx or out is NULL");
    const rk::Plan &pl = ctx->plan;
    rikfad_info info{};
    info.tensors = static_cast<int64_t>(pl.tensors.size());
    info.matrices = pl.matrices;
    info.vectors = pl.vectors;
    info.elements = pl.elements;
    info.state_bytes = pl.state_bytes;
    info.ikfad_state_bytes = pl.ikfad_state_bytes;
    info.workspace_bytes = static_cast<int64_t>(
        4 * pl.ws_floats + sizeof(int) + sizeof(rk::TensorDesc) * pl.tensors.size() +
        sizeof(void *) * pl.grads.size() + sizeof(rk::Tile) * pl.tiles.size() +
        sizeof(rk::FinItem) * pl.fin.size());
    info.min_bytes_per_step = pl.min_bytes;
    info.stream_min_bytes = pl.stream_min_bytes;
    info.stream_tiles = static_cast<int64_t>(pl.tiles.size());
    info.finalize_items = static_cast<int64_t>(pl.fin.size());
    info.pending = ctx->pending ? 1 : 0;
    info.two_pass = ctx->two_pass ? 1 : 0;
    *out = info;
    return RIKFAD_OK;
}

rikfad_status rikfad_nonfinite(rikfad_ctx *ctx, void *stream, int32_t *out)
{
    if (!ctx || !out) return fail(RIKFAD_EINVAL, "ctx or out is NULL");
    HIP_TRY(hipStreamSynchronize(static_cast<hipStream_t>(stream)), "hipStreamSynchronize");
    int v = 0;
    HIP_TRY(hipMemcpy(&v, ctx->dev.flag, sizeof(int), hipMemcpyDeviceToHost), "hipMemcpy flag");
    *out = v ? 1 : 0;
    return RIKFAD_OK;
}

// Sums over the timed steps of each phase's kernel time into ms[0..nph-1]
// and clears the record.
static rikfad_status read_timing(Timing &tm, double *ms, int64_t *steps)
{
    for (int k = 0; k < tm.nph; ++k) ms[k] = 0.0;
    const size_t slots = static_cast<size_t>(tm.steps * tm.nph);
    for (size_t q = slots; q-- > 0;) {          // wait for the last attached stop event
        if (q < tm.ran.size() && tm.ran[q]) {
            HIP_TRY(hipEventSynchronize(tm.ev[2 * q + 1]), "hipEventSynchronize timing");
            break;
        }
    }
    for (size_t q = 0; q < slots && q < tm.ran.size(); ++q) {
        if (!tm.ran[q]) continue;
        float t = 0.f;
        HIP_TRY(hipEventElapsedTime(&t, tm.ev[2 * q], tm.ev[2 * q + 1]), "hipEventElapsedTime");
        ms[q % static_cast<size_t>(tm.nph)] += t;
    }
    *steps = tm.steps;
    tm.steps = 0;
    std::fill(tm.ran.begin(), tm.ran.end(), 0);
    return RIKFAD_OK;
}

rikfad_status rikfad_timing_enable(rikfad_ctx *ctx, int32_t enable)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    ctx->timing.on = enable != 0;
    return RIKFAD_OK;
}

rikfad_status rikfad_timing_read(rikfad_ctx *ctx, double *stream_ms, double *finalize_ms,
                                 double *apply_ms, int64_t *steps)
{
    if (!ctx || !stream_ms || !finalize_ms || !apply_ms || !steps)
        return fail(RIKFAD_EINVAL, "NULL argument");
    double ms[3];
    rikfad_status s = read_timing(ctx->timing, ms, steps);
    if (s != RIKFAD_OK) return s;
    *stream_ms = ms[0];
    *finalize_ms = ms[1];
    *apply_ms = ms[2];
    return RIKFAD_OK;
}

void rikfad_destroy(rikfad_ctx *ctx)
{
    if (!ctx) return;
    free_tables(ctx->dev);
    ctx->ring.release();
    ctx->timing.release();
    delete ctx;
}

// ------------------------------------------------------------ full iKFAD

rikfad_status ikfad_create(const ikfad_tensor *tensors, int64_t count, const rikfad_hparams *hp,
                           ikfad_ctx **out)
{
    if (!out) return fail(RIKFAD_EINVAL, "out is NULL");
    *out = nullptr;
    std::string err;
    rikfad_status s = rk::check_hparams(hp, err);
    if (s != RIKFAD_OK) return fail(s, err);
    ikfad_ctx *ctx = new (std::nothrow) ikfad_ctx();
    if (!ctx) return fail(RIKFAD_ENOMEM, "host allocation failed");
    if ((s = rk::plan_ikfad(tensors, count, ctx->plan, err)) != RIKFAD_OK) {
        delete ctx;
        return fail(s, err);
    }
    ctx->hp = *hp;
    ctx->k = rk::make_coeffs(*hp);
    if ((s = make_tables(ctx->plan, ctx->dev)) != RIKFAD_OK) {
        std::string keep = g_last_error;
        free_tables(ctx->dev);
        delete ctx;
        g_last_error = keep;
        return s;
    }
    *out = ctx;
    return RIKFAD_OK;
}

rikfad_status ikfad_step(ikfad_ctx *ctx, void *stream_)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    hipStream_t stream = static_cast<hipStream_t>(stream_);
    if (ctx->plan.tiles.empty()) return RIKFAD_OK;
    Timing &tm = ctx->timing;
    hipEvent_t t0, t1;
    rikfad_status s;
    if ((s = tm.phase(0, &t0, &t1)) != RIKFAD_OK) return s;
    hipError_t e = rk::launch_ikfad(ctx->dev.tensors, ctx->dev.grads, ctx->dev.tiles,
                                    static_cast<int64_t>(ctx->plan.tiles.size()), ctx->k,
                                    ctx->dev.flag, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch ikfad kernel");
    tm.end_step();
    return RIKFAD_OK;
}

rikfad_status ikfad_set_hparams(ikfad_ctx *ctx, const rikfad_hparams *hp)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    std::string err;
    rikfad_status s = rk::check_hparams(hp, err);
    if (s != RIKFAD_OK) return fail(s, err);
    ctx->hp = *hp;
    ctx->k = rk::make_coeffs(*hp);
    return RIKFAD_OK;
}

rikfad_status ikfad_timing_enable(ikfad_ctx *ctx, int32_t enable)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    ctx->timing.on = enable != 0;
    return RIKFAD_OK;
}

rikfad_status ikfad_timing_read(ikfad_ctx *ctx, double *ms, int64_t *steps)
{
    if (!ctx || !ms || !steps) return fail(RIKFAD_EINVAL, "NULL argument");
    double t[1];
    rikfad_status s = read_timing(ctx->timing, t, steps);
    if (s != RIKFAD_OK) return s;
    *ms = t[0];
    return RIKFAD_OK;
}

rikfad_status ikfad_nonfinite(ikfad_ctx *ctx, void *stream, int32_t *out)
{
    if (!ctx || !out) return fail(RIKFAD_EINVAL, "ctx or out is NULL");
    HIP_TRY(hipStreamSynchronize(static_cast<hipStream_t>(stream)), "hipStreamSynchronize");
    int v = 0;
    HIP_TRY(hipMemcpy(&v, ctx->dev.flag, sizeof(int), hipMemcpyDeviceToHost), "hipMemcpy flag");
    *out = v ? 1 : 0;
    return RIKFAD_OK;
}

void ikfad_destroy(ikfad_ctx *ctx)
{
    if (!ctx) return;
    free_tables(ctx->dev);
    ctx->timing.release();
    delete ctx;
}

// ------------------------------------------------------------ Adafactor-m

static rikfad_status check_adafm_hparams(const adafm_hparams *hp)
{
    if (!hp) return fail(RIKFAD_EINVAL, "hparams is NULL");
    if (hp->reserved != 0) return fail(RIKFAD_EINVAL, "reserved field must be 0");
    if (!(std::isfinite(hp->h) && std::isfinite(hp->beta1) && std::isfinite(hp->decay_rate) &&
          std::isfinite(hp->eps1) && std::isfinite(hp->eps2) &&
          std::isfinite(hp->clip_threshold)))
        return fail(RIKFAD_EINVAL, "hyperparameters must be finite");
    if (!(hp->h > 0) || !(hp->beta1 >= 0 && hp->beta1 < 1) || !(hp->decay_rate <= 0) ||
        !(hp->eps1 >= 0) || !(hp->eps2 >= 0) ||
        (hp->scale_parameter != 0 && hp->scale_parameter != 1))
        return fail(RIKFAD_EINVAL,
                    "need h > 0, 0 <= beta1 < 1, decay_rate <= 0, eps1 >= 0, eps2 >= 0, "
                    "scale_parameter 0 or 1");
    const float fh = static_cast<float>(hp->h), fc = static_cast<float>(hp->clip_threshold);
    const float fe1 = static_cast<float>(hp->eps1), fe2 = static_cast<float>(hp->eps2);
    if (!(std::isfinite(fh) && fh > 0 && std::isfinite(fc) && std::isfinite(fe1) &&
          std::isfinite(fe2)))
        return fail(RIKFAD_EINVAL, "hyperparameters outside the fp32 range");
    return RIKFAD_OK;
}

// Coefficients of step t (>= 1): b = 1 - t^decay_rate with 1 - b taken as
// t^decay_rate itself, in fp64, each rounded once to fp32.
static rk::AdaCoeffs adafm_coeffs(const adafm_hparams &hp, int64_t t)
{
    const double p = std::pow(static_cast<double>(t), hp.decay_rate);
    rk::AdaCoeffs k{};
    k.b = static_cast<float>(1.0 - p);
    k.omb = static_cast<float>(p);
    k.eps1 = static_cast<float>(hp.eps1);
    k.beta1 = static_cast<float>(hp.beta1);
    k.omb1 = static_cast<float>(1.0 - hp.beta1);
    k.h = static_cast<float>(hp.h);
    k.eps2 = static_cast<float>(hp.eps2);
    k.clip = static_cast<float>(hp.clip_threshold);
    k.scale = hp.scale_parameter;
    return k;
}

static void adafm_free(adafm_ctx *ctx)
{
    free_tables(ctx->dev);
    ctx->ring.release();
    ctx->timing.release();
    if (ctx->ranges_dev) (void)hipFree(ctx->ranges_dev);
    if (ctx->tilepart) (void)hipFree(ctx->tilepart);
    if (ctx->scales) (void)hipFree(ctx->scales);
    if (ctx->upd_tiles) (void)hipFree(ctx->upd_tiles);
    ctx->ranges_dev = nullptr;
    ctx->tilepart = nullptr;
    ctx->scales = nullptr;
    ctx->upd_tiles = nullptr;
}

// Tile range of every tensor (the planner emits each tensor's tiles
// contiguously) and the byte counts of the step.
static rikfad_status adafm_layout(adafm_ctx *ctx)
{
    const rk::Plan &pl = ctx->plan;
    const size_t nt = pl.tensors.size();
    ctx->ranges.assign(nt, rk::TensorRange{-1, 0, 0});
    for (size_t q = 0; q < pl.tiles.size(); ++q) {
        rk::TensorRange &r = ctx->ranges[static_cast<size_t>(pl.tiles[q].tensor)];
        if (r.tile0 < 0) r.tile0 = static_cast<int64_t>(q);
        if (r.tile0 + r.ntile != static_cast<int64_t>(q))
            return fail(RIKFAD_EINVAL, "internal: tiles of a tensor are not contiguous");
        r.ntile += 1;
    }
    const int64_t sc = ctx->hp.scale_parameter ? 1 : 0, cl = ctx->hp.clip_threshold > 0 ? 1 : 0;
    ctx->min_bytes = ctx->update_bytes = 0;
    for (size_t i = 0; i < nt; ++i) {
        const rk::TensorDesc &d = pl.tensors[i];
        const int64_t mn = d.m * d.n, eb = d.dtype == rk::DT_BF16 ? 2 : 4;
        ctx->ranges[i].elems = mn;
        if (ctx->ranges[i].tile0 < 0) ctx->ranges[i].tile0 = 0;
        if (d.kind == rk::KIND_VECTOR) {
            // pass 1: g, v in, v out (+x); pass 3: g, x, M, v in, x, M out
            ctx->min_bytes += mn * ((1 + sc) * eb + 8 + 3 * eb + 12);
            ctx->update_bytes += mn * (3 * eb + 12);
        } else {
            // pass 1: g (+x); pass 2: g (with clipping); pass 3: g, x, M in, x, M out; R, C
            ctx->min_bytes += mn * ((1 + sc + cl) * eb + 3 * eb + 8) + 8 * (d.m + d.n);
            ctx->update_bytes += mn * (3 * eb + 8) + 4 * (d.m + d.n);
        }
    }
    return RIKFAD_OK;
}

rikfad_status adafm_create(const rikfad_tensor *tensors, int64_t count, const adafm_hparams *hp,
                           adafm_ctx **out)
{
    if (!out) return fail(RIKFAD_EINVAL, "out is NULL");
    *out = nullptr;
    rikfad_status s = check_adafm_hparams(hp);
    if (s != RIKFAD_OK) return s;
    adafm_ctx *ctx = new (std::nothrow) adafm_ctx();
    if (!ctx) return fail(RIKFAD_ENOMEM, "host allocation failed");
    std::string err;
    if ((s = rk::plan_rikfad(tensors, count, ctx->plan, err, kReadRowsPerWave)) != RIKFAD_OK) {
        delete ctx;
        return fail(s, err);
    }
    if (ctx->plan.matrix_tiles < kReadMinTiles &&
        (s = rk::plan_rikfad(tensors, count, ctx->plan, err, 0)) != RIKFAD_OK) {
        delete ctx;
        return fail(s, err);
    }
    ctx->hp = *hp;
    ctx->grads_host = ctx->plan.grads;
    const size_t ntile = ctx->plan.tiles.size(), nt = ctx->plan.tensors.size();
    rk::Plan upd;
    if ((s = rk::plan_rikfad(tensors, count, upd, err, kUpdateRowsPerWave)) != RIKFAD_OK) {
        delete ctx;
        return fail(s, err);
    }
    ctx->upd_groups = upd.groups;
    if ((s = adafm_layout(ctx)) != RIKFAD_OK ||
        (s = upload(&ctx->upd_tiles, upd.tiles, "hipMalloc/copy update tile table")) != RIKFAD_OK ||
        (s = make_tables(ctx->plan, ctx->dev)) != RIKFAD_OK ||
        (s = ctx->ring.init(nt)) != RIKFAD_OK ||
        (s = upload(&ctx->ranges_dev, ctx->ranges, "hipMalloc/copy tensor ranges")) != RIKFAD_OK) {
        std::string keep = g_last_error;
        adafm_free(ctx);
        delete ctx;
        g_last_error = keep;
        return s;
    }
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&ctx->tilepart),
                             sizeof(float) * 2 * (ntile ? ntile : 1));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&ctx->scales), sizeof(float) * (nt ? nt : 1));
    if (e != hipSuccess) {
        adafm_free(ctx);
        delete ctx;
        return hip_fail(e, "hipMalloc Adafactor-m workspace");
    }
    *out = ctx;
    return RIKFAD_OK;
}

rikfad_status adafm_step(adafm_ctx *ctx, void *stream_)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    hipStream_t stream = static_cast<hipStream_t>(stream_);
    const rk::Plan &pl = ctx->plan;
    const int64_t t = ctx->steps + 1;
    if (pl.tiles.empty()) {
        ctx->steps = t;
        return RIKFAD_OK;
    }
    const rk::AdaCoeffs k = adafm_coeffs(ctx->hp, t);
    rk::Coeffs fk{};            // the factor update R <- b R + (1-b) rowsum
    fk.a = k.b;
    fk.kappa = k.omb;
    const int ng = static_cast<int>(pl.groups.size());
    Timing &tm = ctx->timing;
    hipEvent_t t0, t1;
    rikfad_status s;
    if ((s = tm.phase(0, &t0, &t1)) != RIKFAD_OK) return s;
    hipError_t e = rk::launch_adafm_stats(ctx->dev.tensors, ctx->dev.grads, ctx->dev.tiles,
                                          pl.groups.data(), ng, ctx->dev.ws, ctx->tilepart, k,
                                          ctx->hp.scale_parameter != 0, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch adafm stats kernel");
    const int64_t nfin = static_cast<int64_t>(pl.fin.size());
    if (nfin > 0) {
        if ((s = tm.phase(1, &t0, &t1)) != RIKFAD_OK) return s;
        e = rk::launch_finalize(ctx->dev.fin, nfin, pl.fin_log2, ctx->dev.ws,
                                fk, ctx->dev.flag, 0, stream, t0, t1);
        if (e != hipSuccess) return hip_fail(e, "launch finalize kernel");
    }
    // RMS pass (when clipping and there are matrices), then the scale kernel.
    if (ctx->hp.clip_threshold > 0 && pl.matrix_tiles > 0) {
        if ((s = tm.phase(2, &t0, &t1)) != RIKFAD_OK) return s;
        e = rk::launch_adafm_rms(ctx->dev.tensors, ctx->dev.grads, ctx->dev.tiles,
                                 pl.groups.data(), ng, ctx->dev.ws, ctx->tilepart, stream, t0,
                                 t1);
        if (e != hipSuccess) return hip_fail(e, "launch adafm rms kernel");
    }
    if ((s = tm.phase(3, &t0, &t1)) != RIKFAD_OK) return s;
    e = rk::launch_adafm_scale(ctx->ranges_dev, static_cast<int64_t>(pl.tensors.size()),
                               ctx->tilepart, ctx->scales, k, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch adafm scale kernel");
    if ((s = tm.phase(4, &t0, &t1)) != RIKFAD_OK) return s;
    e = rk::launch_adafm_update(ctx->dev.tensors, ctx->dev.grads, ctx->upd_tiles,
                                ctx->upd_groups.data(), static_cast<int>(ctx->upd_groups.size()),
                                ctx->dev.ws, ctx->scales, k, stream, t0, t1);
    if (e != hipSuccess) return hip_fail(e, "launch adafm update kernel");
    tm.end_step();
    ctx->steps = t;
    return RIKFAD_OK;
}

rikfad_status adafm_step_grads(adafm_ctx *ctx, const void *const *grads, void *stream)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    const size_t n = ctx->plan.tensors.size();
    if (n > 0 && !grads) return fail(RIKFAD_EINVAL, "grads is NULL");
    bool changed = false;
    for (size_t i = 0; i < n; ++i) {
        const rk::TensorDesc &d = ctx->plan.tensors[i];
        if (!rk::grad_fits(grads[i], d.dtype, d.vec))
            return fail(grads[i] ? RIKFAD_EALIGN : RIKFAD_EINVAL,
                        "gradient " + std::to_string(i) +
                            " is NULL or breaks the alignment planned at create");
        changed = changed || grads[i] != ctx->grads_host[i];
    }
    if (changed) {
        rikfad_status s = ctx->ring.push(ctx->dev.grads, grads, static_cast<hipStream_t>(stream));
        if (s != RIKFAD_OK) return s;
        for (size_t i = 0; i < n; ++i) ctx->grads_host[i] = grads[i];
    }
    return adafm_step(ctx, stream);
}

rikfad_status adafm_set_hparams(adafm_ctx *ctx, const adafm_hparams *hp)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    rikfad_status s = check_adafm_hparams(hp);
    if (s != RIKFAD_OK) return s;
    ctx->hp = *hp;
    return adafm_layout(ctx);
}

rikfad_status adafm_set_step(adafm_ctx *ctx, int64_t steps_taken)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    if (steps_taken < 0) return fail(RIKFAD_EINVAL, "steps_taken must be >= 0");
    ctx->steps = steps_taken;
    return RIKFAD_OK;
}

rikfad_status adafm_get_step(const adafm_ctx *ctx, int64_t *steps_taken)
{
    if (!ctx || !steps_taken) return fail(RIKFAD_EINVAL, "ctx or out is NULL");
    *steps_taken = ctx->steps;
    return RIKFAD_OK;
}

rikfad_status adafm_min_bytes(const adafm_ctx *ctx, int64_t *min_bytes_per_step,
                              int64_t *update_min_bytes, int64_t *state_bytes)
{
    if (!ctx || !min_bytes_per_step || !update_min_bytes || !state_bytes)
        return fail(RIKFAD_EINVAL, "NULL argument");
    *min_bytes_per_step = ctx->min_bytes;
    *update_min_bytes = ctx->update_bytes;
    *state_bytes = ctx->plan.state_bytes;
    return RIKFAD_OK;
}

rikfad_status adafm_nonfinite(adafm_ctx *ctx, void *stream, int32_t *out)
{
    if (!ctx || !out) return fail(RIKFAD_EINVAL, "ctx or out is NULL");
    HIP_TRY(hipStreamSynchronize(static_cast<hipStream_t>(stream)), "hipStreamSynchronize");
    int v = 0;
    HIP_TRY(hipMemcpy(&v, ctx->dev.flag, sizeof(int), hipMemcpyDeviceToHost), "hipMemcpy flag");
    *out = v ? 1 : 0;
    return RIKFAD_OK;
}

rikfad_status adafm_timing_enable(adafm_ctx *ctx, int32_t enable)
{
    if (!ctx) return fail(RIKFAD_EINVAL, "ctx is NULL");
    ctx->timing.on = enable != 0;
    return RIKFAD_OK;
}

rikfad_status adafm_timing_read(adafm_ctx *ctx, double *ms5, int64_t *steps)
{
    if (!ctx || !ms5 || !steps) return fail(RIKFAD_EINVAL, "NULL argument");
    return read_timing(ctx->timing, ms5, steps);
}

void adafm_destroy(adafm_ctx *ctx)
{
    if (!ctx) return;
    adafm_free(ctx);
    delete ctx;
}

// ------------------------------------------------------------- probes

rikfad_status rikfad_probe_stream(const float *a, const float *b, const float *c, float *d,
                                  float *e, int64_t nfloat, void *stream)
{
    auto al = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) % 16) == 0; };
    if (!a || !b || !c || !d || !e || nfloat < 0 || nfloat % 4 != 0)
        return fail(RIKFAD_EINVAL, "probe_stream: NULL pointer or nfloat not a multiple of 4");
    if (!al(a) || !al(b) || !al(c) || !al(d) || !al(e))
        return fail(RIKFAD_EALIGN, "probe_stream: pointers must be 16-byte aligned");
    hipError_t err = rk::launch_probe_stream(a, b, c, d, e, nfloat, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? RIKFAD_OK : hip_fail(err, "launch probe_stream");
}

rikfad_status rikfad_probe_mix(void *x, const void *g, float *p, int64_t nelem, int32_t dtype,
                               int32_t shape, void *stream)
{
    if (!x || !g || !p || nelem < 0 || nelem % 256 != 0)
        return fail(RIKFAD_EINVAL, "probe_mix: NULL pointer or nelem not a multiple of 256");
    if (dtype != RIKFAD_FP32 && dtype != RIKFAD_BF16)
        return fail(RIKFAD_EDTYPE, "probe_mix: dtype must be RIKFAD_FP32 or RIKFAD_BF16");
    if (shape != 0 && shape != 1) return fail(RIKFAD_EINVAL, "probe_mix: shape must be 0 or 1");
    const uintptr_t xg = dtype == RIKFAD_FP32 ? 16 : 8;
    if (reinterpret_cast<uintptr_t>(x) % xg || reinterpret_cast<uintptr_t>(g) % xg ||
        reinterpret_cast<uintptr_t>(p) % 16)
        return fail(RIKFAD_EALIGN, "probe_mix: x, g 16-byte (fp32) or 8-byte (bf16) and p "
                                   "16-byte aligned");
    hipError_t err = rk::launch_probe_mix(x, g, p, nelem, dtype, shape,
                                          static_cast<hipStream_t>(stream));
    return err == hipSuccess ? RIKFAD_OK : hip_fail(err, "launch probe_mix");
}

rikfad_status rikfad_probe_read(const void *src, int64_t nbytes, float *out, void *stream)
{
    if (!src || !out || nbytes < 0 || nbytes % 16 != 0)
        return fail(RIKFAD_EINVAL, "probe_read: NULL pointer or nbytes not a multiple of 16");
    if (reinterpret_cast<uintptr_t>(src) % 16 || reinterpret_cast<uintptr_t>(out) % 4)
        return fail(RIKFAD_EALIGN, "probe_read: src must be 16-byte and out 4-byte aligned");
    hipError_t err = rk::launch_probe_read(src, nbytes, out, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? RIKFAD_OK : hip_fail(err, "launch probe_read");
}

rikfad_status rikfad_probe_write(void *dst, int64_t nbytes, uint32_t value, void *stream)
{
    if (!dst || nbytes < 0 || nbytes % 16 != 0)
        return fail(RIKFAD_EINVAL, "probe_write: NULL pointer or nbytes not a multiple of 16");
    if (reinterpret_cast<uintptr_t>(dst) % 16)
        return fail(RIKFAD_EALIGN, "probe_write: dst must be 16-byte aligned");
    hipError_t err = rk::launch_probe_write(dst, nbytes, value, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? RIKFAD_OK : hip_fail(err, "launch probe_write");
}

rikfad_status rikfad_probe_copy(const void *src, void *dst, int64_t nbytes, void *stream)
{
    auto al = [](const void *q) { return (reinterpret_cast<uintptr_t>(q) % 16) == 0; };
    if (!src || !dst || nbytes < 0 || nbytes % 16 != 0)
        return fail(RIKFAD_EINVAL, "probe_copy: NULL pointer or nbytes not a multiple of 16");
    if (!al(src) || !al(dst)) return fail(RIKFAD_EALIGN, "probe_copy: pointers must be 16-byte aligned");
    hipError_t err = rk::launch_probe_copy(src, dst, nbytes, static_cast<hipStream_t>(stream));
    return err == hipSuccess ? RIKFAD_OK : hip_fail(err, "launch probe_copy");
}

}  // extern "C"
