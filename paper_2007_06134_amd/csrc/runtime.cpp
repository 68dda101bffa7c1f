// Host runtime and C ABI of the ADPSGD hot path: argument validation, the tile
// table of the segmented variance reduction, kernel launches on the caller's
// stream, the pipelined Algorithm 2 driver, checkpoint state and timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <deque>
#include <limits>
#include <new>
#include <string>
#include <vector>

#include "adpsgd.h"
#include "common.hpp"
#include "kernels.hpp"

namespace adpsgd {

thread_local std::string g_last_error;

int fail(int code, const std::string &msg) {
    g_last_error = msg;
    return code;
}
int ok() {
    g_last_error.clear();
    return ADPSGD_OK;
}

namespace {

constexpr int kRing = 32;          // syncs whose variances may be in flight at once
constexpr int kTimedMax = 1024;    // pending timed launches before a harvest
constexpr int64_t kMaxK = 65536;
constexpr int64_t kMaxCounter = int64_t(1) << 32;  // Philox counter words are 32-bit

enum TimedKind { tStep = 0, tFused = 1, tAverage = 2, tSegsum = 3, tTrace = 4, tKinds = 5 };

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool shape_valid(int32_t K, int64_t P, int32_t T, const int64_t *off, std::string *why) {
    auto bad = [&](const std::string &m) { if (why) *why = m; return false; };
    if (K < 1 || K > kMaxK) return bad("K must be in [1, 65536]");
    if (P < 0) return bad("P must be >= 0");
    if ((P + 3) / 4 > kMaxCounter) return bad("P/4 must be below 2^32");
    if (T < 1 || T > (1 << 24)) return bad("T must be in [1, 2^24]");
    if (!off) return bad("tensor_offsets is NULL");
    if (off[0] != 0) return bad("tensor_offsets[0] must be 0");
    for (int32_t i = 0; i < T; ++i)
        if (off[i + 1] < off[i]) return bad("tensor_offsets must be non-decreasing");
    if (off[T] != P) return bad("tensor_offsets[T] must equal P");
    return true;
}

// Tiles: each tensor [a, b) is cut at multiples of kTileElems, so no tile
// crosses a tensor boundary and a tile spans at most kTileElems / 4 groups.
// Chunks: runs of at most kChunkTiles consecutive tiles of one tensor.
int64_t tiles_of(int64_t a, int64_t b) { return b > a ? (b + kTileElems - 1) / kTileElems - a / kTileElems : 0; }

struct Plan {
    int64_t n_tiles = 0, n_chunks = 0;
};

Plan count_plan(int32_t T, const int64_t *off) {
    Plan pl;
    for (int32_t tau = 0; tau < T; ++tau) {
        const int64_t nt = tiles_of(off[tau], off[tau + 1]);
        pl.n_tiles += nt;
        pl.n_chunks += (nt + kChunkTiles - 1) / kChunkTiles;
    }
    return pl;
}

void build_plan(int32_t T, const int64_t *off, std::vector<Tile> *tiles, std::vector<Chunk> *chunks,
                std::vector<int32_t> *chunk_begin) {
    tiles->clear();
    chunks->clear();
    chunk_begin->assign(T + 1, 0);
    for (int32_t tau = 0; tau < T; ++tau) {
        (*chunk_begin)[tau] = (int32_t)chunks->size();
        const int32_t first_tile = (int32_t)tiles->size();
        for (int64_t s = off[tau]; s < off[tau + 1];) {
            const int64_t e = std::min(off[tau + 1], (s / kTileElems + 1) * kTileElems);
            tiles->push_back(Tile{s, (int32_t)(e - s), tau});
            s = e;
        }
        const int32_t n = (int32_t)tiles->size() - first_tile;
        for (int32_t c = 0; c < n; c += kChunkTiles)
            chunks->push_back(Chunk{first_tile + c, std::min(kChunkTiles, n - c)});
    }
    (*chunk_begin)[T] = (int32_t)chunks->size();
}

struct Layout {
    size_t tiles, chunks, chunk_begin, tile_partials, chunk_partials, var, total;
};

Layout layout_for(const Plan &pl, int32_t T) {
    auto at_least_one = [](int64_t n) { return (size_t)std::max<int64_t>(n, 1); };
    Layout l;
    l.tiles = 0;
    l.chunks = align_up(l.tiles + sizeof(Tile) * at_least_one(pl.n_tiles), 256);
    l.chunk_begin = align_up(l.chunks + sizeof(Chunk) * at_least_one(pl.n_chunks), 256);
    l.tile_partials = align_up(l.chunk_begin + sizeof(int32_t) * (size_t)(T + 1), 256);
    l.chunk_partials = align_up(l.tile_partials + 2 * sizeof(double) * at_least_one(pl.n_tiles), 256);
    l.var = align_up(l.chunk_partials + 2 * sizeof(double) * at_least_one(pl.n_chunks), 256);
    l.total = align_up(l.var + sizeof(double) * (size_t)kRing * 2 * (size_t)T, 256);
    return l;
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int hip_fail(hipError_t e, const char *what) {
    return fail(ADPSGD_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(expr)                                         \
    do {                                                      \
        hipError_t e_ = (expr);                               \
        if (e_ != hipSuccess) return hip_fail(e_, #expr);     \
    } while (0)

struct TimedLaunch {
    int kind;
    hipEvent_t start, stop;
};

}  // namespace
}  // namespace adpsgd

using namespace adpsgd;

struct adpsgd_ctx {
    int32_t K = 0;
    int64_t P = 0;
    int32_t T = 0;
    std::vector<int64_t> offsets;
    std::vector<Tile> tiles;
    std::vector<Chunk> chunks;
    std::vector<int32_t> chunk_begin;
    adpsgd_hparams hp{};
    adpsgd_buffers buf{};
    hipStream_t stream = nullptr;
    int device = 0;
    Tile *d_tiles = nullptr;
    Chunk *d_chunks = nullptr;
    int32_t *d_chunk_begin = nullptr;
    double *d_tile_partials = nullptr;
    double *d_chunk_partials = nullptr;
    double *d_var = nullptr;        // [kRing][2T] device: variances, then gradient norms
    double *h_var = nullptr;        // [kRing][2T] pinned host
    hipEvent_t ring_ev[kRing] = {};
    adpsgd_state st{};
    bool vec = true;                // P % 4 == 0: dwordx4 rows
    bool nontemporal = false;       // stream x and m past the caches (large working sets)
    RoundKeys rk{};
    bool timing = false;
    std::deque<TimedLaunch> timed;
    std::vector<hipEvent_t> ev_pool;
    double t_ms[tKinds] = {};
    int64_t t_n[tKinds] = {};
};

namespace {

void release(adpsgd_ctx *c) {
    if (!c) return;
    for (auto &ev : c->ring_ev)
        if (ev) (void)hipEventDestroy(ev);
    for (auto &tl : c->timed) {
        (void)hipEventDestroy(tl.start);
        (void)hipEventDestroy(tl.stop);
    }
    for (auto ev : c->ev_pool) (void)hipEventDestroy(ev);
    if (c->h_var) (void)hipHostFree(c->h_var);
    delete c;
}

int pool_event(adpsgd_ctx *c, hipEvent_t *ev) {
    if (!c->ev_pool.empty()) {
        *ev = c->ev_pool.back();
        c->ev_pool.pop_back();
        return ok();
    }
    HIP_TRY(hipEventCreate(ev));
    return ok();
}

// Fold finished timed launches into the totals (all of them if wait_all).
int harvest(adpsgd_ctx *c, bool wait_all) {
    while (!c->timed.empty()) {
        TimedLaunch tl = c->timed.front();
        if (wait_all) {
            HIP_TRY(hipEventSynchronize(tl.stop));
        } else {
            hipError_t q = hipEventQuery(tl.stop);
            if (q == hipErrorNotReady) break;
            if (q != hipSuccess) return hip_fail(q, "hipEventQuery");
        }
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, tl.start, tl.stop));
        c->t_ms[tl.kind] += ms;
        c->t_n[tl.kind] += 1;
        c->ev_pool.push_back(tl.start);
        c->ev_pool.push_back(tl.stop);
        c->timed.pop_front();
    }
    return ok();
}

template <class F>
int timed_launch(adpsgd_ctx *c, int kind, F launch) {
    if (!c->timing) {
        HIP_TRY(launch());
        return ok();
    }
    if ((int)c->timed.size() >= kTimedMax) {
        int rc = harvest(c, false);
        if (rc) return rc;
        if ((int)c->timed.size() >= kTimedMax) {
            rc = harvest(c, true);
            if (rc) return rc;
        }
    }
    TimedLaunch tl{kind, nullptr, nullptr};
    int rc = pool_event(c, &tl.start);
    if (rc) return rc;
    rc = pool_event(c, &tl.stop);
    if (rc) return rc;
    HIP_TRY(hipEventRecord(tl.start, c->stream));
    HIP_TRY(launch());
    HIP_TRY(hipEventRecord(tl.stop, c->stream));
    c->timed.push_back(tl);
    return ok();
}

StepParams step_params(const adpsgd_ctx *c, int64_t t) {
    StepParams p;
    p.x = c->buf.x;
    p.m = c->buf.m;
    p.h = c->buf.h;
    p.xs = c->buf.xstar;
    p.P = c->P;
    p.n_groups = (c->P + 3) / 4;
    p.K = c->K;
    p.t = (uint32_t)t;
    p.sigma = (float)c->hp.sigma;
    p.mu = (float)c->hp.momentum;
    p.wd = (float)c->hp.weight_decay;
    p.gamma = (float)adpsgd_lr(&c->hp, t);
    p.rk = c->rk;
    return p;
}

int enqueue_steps(adpsgd_ctx *c, int64_t t0, int64_t n) {
    for (int64_t j = 0; j < n; ++j) {
        const StepParams p = step_params(c, t0 + j);
        int rc = timed_launch(c, tStep, [&] { return launch_local_step(p, c->vec, c->nontemporal, c->stream); });
        if (rc) return rc;
    }
    return ok();
}

// A sync-tile kernel of the given mode at step t (the step is used by the
// modes with a step), with its per-tensor variances (and gradient norms)
// landing in ring slot `slot`.
int enqueue_sync(adpsgd_ctx *c, int mode, int64_t t, int slot) {
    SyncParams sp;
    sp.s = step_params(c, t);
    sp.tiles = c->d_tiles;
    sp.partials = c->d_tile_partials;
    const int64_t n_tiles = (int64_t)c->tiles.size();
    const int kind = mode == kAverage ? tAverage : mode == kTrace ? tTrace : tFused;
    int rc = timed_launch(c, kind, [&] {
        return launch_tile_sync(sp, n_tiles, mode, c->hp.avg_momentum != 0, c->vec, c->nontemporal, c->stream);
    });
    if (rc) return rc;
    double *dv = c->d_var + (size_t)slot * 2 * c->T;
    rc = timed_launch(c, tSegsum, [&] {
        return launch_segsum(c->d_chunks, (int64_t)c->chunks.size(), c->d_chunk_begin, c->d_tile_partials,
                             c->d_chunk_partials, dv, c->T, c->K, c->stream);
    });
    if (rc) return rc;
    HIP_TRY(hipMemcpyAsync(c->h_var + (size_t)slot * 2 * c->T, dv, 2 * sizeof(double) * c->T,
                           hipMemcpyDeviceToHost, c->stream));
    HIP_TRY(hipEventRecord(c->ring_ev[slot], c->stream));
    return ok();
}

double sum_var(const double *v, int32_t T) {
    double s = 0.0;
    for (int32_t i = 0; i < T; ++i) s += v[i];
    return s;
}

int check_ctx(const adpsgd_ctx *c) {
    if (!c) return fail(ADPSGD_EINVAL, "context is NULL");
    return ok();
}

}  // namespace

extern "C" const char *adpsgd_last_error(void) { return g_last_error.c_str(); }

extern "C" size_t adpsgd_workspace_bytes(int32_t K, int64_t P, int32_t T, const int64_t *offsets) {
    std::string why;
    if (!shape_valid(K, P, T, offsets, &why)) return 0;
    return layout_for(count_plan(T, offsets), T).total;
}

extern "C" int adpsgd_init(int32_t K, int64_t P, const int64_t *offsets, int32_t T, const adpsgd_hparams *hp,
                           const adpsgd_buffers *buf, adpsgd_ctx **out) {
    std::string why;
    if (!out) return fail(ADPSGD_EINVAL, "out is NULL");
    *out = nullptr;
    if (!shape_valid(K, P, T, offsets, &why)) return fail(ADPSGD_EINVAL, why);
    if (!hparams_valid(hp, &why)) return fail(ADPSGD_EINVAL, why);
    if (!buf) return fail(ADPSGD_EINVAL, "buffers is NULL");
    if (P > 0 && (!buf->x || !buf->m || !buf->h || !buf->xstar))
        return fail(ADPSGD_EINVAL, "x, m, h and xstar must be non-NULL");
    if (!aligned(buf->x, 16) || !aligned(buf->m, 16) || !aligned(buf->h, 16) || !aligned(buf->xstar, 16))
        return fail(ADPSGD_EINVAL, "x, m, h and xstar must be 16-byte aligned");
    const Plan plan = count_plan(T, offsets);
    if (plan.n_tiles >= (int64_t(1) << 31) || local_step_blocks((P + 3) / 4, K) >= (int64_t(1) << 31))
        return fail(ADPSGD_EINVAL, "K * P too large for one launch");
    const Layout lay = layout_for(plan, T);
    if (!buf->workspace || !aligned(buf->workspace, 256)) return fail(ADPSGD_EINVAL, "workspace must be 256-byte aligned");
    if (buf->workspace_bytes < lay.total)
        return fail(ADPSGD_EINVAL, "workspace too small: need " + std::to_string(lay.total) + " bytes");

    adpsgd_ctx *c = new (std::nothrow) adpsgd_ctx();
    if (!c) return fail(ADPSGD_EINVAL, "out of host memory");
    c->K = K;
    c->P = P;
    c->T = T;
    c->offsets.assign(offsets, offsets + T + 1);
    build_plan(T, offsets, &c->tiles, &c->chunks, &c->chunk_begin);
    c->hp = *hp;
    c->buf = *buf;
    c->stream = (hipStream_t)buf->stream;
    c->vec = (P % 4) == 0;
    // x and m beyond the 256 MB last-level cache: stream them past the caches
    c->nontemporal = (double)K * (double)P * 8.0 > 256.0 * 1024 * 1024;
    c->rk = round_keys(hp->seed);
    char *ws = (char *)buf->workspace;
    c->d_tiles = (Tile *)(ws + lay.tiles);
    c->d_chunks = (Chunk *)(ws + lay.chunks);
    c->d_chunk_begin = (int32_t *)(ws + lay.chunk_begin);
    c->d_tile_partials = (double *)(ws + lay.tile_partials);
    c->d_chunk_partials = (double *)(ws + lay.chunk_partials);
    c->d_var = (double *)(ws + lay.var);

    auto bail = [&](hipError_t e, const char *what) {
        int rc = hip_fail(e, what);
        std::string msg = g_last_error;
        release(c);
        g_last_error = msg;
        return rc;
    };
    hipError_t e;
    if ((e = hipGetDevice(&c->device)) != hipSuccess) return bail(e, "hipGetDevice");
    if ((e = hipHostMalloc((void **)&c->h_var, sizeof(double) * kRing * 2 * (size_t)T, hipHostMallocDefault)) !=
        hipSuccess)
        return bail(e, "hipHostMalloc");
    for (auto &ev : c->ring_ev)
        if ((e = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) return bail(e, "hipEventCreate");
    if (!c->tiles.empty() &&
        (e = hipMemcpyAsync(c->d_tiles, c->tiles.data(), sizeof(Tile) * c->tiles.size(), hipMemcpyHostToDevice,
                            c->stream)) != hipSuccess)
        return bail(e, "copy tile table");
    if (!c->chunks.empty() &&
        (e = hipMemcpyAsync(c->d_chunks, c->chunks.data(), sizeof(Chunk) * c->chunks.size(), hipMemcpyHostToDevice,
                            c->stream)) != hipSuccess)
        return bail(e, "copy chunk table");
    if ((e = hipMemcpyAsync(c->d_chunk_begin, c->chunk_begin.data(), sizeof(int32_t) * (T + 1),
                            hipMemcpyHostToDevice, c->stream)) != hipSuccess)
        return bail(e, "copy chunk offsets");
    if ((e = hipMemsetAsync(c->d_var, 0, sizeof(double) * kRing * 2 * (size_t)T, c->stream)) != hipSuccess)
        return bail(e, "clear variance ring");
    if (P > 0) {
        if ((e = launch_init_problem(buf->h, buf->xstar, P, hp->seed, hp->h_lo, hp->h_hi, c->stream)) != hipSuccess)
            return bail(e, "init_problem launch");
        const size_t bytes = sizeof(float) * (size_t)K * (size_t)P;
        if ((e = hipMemsetAsync(buf->x, 0, bytes, c->stream)) != hipSuccess) return bail(e, "zero x");
        if ((e = hipMemsetAsync(buf->m, 0, bytes, c->stream)) != hipSuccess) return bail(e, "zero m");
    }
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return bail(e, "hipStreamSynchronize");
    c->st = adpsgd_state{};
    c->st.p = hp->p_init;
    *out = c;
    return ok();
}

extern "C" int adpsgd_reset(adpsgd_ctx *c) {
    if (int rc = check_ctx(c)) return rc;
    if (c->P > 0) {
        const size_t bytes = sizeof(float) * (size_t)c->K * (size_t)c->P;
        HIP_TRY(hipMemsetAsync(c->buf.x, 0, bytes, c->stream));
        HIP_TRY(hipMemsetAsync(c->buf.m, 0, bytes, c->stream));
    }
    c->st = adpsgd_state{};
    c->st.p = c->hp.p_init;
    return ok();
}

extern "C" int adpsgd_local_steps(adpsgd_ctx *c, int32_t n) {
    if (int rc = check_ctx(c)) return rc;
    if (n < 0) return fail(ADPSGD_EINVAL, "n must be >= 0");
    if (c->st.t + n > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");
    if (int rc = enqueue_steps(c, c->st.t, n)) return rc;
    c->st.t += n;
    c->st.cnt += n;
    return ok();
}

static int sync_now(adpsgd_ctx *c, bool fused, double *var_out) {
    if (int rc = check_ctx(c)) return rc;
    if (!var_out) return fail(ADPSGD_EINVAL, "var_out is NULL");
    if (fused && c->st.t + 1 > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");
    if (int rc = enqueue_sync(c, fused ? kFused : kAverage, c->st.t, 0)) return rc;
    HIP_TRY(hipEventSynchronize(c->ring_ev[0]));
    std::memcpy(var_out, c->h_var, sizeof(double) * c->T);
    if (fused) c->st.t += 1;
    c->st.cnt = 0;
    return ok();
}

extern "C" int adpsgd_average(adpsgd_ctx *c, double *var_out) { return sync_now(c, false, var_out); }

extern "C" int adpsgd_step_average(adpsgd_ctx *c, double *var_out) { return sync_now(c, true, var_out); }

extern "C" int adpsgd_schedule(adpsgd_ctx *c, const double *var, int32_t *next_period) {
    if (int rc = check_ctx(c)) return rc;
    if (!var) return fail(ADPSGD_EINVAL, "var is NULL");
    if (c->st.t < 1) return fail(ADPSGD_ESTATE, "no step has been taken yet");
    int rc = adpsgd_sched_on_sync(&c->hp, &c->st, c->st.t - 1, sum_var(var, c->T), nullptr);
    if (next_period) *next_period = c->st.p;
    return rc;
}

// Algorithm 2 for n_steps steps (adpsgd_run, adpsgd_run_traced).  With a
// trace, every step takes a ring slot: plain steps run the tracing mode of the
// sync-tile kernel, sync steps its traced fused mode.
static int run_impl(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap, double *var_log,
                    adpsgd_step_rec *trace, int64_t trace_cap, int64_t *n_syncs) {
    if (int rc = check_ctx(c)) return rc;
    if (n_steps < 0 || log_cap < 0 || trace_cap < 0) return fail(ADPSGD_EINVAL, "n_steps and capacities must be >= 0");
    if (log_cap > 0 && !log) return fail(ADPSGD_EINVAL, "log is NULL with log_cap > 0");
    if (trace_cap > 0 && !trace) return fail(ADPSGD_EINVAL, "trace is NULL with trace_cap > 0");
    if (c->st.t + n_steps > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");

    const adpsgd_hparams &hp = c->hp;
    const bool adaptive = hp.period_mode == ADPSGD_PERIOD_ADAPTIVE;
    const bool traced = trace != nullptr;
    const int64_t t0 = c->st.t, end = c->st.t + n_steps;
    // plan: the schedule as enqueued on the stream (t, cnt, p).  c->st: the
    // controller's view (p, C2, nC2), advanced as syncs are read back in order.
    // They differ only while a decisive sync (one whose decision may move p) is
    // in flight; then only steps that end no period under p - 1, p or p + 1
    // are enqueued, so the GPU keeps working while the host waits.
    adpsgd_state plan = c->st;
    struct Pending { int64_t t; int32_t p; int slot; bool sync, decisive; };
    std::deque<Pending> pend;
    int64_t n_slots = 0, n_done = 0, lookahead = 0;
    bool blocked = false;
    int status = ADPSGD_OK;

    while (true) {
        while (status == ADPSGD_OK && plan.t < end && (int)pend.size() < kRing && (!blocked || lookahead > 0)) {
            const int64_t t = plan.t;
            int32_t due = 0;
            if ((status = adpsgd_sched_step(&hp, &plan, &due))) break;
            if (blocked) {
                // cnt <= max(p-1, 1) - 1 < p - 1: no period ends here for any p' >= p - 1
                --lookahead;
                if (due) { status = fail(ADPSGD_ESTATE, "internal: sync due inside the look-ahead"); break; }
            }
            if (!due && !traced) {
                status = enqueue_steps(c, t, 1);
                continue;
            }
            const int slot = (int)(n_slots % kRing);
            const int mode = due ? (traced ? kFusedTrace : kFused) : kTrace;
            if ((status = enqueue_sync(c, mode, t, slot))) break;
            ++n_slots;
            const bool decisive = due && adaptive && t >= hp.k_s && t >= hp.sync_warmup_steps;
            pend.push_back(Pending{t, plan.p, slot, due != 0, decisive});
            if (!due) continue;
            plan.cnt = 0;
            if (decisive) {
                blocked = true;
                lookahead = std::max(plan.p - 1, 1) - 1;
            }
        }
        if (pend.empty() || status != ADPSGD_OK) break;
        const Pending q = pend.front();
        pend.pop_front();
        hipError_t e = hipEventSynchronize(c->ring_ev[q.slot]);
        if (e != hipSuccess) { status = hip_fail(e, "wait for variance"); break; }
        const double *var = c->h_var + (size_t)q.slot * 2 * c->T;
        const double S = sum_var(var, c->T);
        if (traced && q.t - t0 < trace_cap)
            trace[q.t - t0] = adpsgd_step_rec{q.t, q.sync ? 1 : 0, q.p, S, sum_var(var + c->T, c->T),
                                              adpsgd_lr(&hp, q.t)};
        if (q.sync) {
            double margin = std::numeric_limits<double>::quiet_NaN();
            const int rc = adpsgd_sched_on_sync(&hp, &c->st, q.t, S, &margin);
            if (n_done < log_cap) {
                log[n_done] = adpsgd_sync_rec{q.t, q.p, 0, S, c->st.C2, adpsgd_lr(&hp, q.t), margin};
                if (var_log) std::memcpy(var_log + (size_t)n_done * c->T, var, sizeof(double) * c->T);
            }
            ++n_done;
            if (rc) { status = rc; break; }
            if (q.decisive) {
                plan.p = c->st.p;
                blocked = false;
                lookahead = 0;
            }
        }
        if (c->timing) {
            int hr = harvest(c, false);
            if (hr) { status = hr; break; }
        }
    }
    // whatever was enqueued runs to completion; the state reflects it (on an
    // error, p keeps the value in force before the failing sync)
    hipError_t e = hipStreamSynchronize(c->stream);
    c->st.t = plan.t;
    c->st.cnt = plan.cnt;
    if (!blocked) c->st.p = plan.p;
    if (n_syncs) *n_syncs = n_done;
    if (status != ADPSGD_OK) return status;
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    return ok();
}

extern "C" int adpsgd_run(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap, double *var_log,
                          int64_t *n_syncs) {
    return run_impl(c, n_steps, log, log_cap, var_log, nullptr, 0, n_syncs);
}

extern "C" int adpsgd_run_traced(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap,
                                 double *var_log, adpsgd_step_rec *trace, int64_t trace_cap, int64_t *n_syncs) {
    if (!trace) return fail(ADPSGD_EINVAL, "trace is NULL");
    return run_impl(c, n_steps, log, log_cap, var_log, trace, trace_cap, n_syncs);
}

extern "C" int adpsgd_get_state(const adpsgd_ctx *c, adpsgd_state *out) {
    if (int rc = check_ctx(c)) return rc;
    if (!out) return fail(ADPSGD_EINVAL, "out is NULL");
    *out = c->st;
    return ok();
}

extern "C" int adpsgd_set_state(adpsgd_ctx *c, const adpsgd_state *in) {
    if (int rc = check_ctx(c)) return rc;
    if (!in) return fail(ADPSGD_EINVAL, "state is NULL");
    if (in->t < 0 || in->t >= kMaxCounter || in->cnt < 0 || in->nC2 < 0 || in->p < 1 || in->p > p_max_of(&c->hp) ||
        !std::isfinite(in->C2))
        return fail(ADPSGD_EINVAL, "invalid state");
    c->st = *in;
    return ok();
}

extern "C" int adpsgd_set_timing(adpsgd_ctx *c, int32_t on) {
    if (int rc = check_ctx(c)) return rc;
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (int rc = harvest(c, true)) return rc;
    c->timing = on != 0;
    for (int i = 0; i < tKinds; ++i) { c->t_ms[i] = 0.0; c->t_n[i] = 0; }
    return ok();
}

extern "C" int adpsgd_get_timing(adpsgd_ctx *c, adpsgd_timing *out) {
    if (int rc = check_ctx(c)) return rc;
    if (!out) return fail(ADPSGD_EINVAL, "out is NULL");
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (int rc = harvest(c, true)) return rc;
    *out = adpsgd_timing{c->t_ms[tStep],  c->t_n[tStep],   c->t_ms[tFused],  c->t_n[tFused],
                         c->t_ms[tAverage], c->t_n[tAverage], c->t_ms[tSegsum], c->t_n[tSegsum],
                         c->t_ms[tTrace], c->t_n[tTrace]};
    return ok();
}

extern "C" int adpsgd_destroy(adpsgd_ctx *c) {
    if (!c) return ok();
    hipError_t e = hipStreamSynchronize(c->stream);
    release(c);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    return ok();
}

extern "C" int adpsgd_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n_groups,
                                  uint32_t *dev_out, void *stream) {
    if (n_groups < 0 || g0 < 0 || g0 + n_groups > kMaxCounter) return fail(ADPSGD_EINVAL, "bad group range");
    if (n_groups > 0 && (!dev_out || !aligned(dev_out, 16))) return fail(ADPSGD_EINVAL, "dev_out must be 16-byte aligned");
    HIP_TRY(launch_philox_dump(seed, c1, c2, c3, g0, n_groups, dev_out, (hipStream_t)stream));
    return ok();
}

extern "C" int adpsgd_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n_groups,
                                  float *dev_out, void *stream) {
    if (n_groups < 0 || g0 < 0 || g0 + n_groups > kMaxCounter) return fail(ADPSGD_EINVAL, "bad group range");
    if (n_groups > 0 && (!dev_out || !aligned(dev_out, 16))) return fail(ADPSGD_EINVAL, "dev_out must be 16-byte aligned");
    HIP_TRY(launch_normal_dump(seed, c1, c2, c3, g0, n_groups, dev_out, (hipStream_t)stream));
    return ok();
}
