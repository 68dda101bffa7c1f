// Host runtime and C ABI of the ADPSGD hot path: argument validation, the tile
// table of the segmented variance reduction, kernel launches on the caller's
// stream, the Algorithm 2 driver (host-planned steps, device-decided syncs
// where the host has not yet read a decision back), checkpoint state and
// timing.
#include <hip/hip_runtime.h>

#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <deque>
#include <limits>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
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

// Windows of tensors for the second level of the variance sum when there are
// more chunk partials than one LDS window holds: runs of whole small tensors
// (at most kSmallTensorChunks chunks each) whose chunks fit kFinishWindow, and
// every larger tensor alone.  win_begin receives the first tensor of each
// window and T; returns the window count (0, with win_begin empty, when one
// window holds every chunk partial).
int32_t reduce_windows(int32_t T, const int32_t *chunk_begin, std::vector<int32_t> *win_begin) {
    win_begin->clear();
    if (chunk_begin[T] <= kFinishWindow) return 0;
    win_begin->push_back(0);
    int32_t cur = 0;  // chunks in the current run of small tensors
    for (int32_t tau = 0; tau < T; ++tau) {
        const int32_t c = chunk_begin[tau + 1] - chunk_begin[tau];
        if (c > kSmallTensorChunks) {
            if (tau > win_begin->back()) win_begin->push_back(tau);
            win_begin->push_back(tau + 1);
            cur = 0;
        } else if (cur + c > kFinishWindow) {
            win_begin->push_back(tau);
            cur = c;
        } else {
            cur += c;
        }
    }
    if (win_begin->back() < T) win_begin->push_back(T);
    return (int32_t)win_begin->size() - 1;
}

namespace {

constexpr int kRing = 32;          // record slots: launches with a reduction in flight at once
constexpr int kTimedMax = 4096;    // pending timed launches before a harvest
constexpr int64_t kMaxInflight = 1024;  // launched steps the host has not yet accounted for
// The driver waits for an outstanding decision when at least this many steps
// are queued behind it (the GPU stays busy meanwhile); otherwise it lets the
// device decide, for at most kMaxUncertain steps in a row.
constexpr int64_t kQueueToWait = 1;
constexpr int kMaxUncertain = 2;
// Between waits, the driver polls for finished records every kPollEvery launches
// (each poll is a runtime call; plain steps need no accounting to proceed).
constexpr int64_t kPollEvery = 8;
// adpsgd_init times the local step's block sizes when one step moves at least
// this many elements (below it a launch is too short to time reliably).
constexpr double kTuneMinElems = 16.0 * 1024 * 1024;
// Below the same size a step takes a few microseconds on the GPU, less than
// the host needs to launch it, so runs whose schedule is known in advance
// (the constant-period modes) are captured once as a HIP graph and replayed;
// runs of up to kGraphMaxSteps steps.
constexpr double kGraphMaxElems = kTuneMinElems;
constexpr int64_t kGraphMaxSteps = int64_t(1) << 16;
constexpr int64_t kMaxK = 65536;
constexpr int64_t kMaxCounter = int64_t(1) << 32;  // Philox counter words are 32-bit

enum TimedKind { tStep = 0, tFused = 1, tAverage = 2, tSegsum = 3, tTrace = 4, tKinds = 5 };
// Sampling classes of the timer: the timed kinds, plus the device-decided
// step kernels whose kind is known only when their record is read.
enum { cDeviceStep = tKinds, kTimedClasses = tKinds + 1 };

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
// Chunks: runs of at most chunk_tiles consecutive tiles of one tensor, where
// chunk_tiles is 1 for at most kDirectMaxTiles tiles (the tile partials then
// serve as chunk partials) and kChunkTiles otherwise.
int64_t tiles_of(int64_t a, int64_t b) { return b > a ? (b + kTileElems - 1) / kTileElems - a / kTileElems : 0; }

struct Plan {
    int64_t n_tiles = 0, n_chunks = 0;
    int64_t n_aligned = 0;  // aligned chunks of kTileElems elements (a sync-tile block each)
    int32_t chunk_tiles = kChunkTiles;
    int32_t n_windows = 0;  // windows of tensors for k_reduce_windows (0: none)
};

Plan count_plan(int32_t T, const int64_t *off) {
    Plan pl;
    for (int32_t tau = 0; tau < T; ++tau) pl.n_tiles += tiles_of(off[tau], off[tau + 1]);
    pl.n_aligned = (off[T] + kTileElems - 1) / kTileElems;
    pl.chunk_tiles = pl.n_tiles <= kDirectMaxTiles ? 1 : kChunkTiles;
    std::vector<int32_t> chunk_begin(T + 1, 0);
    for (int32_t tau = 0; tau < T; ++tau) {
        const int64_t n = (tiles_of(off[tau], off[tau + 1]) + pl.chunk_tiles - 1) / pl.chunk_tiles;
        chunk_begin[tau + 1] = chunk_begin[tau] + (int32_t)n;
        pl.n_chunks += n;
    }
    std::vector<int32_t> win_begin;
    pl.n_windows = reduce_windows(T, chunk_begin.data(), &win_begin);
    return pl;
}

void build_plan(int32_t T, const int64_t *off, int32_t chunk_tiles, std::vector<Tile> *tiles,
                std::vector<Chunk> *chunks, std::vector<int32_t> *chunk_begin) {
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
        for (int32_t c = 0; c < n; c += chunk_tiles)
            chunks->push_back(Chunk{first_tile + c, std::min(chunk_tiles, n - c), tau, 0});
    }
    (*chunk_begin)[T] = (int32_t)chunks->size();
}

struct Layout {
    size_t tiles, chunks, chunk_begin, large, tile_partials, chunk_partials, acc, win_begin, win_partials, sched,
        chunk_seg, total;
};

// A record slot (pinned host memory the reduction writes directly): the
// header, then the T variances and the T gradient norms.
size_t slot_bytes_for(int32_t T) { return align_up(kSlotHdrBytes + 2 * sizeof(double) * (size_t)T, 256); }

Layout layout_for(const Plan &pl, int32_t T) {
    auto at_least_one = [](int64_t n) { return (size_t)std::max<int64_t>(n, 1); };
    Layout l;
    l.tiles = 0;
    l.chunks = align_up(l.tiles + sizeof(Tile) * at_least_one(pl.n_tiles), 256);
    l.chunk_begin = align_up(l.chunks + sizeof(Chunk) * at_least_one(pl.n_chunks), 256);
    l.large = align_up(l.chunk_begin + sizeof(int32_t) * (size_t)(T + 1), 256);
    l.tile_partials = align_up(l.large + sizeof(int32_t) * (size_t)T, 256);
    l.chunk_partials = align_up(l.tile_partials + 2 * sizeof(double) * at_least_one(pl.n_tiles), 256);
    l.acc = align_up(l.chunk_partials + 2 * sizeof(double) * at_least_one(pl.n_chunks), 256);
    l.win_begin = align_up(l.acc + 2 * sizeof(double) * (size_t)T, 256);
    l.win_partials = align_up(l.win_begin + sizeof(int32_t) * (size_t)(pl.n_windows + 1), 256);
    l.sched = align_up(l.win_partials + 2 * sizeof(double) * at_least_one(pl.n_windows), 256);
    l.chunk_seg = align_up(l.sched + sizeof(SchedState), 256);
    l.total = align_up(l.chunk_seg + sizeof(int32_t) * (size_t)(pl.n_aligned + 1), 256);
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
    int64_t ld = 0;                 // row stride of x and m (elements)
    int32_t T = 0;
    std::vector<int64_t> offsets;
    std::vector<Tile> tiles;
    std::vector<Chunk> chunks;
    std::vector<int32_t> chunk_begin;
    std::vector<int32_t> large;     // tensors of more than kSmallTensorChunks chunks
    std::vector<int32_t> win_begin; // windows of tensors for k_reduce_windows (empty: none)
    int32_t *d_win_begin = nullptr;
    double *d_win_partials = nullptr;
    adpsgd_hparams hp{};
    adpsgd_buffers buf{};
    hipStream_t stream = nullptr;
    int device = 0;
    Tile *d_tiles = nullptr;
    Chunk *d_chunks = nullptr;
    int32_t *d_chunk_begin = nullptr;
    int32_t *d_large = nullptr;
    std::vector<int32_t> chunk_seg; // first tile of each aligned chunk (the sync-tile kernel's blocks)
    int32_t *d_chunk_seg = nullptr;
    bool chunks_are_tiles = false;  // every tile is its own chunk (small problems)
    double *d_tile_partials = nullptr;
    double *d_chunk_partials = nullptr;
    double *d_acc = nullptr;        // [2T] reduction scratch
    SchedState *d_sched = nullptr;  // the controller state as the device sees it during a run
    char *h_slots = nullptr;        // [kRing] record slots: pinned, coherent host memory
    char *d_slots = nullptr;        // the same slots as the device addresses them
    SchedState *h_sched = nullptr;  // pinned staging for the device controller state
    size_t slot_bytes = 0;
    hipEvent_t ring_ev[kRing] = {};
    adpsgd_state st{};
    bool vec = true;                // row stride % 4 == 0: rows 16-byte aligned, dwordx4 groups
    bool nontemporal = false;       // stream x and m past the caches (large working sets)
    // the sync-tile kernel's choice of the same, timed at init on large working
    // sets: the step + sync modes (fused, device-decided, traced) and the separate sync
    bool sync_nt = false;
    bool average_nt = false;
    int32_t policy = ADPSGD_LAUNCH_HYBRID;
    StepShape step_shape{256, 0, 1};   // launch shape of the plain local step in use
    StepShape tuned_shape{256, 0, 1};  // the fastest one measured at init
    int32_t average_cap = 0;        // resident blocks per CU of the separate sync (0: no cap), timed at init
    RoundKeys rk{};
    bool timing = false;
    int32_t timing_every = 1;       // time every n-th launch of each class
    int64_t class_count[kTimedClasses] = {};
    std::deque<TimedLaunch> timed;
    int64_t timed_popped = 0;       // timed launches harvested so far (sequence of timed.front())
    std::vector<hipEvent_t> ev_pool;
    double t_ms[tKinds] = {};
    int64_t t_n[tKinds] = {};
    // A constant-period run captured as a HIP graph (run_impl): captured on a
    // private non-blocking stream, launched on the context's stream, kept for
    // as long as runs repeat with the same start state, length and launch shape.
    hipStream_t cap_stream = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t graph_exec = nullptr;
    int64_t graph_key[7] = {};
    int64_t graph_captures = 0, graph_replays = 0;   // since the last adpsgd_set_timing
    char *h_gslots = nullptr;       // one record slot per sync of the captured run (pinned)
    char *d_gslots = nullptr;
    int64_t gslot_cap = 0;
};

namespace {

void drop_graph(adpsgd_ctx *c) {
    if (c->graph_exec) (void)hipGraphExecDestroy(c->graph_exec);
    if (c->graph) (void)hipGraphDestroy(c->graph);
    c->graph_exec = nullptr;
    c->graph = nullptr;
}

void release(adpsgd_ctx *c) {
    if (!c) return;
    drop_graph(c);
    if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
    if (c->h_gslots) (void)hipHostFree(c->h_gslots);
    for (auto &ev : c->ring_ev)
        if (ev) (void)hipEventDestroy(ev);
    for (auto &tl : c->timed) {
        (void)hipEventDestroy(tl.start);
        (void)hipEventDestroy(tl.stop);
    }
    for (auto ev : c->ev_pool) (void)hipEventDestroy(ev);
    if (c->h_slots) (void)hipHostFree(c->h_slots);
    if (c->h_sched) (void)hipHostFree(c->h_sched);
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

// Fold finished timed launches into the totals (all of them if wait_all).  A
// launch whose kind is still open (-1: a device-decided step the driver has
// not accounted for) stops a non-waiting harvest.
int harvest(adpsgd_ctx *c, bool wait_all) {
    while (!c->timed.empty()) {
        TimedLaunch tl = c->timed.front();
        if (wait_all) {
            HIP_TRY(hipEventSynchronize(tl.stop));
        } else {
            if (tl.kind < 0) break;
            hipError_t q = hipEventQuery(tl.stop);
            if (q == hipErrorNotReady) break;
            if (q != hipSuccess) return hip_fail(q, "hipEventQuery");
        }
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, tl.start, tl.stop));
        const int kind = tl.kind < 0 ? tStep : tl.kind;
        c->t_ms[kind] += ms;
        c->t_n[kind] += 1;
        c->ev_pool.push_back(tl.start);
        c->ev_pool.push_back(tl.stop);
        c->timed.pop_front();
        ++c->timed_popped;
    }
    return ok();
}

// Launch, with HIP events around it when timing is on and this is the
// sampled launch (every timing_every-th) of its class.  kind -1: decided later
// (set_timed_kind).  *seq (may be null) receives the launch's sequence number,
// or -1 when it is not timed.
template <class F>
int timed_launch(adpsgd_ctx *c, int kind, F launch, int64_t *seq = nullptr) {
    if (seq) *seq = -1;
    const int cls = kind < 0 ? cDeviceStep : kind;
    if (!c->timing || (c->class_count[cls]++ % c->timing_every) != 0) {
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
    if (seq) *seq = c->timed_popped + (int64_t)c->timed.size();
    c->timed.push_back(tl);
    return ok();
}

void set_timed_kind(adpsgd_ctx *c, int64_t seq, int kind) {
    const int64_t i = seq - c->timed_popped;
    if (seq >= 0 && i >= 0 && i < (int64_t)c->timed.size()) c->timed[(size_t)i].kind = kind;
}

StepParams step_params(const adpsgd_ctx *c, int64_t t) {
    StepParams p;
    p.x = c->buf.x;
    p.m = c->buf.m;
    p.h = c->buf.h;
    p.xs = c->buf.xstar;
    p.ld = c->ld;
    p.P = c->P;
    p.n_groups = (c->P + 3) / 4;
    p.K = c->K;
    p.t = (uint32_t)t;
    p.sigma = (float)c->hp.sigma;
    p.mu = (float)c->hp.momentum;
    p.wd = (float)c->hp.weight_decay;
    p.gamma = (float)adpsgd_lr(&c->hp, t);
    p.rk = c->rk;
    p.row_chunks = 1;  // set by launch_local_step from the launch shape
    p.pad_ = 0;
    p.block0 = 0;
    return p;
}

int enqueue_steps(adpsgd_ctx *c, int64_t t0, int64_t n) {
    for (int64_t j = 0; j < n; ++j) {
        const StepParams p = step_params(c, t0 + j);
        int rc = timed_launch(c, tStep, [&] { return launch_local_step(p, c->vec, c->nontemporal, c->step_shape, c->stream); });
        if (rc) return rc;
    }
    return ok();
}

SyncParams sync_params(const adpsgd_ctx *c, int64_t t) {
    SyncParams sp;
    sp.s = step_params(c, t);
    sp.tiles = c->d_tiles;
    sp.partials = c->d_tile_partials;
    sp.chunk_seg = c->d_chunk_seg;
    sp.n_chunks = (int64_t)c->chunk_seg.size() - 1;
    sp.sched = c->d_sched;
    sp.rule = rule_of(&c->hp);
    return sp;
}

char *slot_dev(const adpsgd_ctx *c, int slot) { return c->d_slots + (size_t)slot * c->slot_bytes; }
const char *slot_host(const adpsgd_ctx *c, int slot) { return c->h_slots + (size_t)slot * c->slot_bytes; }

// The reduction after a sync-tile kernel at step t, writing its record to the
// slot at device address `slot` (with the controller on the device when ctl).
ReduceParams reduce_params(const adpsgd_ctx *c, int mode, int64_t t, char *slot, bool ctl) {
    ReduceParams r;
    r.tile_partials = c->d_tile_partials;
    r.chunks = c->d_chunks;
    r.chunk_begin = c->d_chunk_begin;
    r.chunk_partials = c->chunks_are_tiles ? c->d_tile_partials : c->d_chunk_partials;
    r.chunks_are_tiles = c->chunks_are_tiles ? 1 : 0;
    r.block0 = 0;
    r.acc = c->d_acc;
    r.n_chunks = (int32_t)c->chunks.size();
    r.T = c->T;
    r.K = c->K;
    r.large = c->d_large;
    r.n_large = (int32_t)c->large.size();
    r.win_begin = c->d_win_begin;
    r.win_partials = c->d_win_partials;
    r.n_windows = c->win_begin.empty() ? 0 : (int32_t)c->win_begin.size() - 1;
    r.pad2_ = 0;
    r.hdr = reinterpret_cast<SlotHdr *>(slot);
    r.out = reinterpret_cast<double *>(slot + kSlotHdrBytes);
    r.sched = ctl ? c->d_sched : nullptr;
    r.rule = rule_of(&c->hp);
    r.t = t;
    r.gamma = adpsgd_lr(&c->hp, t);
    r.traced = mode == kDeviceTrace ? 1 : 0;
    return r;
}

// The sync-tile kernel of the given mode at step t, then the reduction into
// record slot `slot` (with the controller on the device when ctl), then the
// slot's event.  *step_seq: the timed sequence number of the tile kernel (its
// kind is open for the device-decided modes).
int enqueue_sync(adpsgd_ctx *c, int mode, int64_t t, int slot, bool ctl, int64_t *step_seq) {
    const bool dev = mode == kDevice || mode == kDeviceTrace;
    const SyncParams sp = sync_params(c, t);
    const int64_t n_tiles = (int64_t)c->tiles.size();
    const int kind = dev ? -1 : mode == kAverage ? tAverage : tFused;
    int rc = timed_launch(
        c, kind,
        [&] {
            return launch_tile_sync(sp, n_tiles, mode, c->hp.avg_momentum != 0, c->vec,
                                    mode == kAverage ? c->average_nt : c->sync_nt,
                                    mode == kAverage ? c->average_cap : 0, c->stream);
        },
        step_seq);
    if (rc) return rc;
    const ReduceParams r = reduce_params(c, mode, t, slot_dev(c, slot), ctl);
    rc = timed_launch(c, tSegsum, [&] { return launch_reduce(r, c->stream); });
    if (rc) return rc;
    HIP_TRY(hipEventRecord(c->ring_ev[slot], c->stream));
    return ok();
}

// Capture steps t0 .. t0 + due.size() - 1 as a graph, launched as the eager
// driver launches a schedule it knows in advance: plain steps, and for the
// j-th sync the fused step + sync and the reduction (controller on the device)
// into the j-th graph record slot.  No events: records are read after the
// whole graph has run.
int capture_run(adpsgd_ctx *c, int64_t t0, const std::vector<char> &due, int64_t n_sync) {
    drop_graph(c);
    if (n_sync > c->gslot_cap) {
        if (c->h_gslots) (void)hipHostFree(c->h_gslots);
        c->h_gslots = c->d_gslots = nullptr;
        c->gslot_cap = 0;
        HIP_TRY(hipHostMalloc((void **)&c->h_gslots, (size_t)n_sync * c->slot_bytes,
                              hipHostMallocMapped | hipHostMallocCoherent));
        HIP_TRY(hipHostGetDevicePointer((void **)&c->d_gslots, c->h_gslots, 0));
        c->gslot_cap = n_sync;
    }
    if (!c->cap_stream) HIP_TRY(hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking));
    const hipStream_t cs = c->cap_stream;
    const int64_t n_tiles = (int64_t)c->tiles.size();
    HIP_TRY(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal));
    hipError_t e = hipSuccess;
    int64_t j = 0;
    for (size_t i = 0; i < due.size() && e == hipSuccess; ++i) {
        const int64_t t = t0 + (int64_t)i;
        if (!due[i]) {
            e = launch_local_step(step_params(c, t), c->vec, c->nontemporal, c->step_shape, cs);
        } else {
            e = launch_tile_sync(sync_params(c, t), n_tiles, kFused, c->hp.avg_momentum != 0, c->vec, c->sync_nt, 0,
                                 cs);
            if (e == hipSuccess)
                e = launch_reduce(reduce_params(c, kFused, t, c->d_gslots + (size_t)j * c->slot_bytes, true), cs);
            ++j;
        }
    }
    hipGraph_t g = nullptr;
    const hipError_t e_end = hipStreamEndCapture(cs, &g);
    if (e == hipSuccess) e = e_end;
    if (e == hipSuccess) e = hipGraphInstantiate(&c->graph_exec, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        c->graph_exec = nullptr;
        return hip_fail(e, "capture the run as a HIP graph");
    }
    c->graph = g;
    return ok();
}

double sum_var(const double *v, int32_t T) {
    double s = 0.0;
    for (int32_t i = 0; i < T; ++i) s += v[i];
    return s;
}

// Contexts created by adpsgd_init and not yet destroyed: a call with any other
// pointer (a destroyed context, say) is refused instead of touching freed memory.
std::mutex g_live_mu;
std::unordered_set<const adpsgd_ctx *> g_live;

int check_ctx(const adpsgd_ctx *c) {
    if (!c) return fail(ADPSGD_EINVAL, "context is NULL");
    std::lock_guard<std::mutex> lock(g_live_mu);
    if (!g_live.count(c)) return fail(ADPSGD_EINVAL, "not a live context (destroyed, or not made by adpsgd_init)");
    return ok();
}

// The context's device made current for the duration of a call, and the
// caller's restored afterwards (a context's buffers, stream and events belong
// to the device that was current at adpsgd_init).
struct DeviceScope {
    int prev = -1;
    explicit DeviceScope(const adpsgd_ctx *c) {
        int cur = -1;
        if (hipGetDevice(&cur) == hipSuccess && cur != c->device && hipSetDevice(c->device) == hipSuccess) prev = cur;
    }
    ~DeviceScope() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
    DeviceScope(const DeviceScope &) = delete;
    DeviceScope &operator=(const DeviceScope &) = delete;
};

// A roctx range for the duration of a call (visible with rocprofv3 --marker-trace).
struct Range {
    explicit Range(const char *name) { roctxRangePushA(name); }
    ~Range() { roctxRangePop(); }
    Range(const Range &) = delete;
    Range &operator=(const Range &) = delete;
};

// Zero the K rows of x and m (P elements each, row_stride apart; the padding
// between rows is the caller's and is left alone), with a fill kernel.
hipError_t zero_rows(const adpsgd_ctx *c) {
    hipError_t e = launch_zero_rows(c->buf.x, c->ld, c->P, c->K, c->vec, c->stream);
    if (e == hipSuccess) e = launch_zero_rows(c->buf.m, c->ld, c->P, c->K, c->vec, c->stream);
    return e;
}

// The fastest of n launch variants on the context's stream: one warm-up launch
// each, then five rounds; a round queues every variant back to back with an
// event between consecutive launches, so each interval is the GPU's time for
// one launch (no host round trip inside it).  The fastest minimum wins.
constexpr int kMaxVariants = 8;

template <class Launch>
hipError_t fastest_variant(adpsgd_ctx *c, int n, Launch launch, int *win) {
    if (n < 1 || n > kMaxVariants) return hipErrorInvalidValue;
    hipEvent_t ev[kMaxVariants + 1] = {};
    hipError_t e = hipSuccess;
    for (int j = 0; j <= n && e == hipSuccess; ++j) e = hipEventCreate(&ev[j]);
    float best[kMaxVariants];
    for (int j = 0; j < n; ++j) best[j] = 3.4e38f;
    for (int j = 0; j < n && e == hipSuccess; ++j) e = launch(j);
    for (int round = 0; round < 5 && e == hipSuccess; ++round) {
        e = hipEventRecord(ev[0], c->stream);
        for (int j = 0; j < n && e == hipSuccess; ++j)
            if ((e = launch(j)) == hipSuccess) e = hipEventRecord(ev[j + 1], c->stream);
        if (e == hipSuccess) e = hipEventSynchronize(ev[n]);
        for (int j = 0; j < n && e == hipSuccess; ++j) {
            float ms = 0.f;
            if ((e = hipEventElapsedTime(&ms, ev[j], ev[j + 1])) == hipSuccess) best[j] = std::min(best[j], ms);
        }
    }
    if (e == hipSuccess) {
        *win = 0;
        for (int j = 1; j < n; ++j)
            if (best[j] < best[*win]) *win = j;
    }
    for (int j = 0; j <= n; ++j)
        if (ev[j]) (void)hipEventDestroy(ev[j]);
    return e;
}

// Time the local step in every launch shape on the context's own buffers (the
// launches step x and m, which the caller zeroes afterwards).
hipError_t tune_step_shape(adpsgd_ctx *c) {
    const StepParams p = step_params(c, 0);
    constexpr int n = (int)(sizeof(kStepShapes) / sizeof(kStepShapes[0]));
    static_assert(n <= kMaxVariants, "more step shapes than the timing helper takes");
    int win = 0;
    const hipError_t e = fastest_variant(
        c, n, [&](int j) { return launch_local_step(p, c->vec, c->nontemporal, kStepShapes[j], c->stream); }, &win);
    if (e == hipSuccess) c->tuned_shape = c->step_shape = kStepShapes[win];
    return e;
}

// The fastest of n launch sequences, each timed in a block of its own: one
// untimed call (which also pays for what the sequence before it left in the
// caches), then `reps` timed calls back to back; two passes over the
// variants, the smaller mean of the two counts.
template <class Launch>
hipError_t fastest_in_blocks(adpsgd_ctx *c, int n, int reps, Launch launch, int *win) {
    if (n < 1 || n > kMaxVariants || reps < 1) return hipErrorInvalidValue;
    hipEvent_t ev[2] = {};
    hipError_t e = hipEventCreate(&ev[0]);
    if (e == hipSuccess) e = hipEventCreate(&ev[1]);
    float best[kMaxVariants];
    for (int j = 0; j < n; ++j) best[j] = 3.4e38f;
    for (int pass = 0; pass < 2 && e == hipSuccess; ++pass)
        for (int j = 0; j < n && e == hipSuccess; ++j) {
            e = launch(j);
            if (e == hipSuccess) e = hipEventRecord(ev[0], c->stream);
            for (int r = 0; r < reps && e == hipSuccess; ++r) e = launch(j);
            if (e == hipSuccess) e = hipEventRecord(ev[1], c->stream);
            if (e == hipSuccess) e = hipEventSynchronize(ev[1]);
            float ms = 0.f;
            if (e == hipSuccess && (e = hipEventElapsedTime(&ms, ev[0], ev[1])) == hipSuccess)
                best[j] = std::min(best[j], ms);
        }
    if (e == hipSuccess) {
        *win = 0;
        for (int j = 1; j < n; ++j)
            if (best[j] < best[*win]) *win = j;
    }
    for (hipEvent_t x : ev)
        if (x) (void)hipEventDestroy(x);
    return e;
}

// Whether the step + sync modes keep non-temporal accesses.  Beyond 1 GiB of
// x and m they do (measured 10% faster at K = 8, P = 138M).  Between the
// last-level cache's 256 MB and 1 GiB it depends on the problem (the fused
// step + sync measured 14% faster without them at K = 32, P = 1.2M, and 14%
// slower at K = 8, P = 11.2M), so time periods of four steps (three plain
// steps, non-temporal as always, then the fused step + sync) with the sync's
// accesses non-temporal and not.  The launches step x and m, which the caller
// zeroes afterwards.
constexpr double kSyncNtTuneMaxBytes = 1024.0 * 1024 * 1024;

hipError_t tune_sync_nt(adpsgd_ctx *c) {
    c->sync_nt = c->nontemporal;
    if (!c->nontemporal || c->tiles.empty() || (double)c->K * (double)c->P * 8.0 > kSyncNtTuneMaxBytes)
        return hipSuccess;
    const StepParams stp = step_params(c, 0);
    const SyncParams sp = sync_params(c, 3);
    const int64_t n_tiles = (int64_t)c->tiles.size();
    int win = 0;
    const hipError_t e = fastest_in_blocks(
        c, 2, 3,
        [&](int j) {
            hipError_t le = hipSuccess;
            for (int i = 0; i < 3 && le == hipSuccess; ++i)
                le = launch_local_step(stp, c->vec, c->nontemporal, c->step_shape, c->stream);
            if (le == hipSuccess)
                le = launch_tile_sync(sp, n_tiles, kFused, c->hp.avg_momentum != 0, c->vec, j == 0, 0, c->stream);
            return le;
        },
        &win);
    if (e == hipSuccess) c->sync_nt = win == 0;
    return e;
}

// Time the separate sync (mean, broadcast and variance of every tile, no step)
// without and with an LDS cap that holds a CU to kAverageCapWaves resident
// waves and, on x and m of 256 MB to 1 GiB (beyond the last-level cache, see
// tune_sync_nt), with and without non-temporal accesses, on the context's own
// buffers (zeroed again afterwards).
hipError_t tune_average(adpsgd_ctx *c) {
    const int waves = sync_tile_waves(c->K, kAverage);
    if (waves <= 0 || c->tiles.empty()) return hipSuccess;
    const int caps[2] = {0, std::max(1, kAverageCapWaves / waves)};
    const bool both = c->nontemporal && (double)c->K * (double)c->P * 8.0 <= kSyncNtTuneMaxBytes;
    const int n = both ? 4 : 2;   // j: cap caps[j & 1], non-temporal while j < 2 (if at all)
    const SyncParams sp = sync_params(c, 0);
    const int64_t n_tiles = (int64_t)c->tiles.size();
    int win = 0;
    const hipError_t e = fastest_in_blocks(
        c, n, 3,
        [&](int j) {
            return launch_tile_sync(sp, n_tiles, kAverage, c->hp.avg_momentum != 0, c->vec, c->nontemporal && j < 2,
                                    caps[j & 1], c->stream);
        },
        &win);
    if (e == hipSuccess) {
        c->average_cap = caps[win & 1];
        c->average_nt = c->nontemporal && win < 2;
    }
    return e;
}

}  // namespace

extern "C" const char *adpsgd_last_error(void) { return g_last_error.c_str(); }

extern "C" int64_t adpsgd_padded_row_stride(int64_t P) {
    if (P <= 0) return 0;
    const int64_t n = (P - 1) / 256 + 1;
    return 256 * (n | 1);
}

extern "C" size_t adpsgd_workspace_bytes(int32_t K, int64_t P, int32_t T, const int64_t *offsets) {
    std::string why;
    if (!shape_valid(K, P, T, offsets, &why)) return 0;
    return layout_for(count_plan(T, offsets), T).total;
}

extern "C" int adpsgd_init(int32_t K, int64_t P, const int64_t *offsets, int32_t T, const adpsgd_hparams *hp,
                           const adpsgd_buffers *buf, adpsgd_ctx **out) {
    Range range_("adpsgd_init");
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
    if (buf->row_stride < 0 || (buf->row_stride > 0 && buf->row_stride < P))
        return fail(ADPSGD_EINVAL, "row_stride must be 0 or >= P");
    const Plan plan = count_plan(T, offsets);
    // tile indices are 32-bit in the chunk table (P / 4 < 2^32 keeps them far below)
    if (plan.n_tiles >= (int64_t(1) << 31)) return fail(ADPSGD_EINVAL, "too many sync tiles");
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
    build_plan(T, offsets, plan.chunk_tiles, &c->tiles, &c->chunks, &c->chunk_begin);
    c->chunks_are_tiles = plan.chunk_tiles == 1;
    c->hp = *hp;
    c->buf = *buf;
    c->stream = (hipStream_t)buf->stream;
    c->ld = buf->row_stride > 0 ? buf->row_stride : P;
    c->vec = (c->ld % 4) == 0;
    // x and m beyond the 256 MB last-level cache: stream them past the caches
    c->nontemporal = (double)K * (double)P * 8.0 > 256.0 * 1024 * 1024;
    c->sync_nt = c->average_nt = c->nontemporal;   // until timed
    c->rk = round_keys(hp->seed);
    char *ws = (char *)buf->workspace;
    c->d_tiles = (Tile *)(ws + lay.tiles);
    c->d_chunks = (Chunk *)(ws + lay.chunks);
    c->d_chunk_begin = (int32_t *)(ws + lay.chunk_begin);
    c->d_large = (int32_t *)(ws + lay.large);
    c->d_win_begin = (int32_t *)(ws + lay.win_begin);
    c->d_win_partials = (double *)(ws + lay.win_partials);
    if (reduce_windows(T, c->chunk_begin.data(), &c->win_begin) != plan.n_windows) {
        release(c);
        return fail(ADPSGD_EINVAL, "internal: window table disagrees with the workspace plan");
    }
    for (int32_t tau = 0; tau < T; ++tau)
        if (c->chunk_begin[tau + 1] - c->chunk_begin[tau] > kSmallTensorChunks) c->large.push_back(tau);
    c->d_tile_partials = (double *)(ws + lay.tile_partials);
    c->d_chunk_partials = (double *)(ws + lay.chunk_partials);
    c->d_acc = (double *)(ws + lay.acc);
    c->d_sched = (SchedState *)(ws + lay.sched);
    c->d_chunk_seg = (int32_t *)(ws + lay.chunk_seg);
    if (!chunk_segments(c->tiles, plan.n_aligned, &c->chunk_seg)) {
        release(c);
        return fail(ADPSGD_EINVAL, "internal: the tile table does not cover every aligned chunk");
    }
    c->slot_bytes = slot_bytes_for(T);

    auto bail = [&](hipError_t e, const char *what) {
        int rc = hip_fail(e, what);
        std::string msg = g_last_error;
        release(c);
        g_last_error = msg;
        return rc;
    };
    hipError_t e;
    if ((e = hipGetDevice(&c->device)) != hipSuccess) return bail(e, "hipGetDevice");
    // the reduction writes its records straight into coherent pinned memory
    if ((e = hipHostMalloc((void **)&c->h_slots, (size_t)kRing * c->slot_bytes,
                           hipHostMallocMapped | hipHostMallocCoherent)) != hipSuccess)
        return bail(e, "hipHostMalloc");
    if ((e = hipHostGetDevicePointer((void **)&c->d_slots, c->h_slots, 0)) != hipSuccess)
        return bail(e, "hipHostGetDevicePointer");
    if ((e = hipHostMalloc((void **)&c->h_sched, sizeof(SchedState), hipHostMallocDefault)) != hipSuccess)
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
    if ((e = hipMemcpyAsync(c->d_chunk_seg, c->chunk_seg.data(), sizeof(int32_t) * c->chunk_seg.size(),
                            hipMemcpyHostToDevice, c->stream)) != hipSuccess)
        return bail(e, "copy the aligned chunks' tiles");
    if (!c->large.empty() &&
        (e = hipMemcpyAsync(c->d_large, c->large.data(), sizeof(int32_t) * c->large.size(), hipMemcpyHostToDevice,
                            c->stream)) != hipSuccess)
        return bail(e, "copy large-tensor list");
    if (!c->win_begin.empty() &&
        (e = hipMemcpyAsync(c->d_win_begin, c->win_begin.data(), sizeof(int32_t) * c->win_begin.size(),
                            hipMemcpyHostToDevice, c->stream)) != hipSuccess)
        return bail(e, "copy window table");
    if (P > 0) {
        if ((e = launch_init_problem(buf->h, buf->xstar, P, hp->seed, hp->h_lo, hp->h_hi, c->stream)) != hipSuccess)
            return bail(e, "init_problem launch");
        if ((e = zero_rows(c)) != hipSuccess) return bail(e, "zero x and m");
        if ((double)K * (double)P >= kTuneMinElems) {
            if ((e = tune_step_shape(c)) != hipSuccess) return bail(e, "time the local step");
            if ((e = tune_sync_nt(c)) != hipSuccess) return bail(e, "time the fused step + sync");
            if ((e = tune_average(c)) != hipSuccess) return bail(e, "time the separate sync");
            if ((e = zero_rows(c)) != hipSuccess) return bail(e, "zero x and m");
        }
    }
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) return bail(e, "hipStreamSynchronize");
    c->st = adpsgd_state{};
    c->st.p = hp->p_init;
    {
        std::lock_guard<std::mutex> lock(g_live_mu);
        g_live.insert(c);
    }
    *out = c;
    return ok();
}

extern "C" int adpsgd_reset(adpsgd_ctx *c) {
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    HIP_TRY(zero_rows(c));
    c->st = adpsgd_state{};
    c->st.p = c->hp.p_init;
    return ok();
}

extern "C" int adpsgd_local_steps(adpsgd_ctx *c, int32_t n) {
    Range range_("adpsgd_local_steps");
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    if (n < 0) return fail(ADPSGD_EINVAL, "n must be >= 0");
    if (c->st.t + n > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");
    if (int rc = enqueue_steps(c, c->st.t, n)) return rc;
    c->st.t += n;
    c->st.cnt += n;
    // a constant period that switches at p_switch_step does so for the state too
    if (n > 0) c->st.p = period_at(rule_of(&c->hp), c->st.p, c->st.t - 1);
    return ok();
}

static int sync_now(adpsgd_ctx *c, bool fused, double *var_out) {
    Range range_("adpsgd_sync");
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    if (!var_out) return fail(ADPSGD_EINVAL, "var_out is NULL");
    if (fused && c->st.t + 1 > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");
    if (int rc = enqueue_sync(c, fused ? kFused : kAverage, c->st.t, 0, false, nullptr)) return rc;
    HIP_TRY(hipEventSynchronize(c->ring_ev[0]));
    std::memcpy(var_out, slot_host(c, 0) + kSlotHdrBytes, sizeof(double) * c->T);
    if (fused) {
        c->st.p = period_at(rule_of(&c->hp), c->st.p, c->st.t);
        c->st.t += 1;
    }
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

// Algorithm 2 for n_steps steps (adpsgd_run, adpsgd_run_traced).
//
// The host plans each step from its replay of the schedule: a step that ends
// no period whatever the decisions still in flight runs the plain local step;
// any other step runs the sync-tile kernel in a device-decided mode, which
// steps and, iff Algorithm 2's counter (read from the device copy of the
// controller state) says so, averages, followed by the reduction kernel that
// sums the variances and takes Algorithm 2's period decision on the device.  After a decisive
// sync the host waits for its outcome only while the GPU has queued steps
// behind it; otherwise the device decides the next steps itself, so the GPU
// never idles on a host round trip.  Every record is read back in order,
// replayed by the host controller (same rules, same fp64 operations) and
// checked against the device's decision.  A traced run sends every step
// through the reduction.
static int run_impl(adpsgd_ctx *c, int64_t n_steps, adpsgd_sync_rec *log, int64_t log_cap, double *var_log,
                    adpsgd_step_rec *trace, int64_t trace_cap, int64_t *n_syncs) {
    Range range_("adpsgd_run");
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    if (n_steps < 0 || log_cap < 0 || trace_cap < 0) return fail(ADPSGD_EINVAL, "n_steps and capacities must be >= 0");
    if (log_cap > 0 && !log) return fail(ADPSGD_EINVAL, "log is NULL with log_cap > 0");
    if (trace_cap > 0 && !trace) return fail(ADPSGD_EINVAL, "trace is NULL with trace_cap > 0");
    if (c->st.t + n_steps > kMaxCounter) return fail(ADPSGD_EINVAL, "step index would reach 2^32");

    const adpsgd_hparams &hp = c->hp;
    const SchedRule rule = rule_of(&hp);
    const bool traced = trace != nullptr;
    const int64_t t0 = c->st.t, end = t0 + n_steps;

    // The schedule from the host's point of view: exact, or the period known
    // to lie in [lo, hi] (decisions in flight move p by at most one each), or
    // unknown once a step whose sync the host could not predict is in flight.
    struct Plan { bool exact; int64_t cnt; int32_t lo, hi; };
    enum Cls { cPlain, cDue, cUncertain };
    auto advance = [&](Plan &pl, int64_t t) -> Cls {
        if (!pl.exact) return cUncertain;
        pl.cnt += 1;
        pl.lo = period_at(rule, pl.lo, t);
        pl.hi = period_at(rule, pl.hi, t);
        const bool due_lo = sync_due(rule, pl.cnt, pl.lo, t), due_hi = sync_due(rule, pl.cnt, pl.hi, t);
        if (due_lo != due_hi) { pl.exact = false; return cUncertain; }
        if (!due_lo) return cPlain;
        pl.cnt = 0;
        if (sync_decisive(rule, t)) {
            pl.lo = std::max(pl.lo - 1, 1);
            pl.hi = pl.hi < rule.p_max ? pl.hi + 1 : rule.p_max;
        }
        return cDue;
    };

    // A run whose schedule is fixed in advance (constant-period modes) on a
    // small, launch-bound problem replays a captured graph of the whole run.
    const bool graph_mode = c->policy == ADPSGD_LAUNCH_HYBRID && !traced && !c->timing && n_steps > 0 &&
                            n_steps <= kGraphMaxSteps && hp.period_mode != ADPSGD_PERIOD_ADAPTIVE &&
                            (double)c->K * (double)c->P < kGraphMaxElems;
    auto slot_rec = [&](int slot) -> const char * {
        return graph_mode ? c->h_gslots + (size_t)slot * c->slot_bytes : slot_host(c, slot);
    };

    struct Entry { int64_t t; bool dev, uncertain; int slot; int64_t seq; };
    std::deque<Entry> inflight;
    adpsgd_state known = c->st;   // the host controller after every accounted step
    Plan plan{true, known.cnt, known.p, known.p};
    bool dirty = false;
    int64_t launched = t0, n_done = 0, n_slots = 0;
    int n_dev = 0, n_uncertain = 0;
    int status = ADPSGD_OK;

    // Account for the front entry (finished, or a plain step): replay it on the
    // host and check the device's record against the replay.
    auto account = [&](const Entry &e) -> int {
        int32_t due = 0;
        (void)adpsgd_sched_step(&hp, &known, &due);
        if (!e.dev) {
            if (due) return fail(ADPSGD_ESTATE, "internal: a plain step ended a period");
            return ADPSGD_OK;
        }
        SlotHdr hdr;
        std::memcpy(&hdr, slot_rec(e.slot), sizeof hdr);
        const double *var = reinterpret_cast<const double *>(slot_rec(e.slot) + kSlotHdrBytes);
        if (hdr.t != e.t || hdr.due != due)
            return fail(ADPSGD_ESTATE, "device and host schedules disagree at step " + std::to_string(e.t));
        set_timed_kind(c, e.seq, due ? tFused : traced ? tTrace : tStep);
        const double gamma = adpsgd_lr(&hp, e.t);
        if (traced && e.t - t0 < trace_cap)
            trace[e.t - t0] = adpsgd_step_rec{e.t, due, known.p, hdr.S, hdr.GN, gamma};
        if (!due) return ADPSGD_OK;
        const int32_t p_in_force = known.p;
        double margin = std::numeric_limits<double>::quiet_NaN();
        const int rc = adpsgd_sched_on_sync(&hp, &known, e.t, hdr.S, &margin);
        if (n_done < log_cap) {
            log[n_done] = adpsgd_sync_rec{e.t, p_in_force, 0, hdr.S, known.C2, gamma, margin};
            if (var_log) std::memcpy(var_log + (size_t)n_done * c->T, var, sizeof(double) * c->T);
        }
        ++n_done;
        // (a non-finite S still restarted the counter; only p and C2 stay)
        if (rc) return hdr.status == rc ? rc : fail(ADPSGD_ESTATE, "device and host disagree on a non-finite S");
        if (hdr.status != ADPSGD_OK || hdr.p_next != known.p || hdr.C2 != known.C2 || hdr.nC2 != known.nC2)
            return fail(ADPSGD_ESTATE, "device and host controllers disagree at step " + std::to_string(e.t));
        return ADPSGD_OK;
    };
    // Account for every entry at the front that is finished (all of them,
    // waiting, if wait_front: then at least the front one).
    auto drain = [&](bool wait_front) -> int {
        while (!inflight.empty()) {
            const Entry e = inflight.front();
            if (e.dev) {
                hipError_t q;
                if (wait_front) {
                    Range wait_("adpsgd_run: wait for a record");
                    q = hipEventSynchronize(c->ring_ev[e.slot]);
                } else {
                    q = hipEventQuery(c->ring_ev[e.slot]);
                }
                if (q == hipErrorNotReady) break;
                if (q != hipSuccess) return hip_fail(q, "wait for a record");
                wait_front = false;
                --n_dev;
                if (e.uncertain) --n_uncertain;
                dirty = true;
            }
            inflight.pop_front();
            const int rc = account(e);
            // after a failure the remaining records are still accounted for
            // (the steps ran); the first error is the one reported
            if (rc && status == ADPSGD_OK) status = rc;
        }
        return ADPSGD_OK;
    };

    if (n_steps > 0) {
        *c->h_sched = SchedState{known.t, known.cnt, known.nC2, known.C2, known.p, 0};
        HIP_TRY(hipMemcpyAsync(c->d_sched, c->h_sched, sizeof(SchedState), hipMemcpyHostToDevice, c->stream));
    }
    if (graph_mode) {
        // the schedule, from the host controller alone (no decision moves p)
        std::vector<char> due((size_t)n_steps);
        adpsgd_state pl = known;
        int64_t n_sync = 0;
        for (int64_t j = 0; j < n_steps; ++j) {
            int32_t d = 0;
            (void)adpsgd_sched_step(&hp, &pl, &d);
            due[(size_t)j] = (char)d;
            if (d) { pl.cnt = 0; ++n_sync; }
        }
        const int64_t key[7] = {t0, n_steps, known.cnt, known.p, c->step_shape.block, c->step_shape.lds,
                                c->step_shape.row_chunks};
        if (!c->graph_exec || std::memcmp(key, c->graph_key, sizeof key) != 0) {
            Range cap_("adpsgd_run: capture a graph");
            if (int rc = capture_run(c, t0, due, n_sync)) return rc;
            std::memcpy(c->graph_key, key, sizeof key);
            ++c->graph_captures;
        }
        ++c->graph_replays;
        {
            Range replay_("adpsgd_run: graph replay");
            HIP_TRY(hipGraphLaunch(c->graph_exec, c->stream));
            HIP_TRY(hipStreamSynchronize(c->stream));
        }
        int slot = 0;
        for (int64_t j = 0; j < n_steps; ++j) {
            const Entry e{t0 + j, due[(size_t)j] != 0, false, due[(size_t)j] ? slot++ : -1, -1};
            const int rc = account(e);
            if (rc && status == ADPSGD_OK) status = rc;
        }
        c->st = known;
        if (n_syncs) *n_syncs = n_done;
        return status != ADPSGD_OK ? status : ok();
    }
    int hard = ADPSGD_OK;  // a HIP failure: stop at once
    while (hard == ADPSGD_OK) {
        if ((launched - t0) % kPollEvery == 0) {
            if ((hard = drain(false))) break;
            if (c->timing && (hard = harvest(c, false))) break;
        }
        if (launched == end || status != ADPSGD_OK) {
            if (inflight.empty()) break;
            hard = drain(true);
            continue;
        }
        if (dirty) {
            plan = Plan{true, known.cnt, known.p, known.p};
            for (const Entry &e : inflight) (void)advance(plan, e.t);
            dirty = false;
        }
        Plan next = plan;
        Cls cls = advance(next, launched);
        if (traced || c->policy == ADPSGD_LAUNCH_DEVICE) cls = cDue;
        bool wait = (int64_t)inflight.size() >= kMaxInflight || (cls != cPlain && n_dev >= kRing);
        if (cls == cUncertain && !wait) {
            // steps queued on the GPU behind the oldest record not yet read
            int64_t behind = 0;
            bool seen_dev = false;
            for (const Entry &q : inflight) {
                if (seen_dev) ++behind;
                seen_dev = seen_dev || q.dev;
            }
            wait = c->policy == ADPSGD_LAUNCH_HOST || behind >= kQueueToWait || n_uncertain >= kMaxUncertain;
        }
        if (wait) {
            // account for the plain entries at the front and wait for the
            // first device-decided one (with nothing in flight the plan is
            // exact, so there is always something to wait for)
            if (inflight.empty()) { hard = fail(ADPSGD_ESTATE, "internal: nothing in flight to wait for"); break; }
            hard = drain(true);
            continue;
        }
        Entry e{launched, cls != cPlain, cls == cUncertain, -1, -1};
        if (cls == cPlain) {
            hard = enqueue_steps(c, launched, 1);
        } else {
            // a sync the host planned runs the fused kernel; the device's reduction
            // still confirms it and takes the decision
            const int mode = traced ? kDeviceTrace
                                    : (cls == cDue && c->policy != ADPSGD_LAUNCH_DEVICE) ? kFused : kDevice;
            e.slot = (int)(n_slots++ % kRing);
            hard = enqueue_sync(c, mode, launched, e.slot, true, &e.seq);
            ++n_dev;
            if (e.uncertain) ++n_uncertain;
        }
        if (hard) break;
        inflight.push_back(e);
        plan = next;
        ++launched;
    }
    // whatever was enqueued runs to completion and is accounted for
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e == hipSuccess && hard == ADPSGD_OK) hard = drain(true);
    if (e == hipSuccess && hard == ADPSGD_OK)
        while (!inflight.empty() && hard == ADPSGD_OK) hard = drain(true);
    c->st = known;
    if (n_syncs) *n_syncs = n_done;
    if (hard != ADPSGD_OK) return hard;
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    if (status != ADPSGD_OK) return status;
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

extern "C" int adpsgd_set_step_launch(adpsgd_ctx *c, int32_t block, int32_t lds_bytes, int32_t row_chunks) {
    if (int rc = check_ctx(c)) return rc;
    if (block == 0) {
        c->step_shape = c->tuned_shape;
        return ok();
    }
    bool known = false;
    for (int b : kStepBlocks) known = known || b == block;
    if (!known) return fail(ADPSGD_EINVAL, "block must be 0, 64, 128 or 256");
    if (lds_bytes < 0 || lds_bytes > kMaxStepLds) return fail(ADPSGD_EINVAL, "lds_bytes must be in [0, 65536]");
    if (row_chunks < 1 || row_chunks > kMaxRowChunks) return fail(ADPSGD_EINVAL, "row_chunks must be in [1, 4096]");
    c->step_shape = StepShape{block, lds_bytes, row_chunks};
    return ok();   // (a captured run keys on the shape, so it is captured again)
}

extern "C" int adpsgd_get_step_launch(const adpsgd_ctx *c, int32_t *block, int32_t *lds_bytes,
                                      int32_t *row_chunks) {
    if (int rc = check_ctx(c)) return rc;
    if (!block || !lds_bytes || !row_chunks) return fail(ADPSGD_EINVAL, "block, lds_bytes or row_chunks is NULL");
    *block = c->step_shape.block;
    *lds_bytes = c->step_shape.lds;
    *row_chunks = c->step_shape.row_chunks;
    return ok();
}

extern "C" int adpsgd_set_launch_policy(adpsgd_ctx *c, int32_t policy) {
    if (int rc = check_ctx(c)) return rc;
    if (policy != ADPSGD_LAUNCH_HYBRID && policy != ADPSGD_LAUNCH_DEVICE && policy != ADPSGD_LAUNCH_HOST)
        return fail(ADPSGD_EINVAL, "unknown launch policy");
    c->policy = policy;
    return ok();
}

extern "C" int adpsgd_set_timing(adpsgd_ctx *c, int32_t every) {
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    if (every < 0) return fail(ADPSGD_EINVAL, "every must be >= 0");
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (int rc = harvest(c, true)) return rc;
    c->timing = every != 0;
    c->timing_every = every > 0 ? every : 1;
    for (int i = 0; i < tKinds; ++i) { c->t_ms[i] = 0.0; c->t_n[i] = 0; }
    for (auto &n : c->class_count) n = 0;
    c->graph_captures = c->graph_replays = 0;
    return ok();
}

extern "C" int adpsgd_get_timing(adpsgd_ctx *c, adpsgd_timing *out) {
    if (int rc = check_ctx(c)) return rc;
    DeviceScope dev_(c);
    if (!out) return fail(ADPSGD_EINVAL, "out is NULL");
    HIP_TRY(hipStreamSynchronize(c->stream));
    if (int rc = harvest(c, true)) return rc;
    *out = adpsgd_timing{c->t_ms[tStep],  c->t_n[tStep],   c->t_ms[tFused],  c->t_n[tFused],
                         c->t_ms[tAverage], c->t_n[tAverage], c->t_ms[tSegsum], c->t_n[tSegsum],
                         c->t_ms[tTrace], c->t_n[tTrace], c->graph_captures, c->graph_replays};
    return ok();
}

extern "C" int adpsgd_destroy(adpsgd_ctx *c) {
    if (!c) return ok();
    {
        std::lock_guard<std::mutex> lock(g_live_mu);
        if (!g_live.erase(c)) return fail(ADPSGD_EINVAL, "not a live context (destroyed twice?)");
    }
    hipError_t e;
    {
        DeviceScope dev_(c);
        e = hipStreamSynchronize(c->stream);
        release(c);
    }
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
