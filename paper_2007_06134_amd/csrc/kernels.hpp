// Launch interface between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "rng.hpp"
#include "schedule.hpp"

namespace adpsgd {

constexpr int kBlock = 256;          // threads per workgroup of the streaming kernels
constexpr int64_t kTileElems = 256;  // sync tiles are cut at multiples of 256 elements,
                                     // so a tile spans at most 64 float4 groups (one wave)
constexpr int32_t kChunkTiles = 1024;  // tiles per first-level chunk of the variance sum
// Chunk partials the final reduction block holds in LDS at once.
constexpr int32_t kFinishWindow = 2048;
// Up to this many tiles (one LDS window), every tile is its own chunk: the tile
// partials are the chunk partials and the first reduction launch is skipped.
// (Above it, the one finishing block reading every tile partial costs more
// than the chunk launch: 22 us against 9 us for the pair at 5080 tiles.)
constexpr int64_t kDirectMaxTiles = kFinishWindow;
constexpr int32_t kSmallTensorChunks = 32;  // larger tensors are summed by a wave, not a thread
// Work-items per launch at most; a grid beyond it is issued in pieces of whole
// 8-block groups, so the blocks keep their XCD order across the pieces.
constexpr int64_t kMaxLaunchItems = int64_t(1) << 31;

// One sync tile: a contiguous element range inside one tensor.
struct Tile {
    int64_t start;
    int32_t len;
    int32_t tensor;
};

// Consecutive tiles of one tensor whose partials are summed together.
struct Chunk {
    int32_t first;
    int32_t count;
    int32_t tensor;
    int32_t pad_;
};

// Everything a local step needs.  Replicas are rows of x and m, ld elements apart.
struct StepParams {
    float *x;
    float *m;
    const float *h;
    const float *xs;
    int64_t ld;        // row stride of x and m in elements (>= P)
    int64_t P;
    int64_t n_groups;  // ceil(P / 4)
    int32_t K;
    uint32_t t;        // step index (Philox counter word 2)
    float sigma, mu, wd, gamma;
    RoundKeys rk;
    // Chunks of one worker's row that an XCD takes one after another before
    // the next worker's (the local step's block order; set by
    // launch_local_step, ignored by the sync kernels).
    int32_t row_chunks;
    int32_t pad_;
    // First block of this launch: a dispatch counts its grid in 32-bit
    // work-items, so larger grids go out as several launches (the launchers
    // below set it; callers leave it 0).
    int64_t block0;
};

struct SyncParams {
    StepParams s;      // x, m, P, K; the step fields are used by the modes with a step
    const Tile *tiles;
    double *partials;  // [2 n_tiles]: per tile, sum of sum_k (xbar - x_k)^2, gradient norm^2
    // The sync-tile kernel (not the loop kernel) takes one block per aligned
    // chunk of kTileElems elements, [c kTileElems, (c + 1) kTileElems) cut at P,
    // whatever tensors it holds: its tiles are chunk_seg[c] .. chunk_seg[c+1]-1
    // (every chunk holds at least one), so a tensor boundary inside a chunk
    // costs no block of its own.
    const int32_t *chunk_seg;  // [n_chunks + 1]
    int64_t n_chunks;          // ceil(P / kTileElems)
    // modes decided on the device: step s.t syncs iff Algorithm 2's counter,
    // read from *sched at block start, says so (the state is written only by
    // the reduction kernel that follows a sync)
    const SchedState *sched;
    SchedRule rule;
};

// Launch shapes of the local step: threads per block (= float4 groups per
// block), an LDS reservation per block, and the block order.  The kernel uses
// no LDS; the reservation only holds a CU to floor(160 KB / lds) resident
// blocks, and fewer waves in flight can stream HBM slightly faster.  The
// blocks of a chunk (block groups of every worker's row) go to one XCD;
// row_chunks = S: an XCD takes S chunks of one worker's row, then the same S
// chunks of the next worker's, so that each row is streamed in longer runs.
// The grid size for n_groups groups, K workers and a shape is
// local_step_blocks.
struct StepShape {
    int block;
    int lds;
    int row_chunks;
};
constexpr int kStepBlocks[] = {64, 128, 256};
constexpr int kMaxStepLds = 64 * 1024;
constexpr int kMaxRowChunks = 4096;
// The shapes adpsgd_init times: the three block sizes with one chunk per row
// run, 64-thread blocks held to 20 per CU (8 KB each), and those with runs of
// 16, 32 and 64 chunks.
constexpr StepShape kStepShapes[] = {{64, 0, 1},     {64, 8192, 1},  {128, 0, 1},   {256, 0, 1},
                                     {64, 8192, 16}, {64, 8192, 32}, {64, 8192, 64}};
int64_t local_step_blocks(int64_t n_groups, int32_t K, const StepShape &shape);
// vec: rows are 16-byte aligned (row stride % 4 == 0) so full groups use
// dwordx4; shape: block one of kStepBlocks, lds in [0, kMaxStepLds],
// row_chunks in [1, kMaxRowChunks] (hipErrorInvalidValue otherwise).
hipError_t launch_local_step(const StepParams &p, bool vec, bool nontemporal, const StepShape &shape,
                             hipStream_t st);
// What a sync-tile kernel does:
//   kAverage      average only (a separate sync);
//   kFused        one local step, then average (a period's last step);
//   kDevice       one local step, then average iff a sync is due (decided on
//                 the device); without a sync nothing is measured;
//   kDeviceTrace  one local step, measure (variance and gradient norm at the
//                 mean), then average iff a sync is due.
enum SyncMode : int { kAverage = 0, kFused = 1, kDevice = 2, kDeviceTrace = 3 };

// Tile partials are pairs (sum of squared deviations, squared gradient norm at
// the mean; the latter only when tracing).  avg_m = true: a sync also averages
// the momentum buffers.  cap > 0 reserves LDS (160 KB per CU on gfx950) so
// that at most cap blocks of the sync-tile kernel are resident per CU; 0: none.
// The loop kernel (K above 64, the separate sync at K = 3) ignores it.
hipError_t launch_tile_sync(const SyncParams &p, int64_t n_tiles, int mode, bool avg_m, bool vec,
                            bool nontemporal, int cap, hipStream_t st);
// chunk_seg (SyncParams) of a tile table: out[c] = the first tile that starts in
// chunk c, out[n_chunks] = n_tiles; false if some chunk holds no tile.
bool chunk_segments(const std::vector<Tile> &tiles, int64_t n_chunks, std::vector<int32_t> *out);
// Waves per block of the sync-tile kernel for K workers in a mode (0 when K
// takes the loop kernel).
int sync_tile_waves(int K, int mode);
constexpr int kLdsPerCU = 160 * 1024;
// Resident waves per CU that the separate sync is timed with at init.
constexpr int kAverageCapWaves = 24;

// Record of one launch of the reduction kernel (one step or one sync).
struct SlotHdr {
    int64_t t;        // the step (or the sync's step)
    int32_t due;      // 1: a sync followed the step
    int32_t p;        // period in force for the step
    int32_t p_next;   // period after the sync's decision
    int32_t status;   // ADPSGD_OK, or ADPSGD_ENONFINITE when S was not finite
    double S;         // sum over tensors of the variances (0 without a reduction)
    double GN;        // sum over tensors of the gradient norms^2
    double C2;        // controller state after the step
    int64_t nC2;
};
constexpr size_t kSlotHdrBytes = 64;
static_assert(sizeof(SlotHdr) <= kSlotHdrBytes, "slot header");

struct ReduceParams {
    const double *tile_partials;  // [2 n_tiles]
    const Chunk *chunks;          // [n_chunks], in tensor order
    const int32_t *chunk_begin;   // [T + 1]: chunks of tensor tau
    double *chunk_partials;       // [2 n_chunks]
    double *acc;                  // [2T] device scratch: per-tensor sums
    const int32_t *large;         // [n_large] tensors of more than kSmallTensorChunks chunks
    int32_t n_chunks, T, K, n_large;
    int32_t chunks_are_tiles;     // 1: chunk_partials is tile_partials (one tile per chunk)
    int32_t block0;               // first block of this launch of the chunk sums (set by launch_reduce)
    // More chunk partials than one LDS window: the tensors are cut into
    // windows (a run of whole small tensors whose chunks fit one window, or one
    // large tensor), reduced by one block each; the finishing block then sums
    // the window partials.  n_windows = 0: one block does everything.
    const int32_t *win_begin;     // [n_windows + 1]: first tensor of each window
    double *win_partials;         // [2 n_windows]: per window, sum of variances, of gradient norms^2
    int32_t n_windows;
    int32_t pad2_;
    double *out;                  // [2T]: variance per tensor, then gradient norm^2 (may be mapped host memory)
    SlotHdr *hdr;                 // (may be mapped host memory)
    SchedState *sched;            // non-null: the step's sync is decided and controlled here
    SchedRule rule;
    int64_t t;                    // the step
    double gamma;                 // its rate in fp64 (Algorithm 2's gamma_t)
    int32_t traced;               // reduce even when no sync is due
};

// Segmented fixed-order sums of the tile partials (chunks, then tensors, then
// over tensors) and, with a schedule, Algorithm 2's period decision on the
// result.
// Windows of tensors (ReduceParams::win_begin) are cut by the host:
int32_t reduce_windows(int32_t T, const int32_t *chunk_begin, std::vector<int32_t> *win_begin);
hipError_t launch_reduce(const ReduceParams &r, hipStream_t st);
// Zero elements [0, P) of each of the K rows of a (rows ld apart); vec: ld is
// a multiple of 4 and a 16-byte aligned, so whole groups take one store.
hipError_t launch_zero_rows(float *a, int64_t ld, int64_t P, int32_t K, bool vec, hipStream_t st);
hipError_t launch_init_problem(float *h, float *xs, int64_t P, uint64_t seed, double h_lo,
                               double h_hi, hipStream_t st);
hipError_t launch_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, uint32_t *out, hipStream_t st);
hipError_t launch_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, float *out, hipStream_t st);

}  // namespace adpsgd
