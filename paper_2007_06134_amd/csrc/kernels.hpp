// Launch interface between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rng.hpp"

namespace adpsgd {

constexpr int kBlock = 256;          // threads per workgroup of the streaming kernels
constexpr int64_t kTileElems = 256;  // sync tiles are cut at multiples of 256 elements,
                                     // so a tile spans at most 64 float4 groups (one wave)
constexpr int32_t kChunkTiles = 1024;  // tiles per first-level chunk of the variance sum

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
};

// Everything a local step needs.  Replicas are rows of x/m with stride P.
struct StepParams {
    float *x;
    float *m;
    const float *h;
    const float *xs;
    int64_t P;
    int64_t n_groups;  // ceil(P / 4)
    int32_t K;
    uint32_t t;        // step index (Philox counter word 2)
    float sigma, mu, wd, gamma;
    RoundKeys rk;
};

struct SyncParams {
    StepParams s;      // x, m, P, K; the step fields are used only when fused
    const Tile *tiles;
    double *partials;  // [2 n_tiles]: per tile, sum of sum_k (xbar - x_k)^2, gradient norm^2
};

// Grid size of the local step for n_groups groups and K workers.
int64_t local_step_blocks(int64_t n_groups, int32_t K);
// vec: rows are 16-byte aligned (P % 4 == 0) so full groups use dwordx4.
hipError_t launch_local_step(const StepParams &p, bool vec, bool nontemporal, hipStream_t st);
// What a sync-tile kernel does: average only (a separate sync), one local step
// then average (a period's last step), one local step and only measure
// (tracing: variance and gradient norm at the mean, replicas kept), or one
// local step, measure and average (a traced period's last step).
enum SyncMode : int { kAverage = 0, kFused = 1, kTrace = 2, kFusedTrace = 3 };

// Tile partials are pairs (sum of squared deviations, squared gradient norm at
// the mean; the latter only in the tracing modes).  avg_m = true: a sync also
// averages the momentum buffers.
hipError_t launch_tile_sync(const SyncParams &p, int64_t n_tiles, int mode, bool avg_m, bool vec,
                            bool nontemporal, hipStream_t st);
// chunk_partials[c] = sums of the tile partials of chunk c; then, over tau's
// chunks [chunk_begin[tau], chunk_begin[tau+1]): out[tau] = variance
// (deviation sum / K) and out[T + tau] = squared gradient norm.
hipError_t launch_segsum(const Chunk *chunks, int64_t n_chunks, const int32_t *chunk_begin,
                         const double *tile_partials, double *chunk_partials, double *out, int32_t T,
                         int32_t K, hipStream_t st);
hipError_t launch_init_problem(float *h, float *xs, int64_t P, uint64_t seed, double h_lo,
                               double h_hi, hipStream_t st);
hipError_t launch_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, uint32_t *out, hipStream_t st);
hipError_t launch_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, float *out, hipStream_t st);

}  // namespace adpsgd
