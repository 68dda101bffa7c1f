// Launch interface between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rng.hpp"

namespace adpsgd {

constexpr int kBlock = 256;          // threads per workgroup: four wave64s
constexpr int64_t kTileElems = 4096; // max elements per sync tile (multiple of 4)

// One sync tile: a contiguous element range inside one tensor.
struct Tile {
    int64_t start;
    int32_t len;
    int32_t tensor;
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
    double *partials;  // [n_tiles] sum over the tile of sum_k (xbar - x_k)^2
};

// vec: rows are 16-byte aligned (P % 4 == 0) so full groups use dwordx4.
hipError_t launch_local_step(const StepParams &p, bool vec, bool nontemporal, hipStream_t st);
// fused = true: the local step and the sync in one pass.
hipError_t launch_tile_sync(const SyncParams &p, int64_t n_tiles, bool fused, bool vec,
                            bool nontemporal, hipStream_t st);
// var[tau] = (sum of partials of tau's tiles) / K, tiles of tau are
// [tile_begin[tau], tile_begin[tau+1]).
hipError_t launch_segsum(const int32_t *tile_begin, const double *partials, double *var,
                         int32_t T, int32_t K, hipStream_t st);
hipError_t launch_init_problem(float *h, float *xs, int64_t P, uint64_t seed, double h_lo,
                               double h_hi, hipStream_t st);
hipError_t launch_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, uint32_t *out, hipStream_t st);
hipError_t launch_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0,
                              int64_t n, float *out, hipStream_t st);

}  // namespace adpsgd
