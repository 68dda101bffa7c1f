// adpsgd_average_noalloc: the separate synchronization (Algorithm 2, lines
// 10-12) for callers that cannot allocate device memory, with no context.
// Its scratch also holds the first tile of every aligned chunk, the block
// index of the sync-tile kernel.
//
// It runs the same sync-tile kernel as adpsgd_average (so the replicas get the
// same bits), but every buffer the kernels need beyond the caller's x lives in
// one file-scope device array, `scratch`: the tensor offsets, the tile table
// (built on the device from the offsets), the fp64 tile partials and the
// per-tensor variances.  The library looks up each device's copy of the array
// once, on the first call on that device, and calls no allocating routine.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>

#include "adpsgd.h"
#include "common.hpp"
#include "kernels.hpp"

namespace adpsgd {
namespace {

// Device memory of the no-allocation entry point, per GPU, for the life of the
// process.  Calls on one GPU share it (and so must not overlap).
constexpr size_t kScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char *g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch array, looked up once
// per device (the array's name is only a host-side stand-in).
int scratch_of_current_device(unsigned char **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(ADPSGD_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return fail(ADPSGD_EDEVICE, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(ADPSGD_EDEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[dev] = static_cast<unsigned char *>(p);
    }
    *out = g_scratch_ptr[dev];
    return ok();
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Tiles of tensor [a, b): cut at multiples of kTileElems (the same rule as the
// context's tile table), so no tile crosses a tensor or spans more than one
// wave's 64 float4 groups.
__host__ __device__ inline int64_t tile_count(int64_t a, int64_t b) {
    return b > a ? (b + kTileElems - 1) / kTileElems - a / kTileElems : 0;
}

// Byte offsets of the scratch regions for T tensors and n_tiles tiles.
struct ScratchLayout {
    size_t offsets, first_tile, tiles, partials, var, chunk_seg, total;
};
ScratchLayout scratch_layout(int32_t T, int64_t n_tiles, int64_t n_chunks) {
    ScratchLayout l;
    l.offsets = 0;
    l.first_tile = align256(l.offsets + sizeof(int64_t) * ((size_t)T + 1));
    l.tiles = align256(l.first_tile + sizeof(int64_t) * ((size_t)T + 1));
    l.partials = align256(l.tiles + sizeof(Tile) * (size_t)n_tiles);
    l.var = align256(l.partials + 2 * sizeof(double) * (size_t)n_tiles);
    l.chunk_seg = align256(l.var + sizeof(double) * (size_t)T);
    l.total = align256(l.chunk_seg + sizeof(int32_t) * ((size_t)n_chunks + 1));
    return l;
}

constexpr int kThreads = 256;

// first_tile[tau] = tiles of the tensors before tau (first_tile[T] = all), one
// block: each thread counts a contiguous run of tensors, then the runs are
// offset by an exclusive scan of the thread totals.
__global__ void __launch_bounds__(kThreads) k_tile_prefix(const int64_t *off, int32_t T, int64_t *first_tile) {
    __shared__ int64_t sums[kThreads];
    const int32_t per = (T + kThreads - 1) / kThreads;
    const int32_t b = (int32_t)threadIdx.x * per, e = b + per < T ? b + per : T;
    int64_t n = 0;
    for (int32_t tau = b; tau < e; ++tau) n += tile_count(off[tau], off[tau + 1]);
    sums[threadIdx.x] = n;
    __syncthreads();
    if (threadIdx.x == 0) {
        int64_t run = 0;
        for (int i = 0; i < kThreads; ++i) {
            const int64_t v = sums[i];
            sums[i] = run;
            run += v;
        }
        first_tile[T] = run;
    }
    __syncthreads();
    int64_t run = sums[threadIdx.x];
    for (int32_t tau = b; tau < e; ++tau) {
        first_tile[tau] = run;
        run += tile_count(off[tau], off[tau + 1]);
    }
}

// One thread per tile: its tensor (the last tau with first_tile[tau] <= i, by
// bisection), then its element range.
__global__ void __launch_bounds__(kThreads) k_build_tiles(const int64_t *off, const int64_t *first_tile, int32_t T,
                                                          int64_t n_tiles, Tile *tiles) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= n_tiles) return;
    int32_t lo = 0, hi = T - 1;
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (first_tile[mid] <= i) lo = mid;
        else hi = mid - 1;
    }
    const int64_t a = off[lo], b = off[lo + 1], j = i - first_tile[lo];
    const int64_t start = j == 0 ? a : (a / kTileElems + j) * kTileElems;
    const int64_t cut = (a / kTileElems + j + 1) * kTileElems;
    tiles[i] = Tile{start, (int32_t)((cut < b ? cut : b) - start), lo};
}

// The first tile of every aligned chunk (the sync-tile kernel's blocks), one
// thread per tile: a tile that starts a chunk's run of tiles records itself.
__global__ void __launch_bounds__(kThreads) k_chunk_tiles(const Tile *tiles, int64_t n_tiles, int64_t n_chunks,
                                                          int32_t *chunk_seg) {
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i == 0) chunk_seg[n_chunks] = (int32_t)n_tiles;
    if (i >= n_tiles) return;
    const int64_t c = tiles[i].start / kTileElems;
    if (i == 0 || tiles[i - 1].start / kTileElems != c) chunk_seg[c] = (int32_t)i;
}

// One block per tensor: the sum of its tile partials (strided over the
// threads, then a fixed-order block sum), divided by K.  Empty tensors get 0.
__global__ void __launch_bounds__(kThreads) k_tensor_var(const int64_t *first_tile, const double *partials,
                                                         int32_t K, double *var) {
    __shared__ double wave[kThreads / 64];
    const int32_t tau = blockIdx.x;
    double s = 0.0;
    for (int64_t i = first_tile[tau] + threadIdx.x; i < first_tile[tau + 1]; i += kThreads) s += partials[2 * i];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if ((threadIdx.x & 63) == 0) wave[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) t += wave[w];
        var[tau] = t / (double)K;
    }
}

}  // namespace
}  // namespace adpsgd

using namespace adpsgd;

extern "C" int adpsgd_average_noalloc(int32_t K, int64_t P, int64_t row_stride, const int64_t *offsets, int32_t T,
                                      float *x, double *var_out, void *stream) {
    if (K < 1 || K > 65536) return fail(ADPSGD_EINVAL, "K must be in [1, 65536]");
    if (P < 0 || (P + 3) / 4 > (int64_t(1) << 32)) return fail(ADPSGD_EINVAL, "P must be >= 0 with P/4 below 2^32");
    if (T < 1 || T > (1 << 24)) return fail(ADPSGD_EINVAL, "T must be in [1, 2^24]");
    if (!offsets || !var_out) return fail(ADPSGD_EINVAL, "offsets and var_out must be non-NULL");
    if (offsets[0] != 0 || offsets[T] != P) return fail(ADPSGD_EINVAL, "need offsets[0] = 0 and offsets[T] = P");
    int64_t n_tiles = 0;
    for (int32_t tau = 0; tau < T; ++tau) {
        if (offsets[tau + 1] < offsets[tau]) return fail(ADPSGD_EINVAL, "tensor_offsets must be non-decreasing");
        n_tiles += tile_count(offsets[tau], offsets[tau + 1]);
    }
    const int64_t ld = row_stride > 0 ? row_stride : P;
    if (row_stride < 0 || (row_stride > 0 && row_stride < P)) return fail(ADPSGD_EINVAL, "row_stride must be 0 or >= P");
    if (P > 0 && (!x || reinterpret_cast<uintptr_t>(x) % 16 != 0))
        return fail(ADPSGD_EINVAL, "x must be non-NULL and 16-byte aligned");
    const int64_t n_chunks = (P + kTileElems - 1) / kTileElems;
    const ScratchLayout lay = scratch_layout(T, n_tiles, n_chunks);
    if (lay.total > kScratchBytes)
        return fail(ADPSGD_EINVAL, "problem needs " + std::to_string(lay.total) + " bytes of scratch; the limit is " +
                                       std::to_string(kScratchBytes) + " (about 2 million sync tiles)");
    unsigned char *base = nullptr;
    if (int rc = scratch_of_current_device(&base)) return rc;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    int64_t *d_off = reinterpret_cast<int64_t *>(base + lay.offsets);
    int64_t *d_first = reinterpret_cast<int64_t *>(base + lay.first_tile);
    Tile *d_tiles = reinterpret_cast<Tile *>(base + lay.tiles);
    int32_t *d_chunk_seg = reinterpret_cast<int32_t *>(base + lay.chunk_seg);
    double *d_part = reinterpret_cast<double *>(base + lay.partials);
    double *d_var = reinterpret_cast<double *>(base + lay.var);

    auto hip_err = [](hipError_t e, const char *what) {
        return fail(ADPSGD_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
    };
    hipError_t e = hipMemcpyAsync(d_off, offsets, sizeof(int64_t) * ((size_t)T + 1), hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return hip_err(e, "copy tensor offsets");
    k_tile_prefix<<<1, kThreads, 0, st>>>(d_off, T, d_first);
    if ((e = hipGetLastError()) != hipSuccess) return hip_err(e, "tile prefix launch");
    if (n_tiles > 0) {
        k_build_tiles<<<(unsigned)((n_tiles + kThreads - 1) / kThreads), kThreads, 0, st>>>(d_off, d_first, T, n_tiles,
                                                                                            d_tiles);
        if ((e = hipGetLastError()) != hipSuccess) return hip_err(e, "tile table launch");
        k_chunk_tiles<<<(unsigned)((n_tiles + kThreads - 1) / kThreads), kThreads, 0, st>>>(d_tiles, n_tiles, n_chunks,
                                                                                            d_chunk_seg);
        if ((e = hipGetLastError()) != hipSuccess) return hip_err(e, "chunk table launch");
        SyncParams sp{};
        sp.s.x = x;
        sp.s.ld = ld;
        sp.s.P = P;
        sp.s.n_groups = (P + 3) / 4;
        sp.s.K = K;
        sp.tiles = d_tiles;
        sp.partials = d_part;
        sp.chunk_seg = d_chunk_seg;
        sp.n_chunks = n_chunks;
        const bool vec = ld % 4 == 0;
        // non-temporal accesses only well beyond the 256 MB last-level cache:
        // between 256 MB and 1 GiB cached accesses measured as fast or faster
        // (18% at K = 32, P = 1.2M), at 8.8 GB 4% slower
        const bool nt = (double)K * (double)P * 8.0 > 1024.0 * 1024 * 1024;
        if ((e = launch_tile_sync(sp, n_tiles, kAverage, false, vec, nt, 0, st)) != hipSuccess)
            return hip_err(e, "sync launch");
    }
    k_tensor_var<<<(unsigned)T, kThreads, 0, st>>>(d_first, d_part, K, d_var);
    if ((e = hipGetLastError()) != hipSuccess) return hip_err(e, "variance launch");
    if ((e = hipMemcpyAsync(var_out, d_var, sizeof(double) * (size_t)T, hipMemcpyDeviceToHost, st)) != hipSuccess)
        return hip_err(e, "copy variances");
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_err(e, "hipStreamSynchronize");
    return ok();
}
