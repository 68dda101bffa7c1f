// gfx950 kernels of the ADPSGD hot path.
//
//   k_local_step   one local step of every worker (Algorithm 2, lines 5-7):
//                  a streaming pass over x and m, with the per-worker noisy
//                  quadratic gradient generated in registers.
//   k_tile_sync    the synchronization (Algorithm 2, lines 10-12) per tile of
//                  one tensor: replica mean, per-element squared deviations
//                  (the parameter variance of Section II-B), broadcast of the
//                  mean; optionally fused behind the period's last local step
//                  so the sync costs no extra pass over HBM.
//   k_segsum       fixed-order sum of the tile partials of each tensor.
//
// Work unit: a group of four consecutive elements (one dwordx4 per row and one
// Philox call per worker).  Every kernel is HBM-bound streaming work: no
// atomics, no data-dependent control flow, and a fixed reduction order, so
// results are bit-reproducible for a given (K, P, offsets).
#include <cmath>

#include "kernels.hpp"

namespace adpsgd {

namespace {

__device__ __forceinline__ f4 fma4(f4 a, f4 b, f4 c) {
    return f4{fmaf(a.x, b.x, c.x), fmaf(a.y, b.y, c.y), fmaf(a.z, b.z, c.z), fmaf(a.w, b.w, c.w)};
}
__device__ __forceinline__ f4 splat(float v) { return f4{v, v, v, v}; }

template <bool NT>
__device__ __forceinline__ f4 ld4(const float *p) {
    if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p));
    else return *reinterpret_cast<const f4 *>(p);
}
template <bool NT>
__device__ __forceinline__ void st4(float *p, f4 v) {
    if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<f4 *>(p));
    else *reinterpret_cast<f4 *>(p) = v;
}

// Masked scalar access to the lanes of group g that lie in [lo, hi).
__device__ __forceinline__ f4 ld4_masked(const float *base, int64_t e0, int64_t lo, int64_t hi) {
    f4 v = splat(0.0f);
    if (e0 + 0 >= lo && e0 + 0 < hi) v.x = base[0];
    if (e0 + 1 >= lo && e0 + 1 < hi) v.y = base[1];
    if (e0 + 2 >= lo && e0 + 2 < hi) v.z = base[2];
    if (e0 + 3 >= lo && e0 + 3 < hi) v.w = base[3];
    return v;
}
__device__ __forceinline__ void st4_masked(float *base, f4 v, int64_t e0, int64_t lo, int64_t hi) {
    if (e0 + 0 >= lo && e0 + 0 < hi) base[0] = v.x;
    if (e0 + 1 >= lo && e0 + 1 < hi) base[1] = v.y;
    if (e0 + 2 >= lo && e0 + 2 < hi) base[2] = v.z;
    if (e0 + 3 >= lo && e0 + 3 < hi) base[3] = v.w;
}
__device__ __forceinline__ f4 mask4(f4 v, int64_t e0, int64_t lo, int64_t hi) {
    return f4{(e0 + 0 >= lo && e0 + 0 < hi) ? v.x : 0.0f, (e0 + 1 >= lo && e0 + 1 < hi) ? v.y : 0.0f,
              (e0 + 2 >= lo && e0 + 2 < hi) ? v.z : 0.0f, (e0 + 3 >= lo && e0 + 3 < hi) ? v.w : 0.0f};
}

// Gradient noise of worker k at step t for group g.
__device__ __forceinline__ f4 step_noise(const StepParams &a, int64_t g, int k) {
    return normals4(philox10(u4{(uint32_t)g, (uint32_t)k, a.t, TAG_NOISE}, a.rk));
}

// Momentum SGD on the noisy quadratic, PyTorch-SGD form with coupled weight
// decay: d = h (x - x*) + sigma z + wd x;  m = mu m + d;  x = x - gamma m.
// Explicit fmaf fixes the rounding so every kernel computes identical bits.
__device__ __forceinline__ void sgd_update(const StepParams &a, f4 &x, f4 &m, f4 h, f4 xs, f4 z) {
    const f4 d = fma4(h, x - xs, fma4(splat(a.sigma), z, splat(a.wd) * x));
    m = fma4(splat(a.mu), m, d);
    x = fma4(splat(-a.gamma), m, x);
}

// Wave64 butterfly, then the four waves in a fixed order.  Valid on thread 0.
__device__ __forceinline__ double block_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    __shared__ double wave_sum[kBlock / 64];
    if ((threadIdx.x & 63) == 0) wave_sum[threadIdx.x >> 6] = v;
    __syncthreads();
    double total = 0.0;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) total += wave_sum[w];
    }
    return total;
}

// ---------------------------------------------------------------- local step

// One thread per group, the worker loop inside: h and x* are loaded once and
// reused by all K workers; each worker's row costs one dwordx4 load and store
// of x and of m.  KT > 0 fixes K at compile time (fully unrolled).
template <int KT, bool VEC, bool NT>
__global__ void __launch_bounds__(kBlock) k_local_step(StepParams a) {
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (g >= a.n_groups) return;
    const int K = KT > 0 ? KT : a.K;
    const int64_t e0 = 4 * g;
    if constexpr (VEC) {
        const f4 h = ld4<false>(a.h + e0);
        const f4 xs = ld4<false>(a.xs + e0);
        auto one_worker = [&](int k) {
            float *xr = a.x + (int64_t)k * a.P + e0;
            float *mr = a.m + (int64_t)k * a.P + e0;
            f4 x = ld4<NT>(xr), m = ld4<NT>(mr);
            sgd_update(a, x, m, h, xs, step_noise(a, g, k));
            st4<NT>(xr, x);
            st4<NT>(mr, m);
        };
        if constexpr (KT > 0) {
#pragma unroll
            for (int k = 0; k < KT; ++k) one_worker(k);
        } else {
            for (int k = 0; k < K; ++k) one_worker(k);
        }
    } else {
        // P not a multiple of 4: rows are not 16-byte aligned, so every access
        // is a scalar one, masked to [0, P) in the ragged last group
        const f4 h = ld4_masked(a.h + e0, e0, 0, a.P);
        const f4 xs = ld4_masked(a.xs + e0, e0, 0, a.P);
        for (int k = 0; k < K; ++k) {
            float *xr = a.x + (int64_t)k * a.P + e0;
            float *mr = a.m + (int64_t)k * a.P + e0;
            f4 x = ld4_masked(xr, e0, 0, a.P), m = ld4_masked(mr, e0, 0, a.P);
            sgd_update(a, x, m, h, xs, step_noise(a, g, k));
            st4_masked(xr, x, e0, 0, a.P);
            st4_masked(mr, m, e0, 0, a.P);
        }
    }
}

// ---------------------------------------------------------------- sync

// Mean of the replicas: a pairwise sum in a fixed tree order (exact when all
// replicas are equal and K is a power of two, so a sync right after a sync
// leaves zero variance), then one correctly rounded division.
template <int N>
__device__ __forceinline__ f4 tree_sum(const f4 *v) {
    if constexpr (N == 1) return v[0];
    else return tree_sum<N / 2>(v) + tree_sum<N - N / 2>(v + N / 2);
}
template <int KT>
__device__ __forceinline__ f4 replica_mean(const f4 (&xr)[KT]) {
    return tree_sum<KT>(xr) / splat((float)KT);
}

// Tile of one tensor, groups [start/4, ceil(end/4)).  Groups cut by the tile
// bounds (tensor boundaries that are not multiples of 4, or an unaligned P)
// go through masked scalar accesses; the arithmetic per element is the same.
template <int KT, bool VEC, bool NT, bool FUSED>
__global__ void __launch_bounds__(kBlock) k_tile_sync(SyncParams p) {
    const StepParams &a = p.s;
    const Tile tile = p.tiles[blockIdx.x];
    const int64_t lo = tile.start, hi = tile.start + tile.len;
    const int64_t g_end = (hi + 3) >> 2;
    double acc = 0.0;
    for (int64_t g = (lo >> 2) + threadIdx.x; g < g_end; g += kBlock) {
        const int64_t e0 = 4 * g;
        const bool full = VEC && e0 >= lo && e0 + 4 <= hi;
        f4 h = splat(0.0f), xs = splat(0.0f);
        if (FUSED) {
            if (full) { h = ld4<false>(a.h + e0); xs = ld4<false>(a.xs + e0); }
            else { h = ld4_masked(a.h + e0, e0, lo, hi); xs = ld4_masked(a.xs + e0, e0, lo, hi); }
        }
        f4 dev2 = splat(0.0f);
        if constexpr (KT > 0) {
            f4 xr[KT];
#pragma unroll
            for (int k = 0; k < KT; ++k) {
                float *xrow = a.x + (int64_t)k * a.P + e0;
                xr[k] = full ? ld4<NT>(xrow) : ld4_masked(xrow, e0, lo, hi);
                if (FUSED) {
                    float *mrow = a.m + (int64_t)k * a.P + e0;
                    f4 m = full ? ld4<NT>(mrow) : ld4_masked(mrow, e0, lo, hi);
                    sgd_update(a, xr[k], m, h, xs, step_noise(a, g, k));
                    if (full) st4<NT>(mrow, m); else st4_masked(mrow, m, e0, lo, hi);
                }
            }
            const f4 mean = replica_mean<KT>(xr);
#pragma unroll
            for (int k = 0; k < KT; ++k) {
                const f4 dk = mean - xr[k];
                dev2 = fma4(dk, dk, dev2);
                float *xrow = a.x + (int64_t)k * a.P + e0;
                if (full) st4<NT>(xrow, mean); else st4_masked(xrow, mean, e0, lo, hi);
            }
        } else {
            // K not fixed at compile time: sum in a first pass (stepping and
            // storing the new replicas if fused), re-read them in a second.
            f4 s = splat(0.0f);
            for (int k = 0; k < a.K; ++k) {
                float *xrow = a.x + (int64_t)k * a.P + e0;
                f4 x = full ? ld4<NT>(xrow) : ld4_masked(xrow, e0, lo, hi);
                if (FUSED) {
                    float *mrow = a.m + (int64_t)k * a.P + e0;
                    f4 m = full ? ld4<NT>(mrow) : ld4_masked(mrow, e0, lo, hi);
                    sgd_update(a, x, m, h, xs, step_noise(a, g, k));
                    if (full) { st4<NT>(mrow, m); st4<NT>(xrow, x); }
                    else { st4_masked(mrow, m, e0, lo, hi); st4_masked(xrow, x, e0, lo, hi); }
                }
                s = (k == 0) ? x : s + x;
            }
            const f4 mean = s / splat((float)a.K);
            for (int k = 0; k < a.K; ++k) {
                float *xrow = a.x + (int64_t)k * a.P + e0;
                const f4 x = full ? ld4<NT>(xrow) : ld4_masked(xrow, e0, lo, hi);
                const f4 dk = mean - x;
                dev2 = fma4(dk, dk, dev2);
                if (full) st4<NT>(xrow, mean); else st4_masked(xrow, mean, e0, lo, hi);
            }
        }
        if (!full) dev2 = mask4(dev2, e0, lo, hi);
        acc += ((double)dev2.x + (double)dev2.y) + ((double)dev2.z + (double)dev2.w);
    }
    const double total = block_sum(acc);
    if (threadIdx.x == 0) p.partials[blockIdx.x] = total;
}

__global__ void __launch_bounds__(kBlock) k_segsum(const int32_t *tile_begin, const double *partials,
                                                   double *var, int32_t K) {
    const int32_t tau = blockIdx.x;
    const int32_t b = tile_begin[tau], e = tile_begin[tau + 1];
    double acc = 0.0;
    for (int32_t i = b + (int32_t)threadIdx.x; i < e; i += kBlock) acc += partials[i];
    const double total = block_sum(acc);
    if (threadIdx.x == 0) var[tau] = total / (double)K;
}

// ---------------------------------------------------------------- problem data

__global__ void __launch_bounds__(kBlock) k_init_problem(float *h, float *xs, int64_t P, RoundKeys rk,
                                                         float log_lo, float log_span) {
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t e0 = 4 * g;
    if (e0 >= P) return;
    const u4 rh = philox10(u4{(uint32_t)g, 0u, 0u, TAG_CURVATURE}, rk);
    const f4 hv = f4{expf(fmaf(unif24(rh.x), log_span, log_lo)), expf(fmaf(unif24(rh.y), log_span, log_lo)),
                     expf(fmaf(unif24(rh.z), log_span, log_lo)), expf(fmaf(unif24(rh.w), log_span, log_lo))};
    const f4 xv = normals4(philox10(u4{(uint32_t)g, 0u, 0u, TAG_OPTIMUM}, rk));
    st4_masked(h + e0, hv, e0, 0, P);
    st4_masked(xs + e0, xv, e0, 0, P);
}

__global__ void __launch_bounds__(kBlock) k_philox_dump(RoundKeys rk, uint32_t c1, uint32_t c2, uint32_t c3,
                                                        int64_t g0, int64_t n, uint32_t *out) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= n) return;
    const u4 r = philox10(u4{(uint32_t)(g0 + j), c1, c2, c3}, rk);
    *reinterpret_cast<u4 *>(out + 4 * j) = r;
}

__global__ void __launch_bounds__(kBlock) k_normal_dump(RoundKeys rk, uint32_t c1, uint32_t c2, uint32_t c3,
                                                        int64_t g0, int64_t n, float *out) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= n) return;
    const f4 z = normals4(philox10(u4{(uint32_t)(g0 + j), c1, c2, c3}, rk));
    *reinterpret_cast<f4 *>(out + 4 * j) = z;
}

inline unsigned blocks_for(int64_t n) { return (unsigned)((n + kBlock - 1) / kBlock); }

template <int KT>
hipError_t step_dispatch(const StepParams &p, bool vec, bool nt, hipStream_t st) {
    const dim3 grid(blocks_for(p.n_groups)), block(kBlock);
    if (vec && nt) k_local_step<KT, true, true><<<grid, block, 0, st>>>(p);
    else if (vec) k_local_step<KT, true, false><<<grid, block, 0, st>>>(p);
    else k_local_step<KT, false, false><<<grid, block, 0, st>>>(p);
    return hipGetLastError();
}

template <int KT>
hipError_t sync_dispatch(const SyncParams &p, int64_t n_tiles, bool fused, bool vec, bool nt,
                         hipStream_t st) {
    const dim3 grid((unsigned)n_tiles), block(kBlock);
    if (fused) {
        if (vec && nt) k_tile_sync<KT, true, true, true><<<grid, block, 0, st>>>(p);
        else if (vec) k_tile_sync<KT, true, false, true><<<grid, block, 0, st>>>(p);
        else k_tile_sync<KT, false, false, true><<<grid, block, 0, st>>>(p);
    } else {
        if (vec && nt) k_tile_sync<KT, true, true, false><<<grid, block, 0, st>>>(p);
        else if (vec) k_tile_sync<KT, true, false, false><<<grid, block, 0, st>>>(p);
        else k_tile_sync<KT, false, false, false><<<grid, block, 0, st>>>(p);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_local_step(const StepParams &p, bool vec, bool nt, hipStream_t st) {
    if (p.n_groups <= 0) return hipSuccess;
    switch (p.K) {
    case 1: return step_dispatch<1>(p, vec, nt, st);
    case 2: return step_dispatch<2>(p, vec, nt, st);
    case 4: return step_dispatch<4>(p, vec, nt, st);
    case 8: return step_dispatch<8>(p, vec, nt, st);
    case 16: return step_dispatch<16>(p, vec, nt, st);
    case 32: return step_dispatch<32>(p, vec, nt, st);
    default: return step_dispatch<0>(p, vec, nt, st);
    }
}

hipError_t launch_tile_sync(const SyncParams &p, int64_t n_tiles, bool fused, bool vec, bool nt,
                            hipStream_t st) {
    if (n_tiles <= 0) return hipSuccess;
    switch (p.s.K) {
    case 1: return sync_dispatch<1>(p, n_tiles, fused, vec, nt, st);
    case 2: return sync_dispatch<2>(p, n_tiles, fused, vec, nt, st);
    case 4: return sync_dispatch<4>(p, n_tiles, fused, vec, nt, st);
    case 8: return sync_dispatch<8>(p, n_tiles, fused, vec, nt, st);
    case 16: return sync_dispatch<16>(p, n_tiles, fused, vec, nt, st);
    case 32: return sync_dispatch<32>(p, n_tiles, fused, vec, nt, st);
    default: return sync_dispatch<0>(p, n_tiles, fused, vec, nt, st);
    }
}

hipError_t launch_segsum(const int32_t *tile_begin, const double *partials, double *var, int32_t T,
                         int32_t K, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    k_segsum<<<dim3((unsigned)T), dim3(kBlock), 0, st>>>(tile_begin, partials, var, K);
    return hipGetLastError();
}

hipError_t launch_init_problem(float *h, float *xs, int64_t P, uint64_t seed, double h_lo, double h_hi,
                               hipStream_t st) {
    if (P <= 0) return hipSuccess;
    const double llo = std::log(h_lo), lhi = std::log(h_hi);
    k_init_problem<<<dim3(blocks_for((P + 3) / 4)), dim3(kBlock), 0, st>>>(
        h, xs, P, round_keys(seed), (float)llo, (float)(lhi - llo));
    return hipGetLastError();
}

hipError_t launch_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n,
                              uint32_t *out, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    k_philox_dump<<<dim3(blocks_for(n)), dim3(kBlock), 0, st>>>(round_keys(seed), c1, c2, c3, g0, n, out);
    return hipGetLastError();
}

hipError_t launch_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n,
                              float *out, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    k_normal_dump<<<dim3(blocks_for(n)), dim3(kBlock), 0, st>>>(round_keys(seed), c1, c2, c3, g0, n, out);
    return hipGetLastError();
}

}  // namespace adpsgd
