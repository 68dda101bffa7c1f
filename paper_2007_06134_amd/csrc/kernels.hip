// gfx950 kernels of the ADPSGD hot path.
//
//   k_local_step   one local step of every worker (Algorithm 2's update): a
//                  streaming pass over x and m with the noisy quadratic
//                  gradient generated in registers.
//   k_sync_lds     the synchronization of Algorithm 2 on one aligned chunk
//                  of 256 elements: replica mean, per-element squared deviations
//                  (the parameter variance of Section II-B), broadcast of the
//                  mean; optionally fused behind the period's last local step
//                  so a sync costs no extra pass over HBM.
//   k_sync_loop    the same for K above 64 and the separate sync at K = 3
//                  (other K take k_sync_lds, compiled for powers of two up to
//                  32 or with K as an argument).
//   k_reduce_chunks,  fixed-order sums of the tile partials per chunk, then
//   k_reduce_windows  per tensor (in windows of tensors when there are more
//   k_reduce_finish   chunk partials than one block's LDS holds) and over
//                     tensors, and Algorithm 2's period decision when a run's
//                     schedule lives on the device.
//   k_init_problem, k_zero_rows, k_philox_dump, k_normal_dump: problem data,
//                  row clearing and the raw generator streams.
//
// Work unit: a group of four consecutive elements of one worker's row, moved
// with one dwordx4 load and store and fed by one Philox call.  On MI355X a
// stream of one dwordx4 access per thread over a large grid sustains far more
// HBM bandwidth than threads that each walk many rows, so every thread of the
// local step owns a single (group, worker) pair.  At a sync the waves of a
// tile's block own the K rows and exchange their row sums through LDS.  No
// atomics and fixed reduction orders make results bit-reproducible for a
// given (K, P, offsets).
#include <algorithm>
#include <cmath>

#include "kernels.hpp"

namespace adpsgd {

namespace {

__device__ __forceinline__ f4 fma4(f4 a, f4 b, f4 c) {
    return f4{fmaf(a.x, b.x, c.x), fmaf(a.y, b.y, c.y), fmaf(a.z, b.z, c.z), fmaf(a.w, b.w, c.w)};
}
__device__ __forceinline__ f4 splat(float v) { return f4{v, v, v, v}; }

// Replica rows are touched once per step and never reused before the next
// step, so with a working set beyond the on-chip caches they are streamed with
// non-temporal loads and stores.
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

// Masked scalar access to the lanes of a group that lie in [lo, hi).
__device__ __forceinline__ bool in(int64_t e, int64_t lo, int64_t hi) { return e >= lo && e < hi; }
__device__ __forceinline__ f4 ld4_masked(const float *base, int64_t e0, int64_t lo, int64_t hi) {
    f4 v = splat(0.0f);
    if (in(e0 + 0, lo, hi)) v.x = base[0];
    if (in(e0 + 1, lo, hi)) v.y = base[1];
    if (in(e0 + 2, lo, hi)) v.z = base[2];
    if (in(e0 + 3, lo, hi)) v.w = base[3];
    return v;
}
__device__ __forceinline__ void st4_masked(float *base, f4 v, int64_t e0, int64_t lo, int64_t hi) {
    if (in(e0 + 0, lo, hi)) base[0] = v.x;
    if (in(e0 + 1, lo, hi)) base[1] = v.y;
    if (in(e0 + 2, lo, hi)) base[2] = v.z;
    if (in(e0 + 3, lo, hi)) base[3] = v.w;
}
__device__ __forceinline__ f4 mask4(f4 v, int64_t e0, int64_t lo, int64_t hi) {
    return f4{in(e0 + 0, lo, hi) ? v.x : 0.0f, in(e0 + 1, lo, hi) ? v.y : 0.0f,
              in(e0 + 2, lo, hi) ? v.z : 0.0f, in(e0 + 3, lo, hi) ? v.w : 0.0f};
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

// Sums of a pair of values over the block in a fixed order: wave64 butterfly,
// then the waves in order.  Valid on thread 0.  TWO = false: b is known to be
// zero everywhere (no gradient norm outside tracing) and is not reduced.
struct Pair {
    double a, b;
};
template <int WAVES, bool TWO = true>
__device__ __forceinline__ Pair block_sum2(double a, double b) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        a += __shfl_xor(a, off, 64);
        if (TWO) b += __shfl_xor(b, off, 64);
    }
    if constexpr (WAVES == 1) {
        return Pair{a, TWO ? b : 0.0};
    } else {
        __shared__ double wave_a[WAVES], wave_b[TWO ? WAVES : 1];
        if ((threadIdx.x & 63) == 0) {
            wave_a[threadIdx.x >> 6] = a;
            if (TWO) wave_b[threadIdx.x >> 6] = b;
        }
        __syncthreads();
        Pair total{0.0, 0.0};
        if (threadIdx.x == 0) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) {
                total.a += wave_a[w];
                if (TWO) total.b += wave_b[w];
            }
        }
        return total;
    }
}

// Squared norm of the gradient of F(x) = 1/2 sum h (x - x*)^2 + wd/2 |x|^2 at
// the replica mean, summed over the lanes of one group in [lo, hi).
__device__ __forceinline__ double grad_norm2(const StepParams &a, f4 mean, f4 h, f4 xs, bool full, int64_t e0,
                                             int64_t lo, int64_t hi) {
    const f4 gr = fma4(h, mean - xs, splat(a.wd) * mean);
    f4 g2 = gr * gr;
    if (!full) g2 = mask4(g2, e0, lo, hi);
    return ((double)g2.x + (double)g2.y) + ((double)g2.z + (double)g2.w);
}

// ---------------------------------------------------------------- local step

// Thread = (group g, worker k); a block covers BS consecutive groups (a
// chunk) of one worker's row.  Workgroups go round-robin over the 8 XCDs, and
// the blocks are ordered so that the K blocks of a chunk run on the same XCD:
// h and x* of the chunk come from HBM once and from that XCD's L2 for the
// other K-1 workers.  Within an XCD, S = row_chunks chunks of one worker's
// row come one after another, then the same S chunks of the next worker's
// row, so each row is streamed in runs of S chunks (S = 1: the K workers of
// one chunk in turn).  The best BS, S and LDS reservation depend on the shape
// and the machine; the runtime times a few.
// TAIL: P is not a multiple of 4, so the last group of every row is partial.
template <int BS, bool VEC, bool NT, bool TAIL>
__global__ void __launch_bounds__(BS) k_local_step(StepParams a) {
    const int64_t b = a.block0 + blockIdx.x;
    const int64_t s = b >> 3;                        // position within the XCD
    const int64_t run = s / a.row_chunks;            // (super-chunk, worker)
    const int k = (int)(run % a.K);
    const int64_t chunk = ((run / a.K) * a.row_chunks + (s - run * a.row_chunks)) * 8 + (b & 7);
    const int64_t g = chunk * BS + threadIdx.x;
    if (g >= a.n_groups) return;
    const int64_t e0 = 4 * g;
    float *xr = a.x + (int64_t)k * a.ld + e0;
    float *mr = a.m + (int64_t)k * a.ld + e0;
    if (VEC && (!TAIL || e0 + 4 <= a.P)) {
        f4 x = ld4<NT>(xr), m = ld4<NT>(mr);
        const f4 h = ld4<false>(a.h + e0), xs = ld4<false>(a.xs + e0);
        sgd_update(a, x, m, h, xs, step_noise(a, g, k));
        st4<NT>(xr, x);
        st4<NT>(mr, m);
    } else {
        // the ragged last group of a row, or rows that are not 16-byte aligned
        // (a row stride that is not a multiple of 4): scalar accesses, masked
        // to [0, P)
        f4 x = ld4_masked(xr, e0, 0, a.P), m = ld4_masked(mr, e0, 0, a.P);
        const f4 h = ld4_masked(a.h + e0, e0, 0, a.P), xs = ld4_masked(a.xs + e0, e0, 0, a.P);
        sgd_update(a, x, m, h, xs, step_noise(a, g, k));
        st4_masked(xr, x, e0, 0, a.P);
        st4_masked(mr, m, e0, 0, a.P);
    }
}

// ---------------------------------------------------------------- sync

// Pairwise sum of rows[base .. base+N) at one lane, in a fixed tree order (left
// half, right half).  Exact when all rows are equal and N is a power of two,
// so a sync right after a sync leaves zero variance.  Depth-first evaluation
// keeps only O(log N) partial sums live.
template <int N>
__device__ __forceinline__ f4 tree_sum_lds(const f4 (*rows)[64], int lane, int base) {
    if constexpr (N == 1) {
        return rows[base][lane];
    } else {
        const f4 l = tree_sum_lds<N / 2>(rows, lane, base);
        const f4 r = tree_sum_lds<N - N / 2>(rows, lane, base + N / 2);
        return l + r;
    }
}

// The same tree over a thread's own registers v[base .. base+N).  For N and K
// powers of two, rows R w .. R w + R - 1 form one node of the K-row tree, so
// summing a wave's R rows here and the W node sums through LDS gives the same
// bits as the K-row tree.
template <int N>
__device__ __forceinline__ f4 tree_sum_regs(const f4 *v, int base) {
    if constexpr (N == 1) {
        return v[base];
    } else {
        return tree_sum_regs<N / 2>(v, base) + tree_sum_regs<N - N / 2>(v, base + N / 2);
    }
}

// The pairwise tree over a run-time number (1 to 16) of LDS entries.
__device__ __forceinline__ f4 tree_sum_lds_n(const f4 (*rows)[64], int lane, int n) {
    switch (n) {
    case 1: return tree_sum_lds<1>(rows, lane, 0);
    case 2: return tree_sum_lds<2>(rows, lane, 0);
    case 3: return tree_sum_lds<3>(rows, lane, 0);
    case 4: return tree_sum_lds<4>(rows, lane, 0);
    case 5: return tree_sum_lds<5>(rows, lane, 0);
    case 6: return tree_sum_lds<6>(rows, lane, 0);
    case 7: return tree_sum_lds<7>(rows, lane, 0);
    case 8: return tree_sum_lds<8>(rows, lane, 0);
    case 9: return tree_sum_lds<9>(rows, lane, 0);
    case 10: return tree_sum_lds<10>(rows, lane, 0);
    case 11: return tree_sum_lds<11>(rows, lane, 0);
    case 12: return tree_sum_lds<12>(rows, lane, 0);
    case 13: return tree_sum_lds<13>(rows, lane, 0);
    case 14: return tree_sum_lds<14>(rows, lane, 0);
    case 15: return tree_sum_lds<15>(rows, lane, 0);
    default: return tree_sum_lds<16>(rows, lane, 0);
    }
}

// The replica mean at one lane from the W wave sums in LDS: the pairwise tree
// (WC = W waves for a compiled K, else W from K), so that with R rows per wave
// the mean is the K-row tree when K is a power of two and exact for equal
// replicas; with one row per wave (RD = 1, K = 3) the rows in row order, as
// the loop kernel adds them.
template <int KT, int WC, int RD>
__device__ __forceinline__ f4 lds_mean(const f4 (*rows)[64], int lane, int W, int K) {
    if constexpr (KT > 0) {
        // every compiled K is a power of two: the product by 1/K is the
        // correctly rounded quotient, the same bits as the division, at a
        // fraction of its instructions
        static_assert((KT & (KT - 1)) == 0, "compiled worker counts are powers of two");
        return tree_sum_lds<WC>(rows, lane, 0) * splat(1.0f / (float)KT);
    } else if constexpr (RD > 1) {
        return tree_sum_lds_n(rows, lane, W) / splat((float)K);
    } else {
        // the reads go out four at a time, and the adds run in wave order
        f4 s = rows[0][lane];
#pragma unroll 1
        for (int w0 = 1; w0 < W; w0 += 4) {
            f4 v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = w0 + j < W ? rows[w0 + j][lane] : splat(0.0f);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (w0 + j < W) s = s + v[j];
        }
        return s / splat((float)K);
    }
}

__device__ __forceinline__ f4 shfl_xor4(f4 v, int off) {
    return f4{__shfl_xor(v.x, off, 64), __shfl_xor(v.y, off, 64), __shfl_xor(v.z, off, 64), __shfl_xor(v.w, off, 64)};
}

// The replica mean of every group of a tile from the W wave sums in LDS,
// formed once per group instead of by every wave: wave w takes groups
// w G .. w G + G - 1 (G = 64 / W), its lane l the wave sum l % W of group
// w G + l / W, and a butterfly over those W lanes adds them as the pairwise
// tree does (each pair in the tree's order up to commutation, so the same bits
// as tree_sum_lds<W>).  The means of the first n groups go to out[64]; callers
// put a barrier before (the wave sums) and after (the means).  For a block of
// 16 waves this reads 1/16 of the LDS that every wave reading all 16 sums
// reads (+2 to +3% for the fused sync at K = 16 and 32; no gain at 8 waves).
template <int W, int KT>
__device__ __forceinline__ void group_means(const f4 (*sums)[64], f4 *out, int lane, int w, int n) {
    static_assert((W & (W - 1)) == 0 && (KT & (KT - 1)) == 0, "power-of-two waves and workers");
    constexpr int G = 64 / W;
    const int j = w * G + lane / W, i = lane % W;
    f4 v = j < n ? sums[i][j] : splat(0.0f);
#pragma unroll
    for (int off = 1; off < W; off <<= 1) v = v + shfl_xor4(v, off);
    if (i == 0) out[j] = v * splat(1.0f / (float)KT);
}

// Step s.t of a run whose schedule lives on the device: does a sync follow
// it?  Every thread reads the same state (written only by the reduction
// kernel after a sync), so the answer is uniform over the launch.
__device__ __forceinline__ bool device_due(const SyncParams &p) {
    const SchedState s = *p.sched;
    const int64_t t = (int64_t)p.s.t;
    return sync_due(p.rule, s.cnt + (t - s.t) + 1, period_at(p.rule, s.p, t), t);
}

// One tile (at most 64 groups, one per lane) of one tensor.  Wave w owns the
// rows k = R w .. R w + R - 1 (W waves, R = K / W rows each; see sync_waves).
// Each thread steps its rows (modes with a step), publishes their pairwise sum
// in LDS, reads the W sums of its lane back to form the mean in a fixed order
// (the same bits in every thread, and the same as a tree over all K rows),
// sums its squared deviations and, when a sync is due, writes the mean over
// its rows (with averaged momentum, the momentum rows too).  The
// traced mode also sums the squared gradient norm at the mean (wave 0 counts
// each element once).  partials[2 tile + {0, 1}] = (sum of squared
// deviations, gradient norm^2).  In kDevice a step without a sync stores the
// stepped rows and measures nothing.  Lanes of groups cut by the tile bounds
// use masked scalar accesses.
// Waves per block: one per worker row (at most 16) when the rows are stepped;
// the averaging-only mode does best with two rows per wave (measured +2 to +15%).
// KT = 0: K is a kernel argument (a K up to 64 without a compiled variant,
// with RD = 2 or 4 rows per wave, or K = 3 with one); see lds_mean for the
// order of the mean.
template <int KT, int MODE>
constexpr int sync_waves() {
    if constexpr (KT == 0) return 16;  // the most waves a block of the K-argument kernel has
    else if constexpr (MODE == kAverage && KT >= 2) return KT / 2 < 16 ? KT / 2 : 16;
    else return KT < 16 ? KT : 16;
}

// block_sum2 over a run-time number of waves (at most 16), in the same order.
template <bool TWO = true>
__device__ __forceinline__ Pair block_sum2_waves(double a, double b, int waves) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        a += __shfl_xor(a, off, 64);
        if (TWO) b += __shfl_xor(b, off, 64);
    }
    __shared__ double wave_a[16], wave_b[TWO ? 16 : 1];
    if ((threadIdx.x & 63) == 0) {
        wave_a[threadIdx.x >> 6] = a;
        if (TWO) wave_b[threadIdx.x >> 6] = b;
    }
    __syncthreads();
    Pair total{0.0, 0.0};
    if (threadIdx.x == 0)
        for (int w = 0; w < waves; ++w) {
            total.a += wave_a[w];
            if (TWO) total.b += wave_b[w];
        }
    return total;
}

// RAGGED (K an argument, K not a multiple of RD): the last wave holds fewer
// rows; the missing ones count as zeros in its sum.
template <int KT, bool VEC, bool NT, int MODE, bool AVGM, int RD = 0, bool RAGGED = false>
__global__ void __launch_bounds__((64 * sync_waves<KT, MODE>())) k_sync_lds(SyncParams p) {
    static_assert((KT == 0) == (RD > 0), "RD (rows per wave) is given exactly when K is an argument");
    static_assert(!RAGGED || RD >= 2, "a ragged last wave comes with several rows per wave");
    constexpr int WMAX = sync_waves<KT, MODE>();
    constexpr int R = KT > 0 ? KT / WMAX : RD;
    const int W = KT > 0 ? WMAX : (p.s.K + (RD > 0 ? RD : 1) - 1) / (RD > 0 ? RD : 1);
    constexpr bool STEP = MODE != kAverage;
    constexpr bool GN = MODE == kDeviceTrace;
    // a block of 16 waves forms each group's mean once (group_means)
    constexpr bool SPLIT = KT > 0 && WMAX >= 16;
    // wave w owns rows R w .. R w + R - 1 and publishes their subtree sum
    __shared__ f4 part[WMAX][64];
    __shared__ f4 mpart[AVGM ? WMAX : 1][64];
    __shared__ f4 means[SPLIT ? 64 : 1], mmeans[SPLIT && AVGM ? 64 : 1];
    const StepParams &a = p.s;
    bool bcast = true;  // the host-decided modes always average
    if constexpr (MODE == kDevice || MODE == kDeviceTrace) bcast = device_due(p);
    const bool measure = MODE != kDevice || bcast;
    const bool avg_m = AVGM && bcast;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // the block's aligned chunk and its tiles (one per tensor in it)
    const int64_t c = p.s.block0 + blockIdx.x;
    const int64_t lo = c * kTileElems, hi = lo + kTileElems < a.P ? lo + kTileElems : a.P;
    // The chunk's first tile and the next chunk's.  Blocks of 16 waves read
    // them as scalars here; smaller blocks load them in lanes 0 and 1 (a
    // vector load, so that no wait for them comes ahead of the row loads) and
    // take them after the barrier.  Measured on the fused step + sync: the
    // vector load 2% faster at K = 8, the scalars 0.3-2% faster at K >= 16.
    constexpr bool SEG_VEC = WMAX < 16;
    int32_t s0 = 0, s1 = 0, seg_l = 0;
    if constexpr (SEG_VEC) {
        seg_l = p.chunk_seg[c + (lane & 1)];
    } else {
        s0 = p.chunk_seg[c];
        s1 = p.chunk_seg[c + 1];
    }
    const int64_t g = (lo >> 2) + lane;
    const int64_t e0 = 4 * g;
    const bool active = e0 < hi;
    const bool full = VEC && e0 + 4 <= hi;
    // row R w + r exists (only the last wave's second row can be missing)
    bool has[R];
#pragma unroll
    for (int r = 0; r < R; ++r) has[r] = !RAGGED || R * w + r < a.K;
    f4 xr[R];
    f4 h = splat(0.0f), xs = splat(0.0f);
    if (active) {
        f4 m[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            xr[r] = splat(0.0f);
            m[r] = splat(0.0f);
            if (!has[r]) continue;
            float *xrow = a.x + (int64_t)(R * w + r) * a.ld + e0;
            xr[r] = full ? ld4<NT>(xrow) : ld4_masked(xrow, e0, lo, hi);
            if (STEP || AVGM) {
                float *mrow = a.m + (int64_t)(R * w + r) * a.ld + e0;
                m[r] = full ? ld4<NT>(mrow) : ld4_masked(mrow, e0, lo, hi);
            }
        }
        if (STEP || GN) {
            if (full) { h = ld4<false>(a.h + e0); xs = ld4<false>(a.xs + e0); }
            else { h = ld4_masked(a.h + e0, e0, lo, hi); xs = ld4_masked(a.xs + e0, e0, lo, hi); }
        }
        if (STEP) {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (!has[r]) continue;
                const int k = R * w + r;
                sgd_update(a, xr[r], m[r], h, xs, step_noise(a, g, k));
                if (!avg_m) {
                    float *mrow = a.m + (int64_t)k * a.ld + e0;
                    if (full) st4<NT>(mrow, m[r]); else st4_masked(mrow, m[r], e0, lo, hi);
                }
                if (!bcast) {     // no sync: the replicas keep their new values
                    float *xrow = a.x + (int64_t)k * a.ld + e0;
                    if (full) st4<NT>(xrow, xr[r]); else st4_masked(xrow, xr[r], e0, lo, hi);
                }
            }
        }
        if (measure) {  // (rows a ragged last wave lacks hold zeros)
            part[w][lane] = tree_sum_regs<R>(xr, 0);
            if (AVGM) mpart[w][lane] = tree_sum_regs<R>(m, 0);
        }
    }
    if (!measure) return;  // uniform over the block
    __syncthreads();
    if constexpr (SEG_VEC) {
        s0 = __builtin_amdgcn_readlane(seg_l, 0);
        s1 = __builtin_amdgcn_readlane(seg_l, 1);
    }
    const bool one_tile = s1 - s0 == 1;   // uniform over the block
    if constexpr (SPLIT) {
        // groups of the tile with elements in [lo, hi): the lanes that stored a sum
        const int64_t n64 = (hi - 4 * (lo >> 2) + 3) / 4;
        const int n = n64 < 64 ? (int)n64 : 64;
        group_means<WMAX, KT>(part, means, lane, w, n);
        if (AVGM) group_means<WMAX, KT>(mpart, mmeans, lane, w, n);
        __syncthreads();
    }
    // a chunk of one tile sums its squared deviations per row; a chunk of
    // several keeps them per element (over the rows), to split them by tile
    double acc = 0.0, gn = 0.0;
    double acc4[4] = {0.0, 0.0, 0.0, 0.0}, gn4[4] = {0.0, 0.0, 0.0, 0.0};
    if (active) {
        f4 mean;
        if constexpr (SPLIT) mean = means[lane];
        else mean = lds_mean<KT, WMAX, RD>(part, lane, W, a.K);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            if (!has[r]) continue;
            // squared deviations in fp32 per element, each row's sum in fp64
            const f4 dk = mean - xr[r];
            f4 d2 = dk * dk;
            if (!full) d2 = mask4(d2, e0, lo, hi);
            if (one_tile) {
                acc += ((double)d2.x + (double)d2.y) + ((double)d2.z + (double)d2.w);
            } else {
                acc4[0] += (double)d2.x;
                acc4[1] += (double)d2.y;
                acc4[2] += (double)d2.z;
                acc4[3] += (double)d2.w;
            }
            if (bcast) {
                float *xrow = a.x + (int64_t)(R * w + r) * a.ld + e0;
                if (full) st4<NT>(xrow, mean); else st4_masked(xrow, mean, e0, lo, hi);
            }
        }
        if (avg_m) {
            f4 mmean;
            if constexpr (SPLIT) mmean = mmeans[lane];
            else mmean = lds_mean<KT, WMAX, RD>(mpart, lane, W, a.K);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (!has[r]) continue;
                float *mrow = a.m + (int64_t)(R * w + r) * a.ld + e0;
                if (full) st4<NT>(mrow, mmean); else st4_masked(mrow, mmean, e0, lo, hi);
            }
        }
        if (GN && w == 0) {
            if (one_tile) {
                gn = grad_norm2(a, mean, h, xs, full, e0, lo, hi);
            } else {
                const f4 gr = fma4(h, mean - xs, splat(a.wd) * mean);
                f4 g2 = gr * gr;
                if (!full) g2 = mask4(g2, e0, lo, hi);
                gn4[0] = g2.x;
                gn4[1] = g2.y;
                gn4[2] = g2.z;
                gn4[3] = g2.w;
            }
        }
    }
    if (one_tile) {
        Pair total;
        if constexpr (KT > 0) total = block_sum2<WMAX, GN>(acc, gn);
        else total = block_sum2_waves<GN>(acc, gn, W);
        if (threadIdx.x == 0) {
            p.partials[2 * s0] = total.a;
            p.partials[2 * s0 + 1] = total.b;
        }
        return;
    }
    // several tiles (tensors) in the chunk: one fixed-order block sum each, of
    // the elements in its range
    for (int32_t sgi = s0; sgi < s1; ++sgi) {
        const Tile t = p.tiles[sgi];
        double v = 0.0, gv = 0.0;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (in(e0 + j, t.start, t.start + t.len)) {
                v += acc4[j];
                gv += gn4[j];
            }
        Pair total;
        if constexpr (KT > 0) total = block_sum2<WMAX, GN>(v, gv);
        else total = block_sum2_waves<GN>(v, gv, W);
        if (threadIdx.x == 0) {
            p.partials[2 * sgi] = total.a;
            p.partials[2 * sgi + 1] = total.b;
        }
        __syncthreads();   // the block sum's LDS is used again for the next tile
    }
}

// Any K: one wave per tile, lane = group, the workers walked in a loop.  The
// first pass steps and stores the replicas (modes with a step) and sums them;
// the second re-reads them for the deviations and, when a sync is due, writes
// the mean.  With averaged momentum the first pass also sums the momentum
// buffers and the second writes their mean.  In kDevice a step without a sync
// is the first pass alone.
template <bool VEC, int MODE, bool AVGM>
__global__ void __launch_bounds__(64) k_sync_loop(SyncParams p) {
    constexpr bool STEP = MODE != kAverage;
    constexpr bool GN = MODE == kDeviceTrace;
    const StepParams &a = p.s;
    bool bcast = true;
    if constexpr (MODE == kDevice || MODE == kDeviceTrace) bcast = device_due(p);
    const bool measure = MODE != kDevice || bcast;
    const bool avg_m = AVGM && bcast;
    const int64_t ti = p.s.block0 + blockIdx.x;
    const Tile tile = p.tiles[ti];
    const int64_t lo = tile.start, hi = tile.start + tile.len;
    const int64_t g = (lo >> 2) + threadIdx.x;
    const int64_t e0 = 4 * g;
    double acc = 0.0, gn = 0.0;
    if (e0 < hi) {
        const bool full = VEC && e0 >= lo && e0 + 4 <= hi;
        f4 h = splat(0.0f), xs = splat(0.0f);
        if (STEP || GN) {
            if (full) { h = ld4<false>(a.h + e0); xs = ld4<false>(a.xs + e0); }
            else { h = ld4_masked(a.h + e0, e0, lo, hi); xs = ld4_masked(a.xs + e0, e0, lo, hi); }
        }
        f4 s = splat(0.0f), sm = splat(0.0f);
        for (int k = 0; k < a.K; ++k) {
            float *xrow = a.x + (int64_t)k * a.ld + e0;
            float *mrow = a.m + (int64_t)k * a.ld + e0;
            f4 x = full ? ld4<false>(xrow) : ld4_masked(xrow, e0, lo, hi);
            f4 m = splat(0.0f);
            if (STEP || AVGM) m = full ? ld4<false>(mrow) : ld4_masked(mrow, e0, lo, hi);
            if (STEP) {
                sgd_update(a, x, m, h, xs, step_noise(a, g, k));
                if (full) st4<false>(xrow, x); else st4_masked(xrow, x, e0, lo, hi);
                if (!avg_m) { if (full) st4<false>(mrow, m); else st4_masked(mrow, m, e0, lo, hi); }
            }
            s = (k == 0) ? x : s + x;
            if (AVGM) sm = (k == 0) ? m : sm + m;
        }
        if (measure) {
            const f4 mean = s / splat((float)a.K);
            const f4 mmean = sm / splat((float)a.K);
            for (int k = 0; k < a.K; ++k) {
                float *xrow = a.x + (int64_t)k * a.ld + e0;
                const f4 x = full ? ld4<false>(xrow) : ld4_masked(xrow, e0, lo, hi);
                // squared deviations in fp32 per element, each row's sum in fp64
                const f4 dk = mean - x;
                f4 d2 = dk * dk;
                if (!full) d2 = mask4(d2, e0, lo, hi);
                acc += ((double)d2.x + (double)d2.y) + ((double)d2.z + (double)d2.w);
                if (bcast) { if (full) st4<false>(xrow, mean); else st4_masked(xrow, mean, e0, lo, hi); }
                if (avg_m) {
                    float *mrow = a.m + (int64_t)k * a.ld + e0;
                    if (full) st4<false>(mrow, mmean); else st4_masked(mrow, mmean, e0, lo, hi);
                }
            }
            if (GN) gn = grad_norm2(a, mean, h, xs, full, e0, lo, hi);
        }
    }
    if (!measure) return;
    const Pair total = block_sum2<1, GN>(acc, gn);
    if (threadIdx.x == 0) {
        p.partials[2 * ti] = total.a;
        p.partials[2 * ti + 1] = total.b;
    }
}

// ---------------------------------------------------------------- reduction

__device__ __forceinline__ void write_hdr(const ReduceParams &r, int32_t due, int32_t p, int32_t p_next,
                                          int32_t status, double S, double GN, const SchedState &st) {
    SlotHdr h;
    h.t = r.t;
    h.due = due;
    h.p = p;
    h.p_next = p_next;
    h.status = status;
    h.S = S;
    h.GN = GN;
    h.C2 = st.C2;
    h.nC2 = st.nC2;
    *r.hdr = h;
}

// Is there a sync (or, when tracing, a step) to reduce?  Without a schedule
// the caller decided there is one.  Uniform over a launch: the state changes
// only at the end of k_reduce_finish.
__device__ __forceinline__ bool reduce_due(const ReduceParams &r, int32_t *p_t, SchedState *st) {
    *p_t = 0;
    *st = SchedState{};
    if (!r.sched) return true;
    *st = *r.sched;
    *p_t = period_at(r.rule, st->p, r.t);
    return sync_due(r.rule, st->cnt + (r.t - st->t) + 1, *p_t, r.t);
}

// Level 1, one wave per chunk (kChunksPerBlock chunks per block): the chunk's
// tile partials, summed in a fixed order (strided over the lanes, then a
// butterfly).  A chunk holds at most kChunkTiles = 1024 tiles, 16 per lane;
// problems of thousands of small tensors have as many one-tile chunks, which
// would otherwise cost a block each.
constexpr int kChunksPerBlock = kBlock / 64;
__global__ void __launch_bounds__(kBlock) k_reduce_chunks(ReduceParams r) {
    int32_t p_t;
    SchedState st;
    if (!reduce_due(r, &p_t, &st) && !r.traced) return;
    const int lane = threadIdx.x & 63;
    const int64_t ci = ((int64_t)r.block0 + blockIdx.x) * kChunksPerBlock + (threadIdx.x >> 6);
    if (ci >= r.n_chunks) return;  // whole waves: no block-wide barrier follows
    const Chunk c = r.chunks[ci];
    double a = 0.0, b = 0.0;
    if (c.count <= 64) {  // uniform over the wave: one tile partial per lane at most
        if (lane < c.count) {
            a = r.tile_partials[2 * (int64_t)(c.first + lane)];
            b = r.tile_partials[2 * (int64_t)(c.first + lane) + 1];
        }
    } else {
        // all of a lane's loads are issued before the first add; the sum is
        // then taken in lane-stride order (the zeros of lanes past the chunk
        // leave it unchanged, so both branches give the same bits)
        constexpr int kPerLane = kChunkTiles / 64;
        static_assert(kPerLane * 64 == kChunkTiles, "chunk tiles per lane");
        double va[kPerLane], vb[kPerLane];
#pragma unroll
        for (int j = 0; j < kPerLane; ++j) {
            const int32_t i = lane + 64 * j;
            const bool in_chunk = i < c.count;
            va[j] = in_chunk ? r.tile_partials[2 * (int64_t)(c.first + i)] : 0.0;
            vb[j] = in_chunk ? r.tile_partials[2 * (int64_t)(c.first + i) + 1] : 0.0;
        }
#pragma unroll
        for (int j = 0; j < kPerLane; ++j) {
            a += va[j];
            b += vb[j];
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        a += __shfl_xor(a, off, 64);
        b += __shfl_xor(b, off, 64);
    }
    if (lane == 0) {
        r.chunk_partials[2 * ci] = a;
        r.chunk_partials[2 * ci + 1] = b;
    }
}

constexpr int kFinishThreads = 256;

// Level 2 for problems with more chunk partials than one LDS window: one block
// per window of tensors.  A window of small tensors loads its chunk partials
// (at most kFinishWindow) into LDS and gives each tensor to a thread, which
// adds its chunks in a fixed order (four interleaved partial sums); a window
// holding one large tensor adds its chunks strided over the block.  Writes
// out[tau] = variance (deviation sum / K) and out[T + tau] = gradient norm^2
// for its tensors, and the window's sums in a fixed order to win_partials.
__global__ void __launch_bounds__(kFinishThreads) k_reduce_windows(ReduceParams r) {
    __shared__ double la[kFinishWindow], lb[kFinishWindow];
    int32_t p_t;
    SchedState st;
    if (!reduce_due(r, &p_t, &st) && !r.traced) return;
    const int32_t w = blockIdx.x;
    const int32_t t0 = r.win_begin[w], t1 = r.win_begin[w + 1];
    const int32_t c0 = r.chunk_begin[t0], c1 = r.chunk_begin[t1];
    if (t1 == t0 + 1 && c1 - c0 > kSmallTensorChunks) {  // one large tensor
        double a = 0.0, g = 0.0;
        for (int32_t i = c0 + (int32_t)threadIdx.x; i < c1; i += kFinishThreads) {
            a += r.chunk_partials[2 * (int64_t)i];
            g += r.chunk_partials[2 * (int64_t)i + 1];
        }
        const Pair tot = block_sum2<kFinishThreads / 64>(a, g);
        if (threadIdx.x == 0) {
            const double v = tot.a / (double)r.K;
            r.out[t0] = v;
            r.out[r.T + t0] = tot.b;
            r.win_partials[2 * w] = v;
            r.win_partials[2 * w + 1] = tot.b;
        }
        return;
    }
    const int32_t n = c1 - c0;  // <= kFinishWindow (the host cut the window so)
    for (int32_t i = (int32_t)threadIdx.x; i < n; i += kFinishThreads) {
        la[i] = r.chunk_partials[2 * (int64_t)(c0 + i)];
        lb[i] = r.chunk_partials[2 * (int64_t)(c0 + i) + 1];
    }
    __syncthreads();
    double sa = 0.0, sb = 0.0;
    for (int32_t tau = t0 + (int32_t)threadIdx.x; tau < t1; tau += kFinishThreads) {
        const int32_t b = r.chunk_begin[tau] - c0, e = r.chunk_begin[tau + 1] - c0;
        double a[4] = {0.0, 0.0, 0.0, 0.0}, g[4] = {0.0, 0.0, 0.0, 0.0};
        int32_t i = b;
        for (; i + 4 <= e; i += 4) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                a[j] += la[i + j];
                g[j] += lb[i + j];
            }
        }
        if (i < e) { a[0] += la[i]; g[0] += lb[i]; }
        if (i + 1 < e) { a[1] += la[i + 1]; g[1] += lb[i + 1]; }
        if (i + 2 < e) { a[2] += la[i + 2]; g[2] += lb[i + 2]; }
        const double v = e > b ? ((a[0] + a[1]) + (a[2] + a[3])) / (double)r.K : 0.0;
        const double gn = e > b ? (g[0] + g[1]) + (g[2] + g[3]) : 0.0;
        r.out[tau] = v;
        r.out[r.T + tau] = gn;
        sa += v;
        sb += gn;
    }
    const Pair tot = block_sum2<kFinishThreads / 64>(sa, sb);
    if (threadIdx.x == 0) {
        r.win_partials[2 * w] = tot.a;
        r.win_partials[2 * w + 1] = tot.b;
    }
}

// Level 2 and the decision, one block.  With at most kFinishWindow chunk
// partials (n_windows = 0) it sums the tensors itself, in a fixed order chosen
// by the tensor's chunk count: a tensor of at most kSmallTensorChunks chunks is
// owned by one thread, which adds its chunks from LDS (four interleaved partial
// sums); a larger tensor is owned by one wave, whose lanes add strided chunks
// from LDS before a butterfly; then out[tau] = variance (deviation sum / K),
// out[T + tau] = gradient norm^2, and S and the norm total are block sums.
// Otherwise k_reduce_windows has written out, and S and the norm total are
// block sums of its window partials.  With a schedule, thread 0 then applies
// Algorithm 2's sampling and period decision (the same apply_sync as the host
// controller) and
// writes the new state.  out and the record header are the host's pinned
// record slot, written directly; the header is written in every case.
__global__ void __launch_bounds__(kFinishThreads) k_reduce_finish(ReduceParams r) {
    __shared__ double la[kFinishWindow], lb[kFinishWindow];
    int32_t p_t;
    SchedState st;
    const bool due = reduce_due(r, &p_t, &st);
    if (!due && !r.traced) {
        if (threadIdx.x == 0) write_hdr(r, 0, p_t, p_t, ADPSGD_OK, 0.0, 0.0, st);
        return;
    }
    double sa = 0.0, sb = 0.0;
    if (r.n_windows > 0) {
        // the tensors were reduced by k_reduce_windows: add the window sums
        for (int32_t w = (int32_t)threadIdx.x; w < r.n_windows; w += kFinishThreads) {
            sa += r.win_partials[2 * w];
            sb += r.win_partials[2 * w + 1];
        }
    } else {
        // every chunk partial fits one LDS window (the host cuts the tensors
        // into windows for k_reduce_windows otherwise)
        const int32_t n = r.n_chunks;
        for (int32_t i = (int32_t)threadIdx.x; i < n; i += kFinishThreads) {
            la[i] = r.chunk_partials[2 * (int64_t)i];
            lb[i] = r.chunk_partials[2 * (int64_t)i + 1];
        }
        __syncthreads();
        // small tensors: a thread each
        for (int32_t tau = (int32_t)threadIdx.x; tau < r.T; tau += kFinishThreads) {
            const int32_t b = r.chunk_begin[tau], e = r.chunk_begin[tau + 1];
            if (e - b > kSmallTensorChunks || b >= e) continue;
            double a[4] = {0.0, 0.0, 0.0, 0.0}, g[4] = {0.0, 0.0, 0.0, 0.0};
            int32_t i = b;
            for (; i + 4 <= e; i += 4) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    a[j] += la[i + j];
                    g[j] += lb[i + j];
                }
            }
            if (i < e) { a[0] += la[i]; g[0] += lb[i]; }
            if (i + 1 < e) { a[1] += la[i + 1]; g[1] += lb[i + 1]; }
            if (i + 2 < e) { a[2] += la[i + 2]; g[2] += lb[i + 2]; }
            r.acc[tau] = (a[0] + a[1]) + (a[2] + a[3]);
            r.acc[r.T + tau] = (g[0] + g[1]) + (g[2] + g[3]);
        }
        // large tensors (listed by the host): a wave each, strided lanes, then
        // a butterfly
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        for (int32_t j = wave; j < r.n_large; j += kFinishThreads / 64) {
            const int32_t tau = r.large[j];
            const int32_t cb = r.chunk_begin[tau], ce = r.chunk_begin[tau + 1];
            double a = 0.0, g = 0.0;
            for (int32_t i = cb + lane; i < ce; i += 64) {
                a += la[i];
                g += lb[i];
            }
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                a += __shfl_xor(a, off, 64);
                g += __shfl_xor(g, off, 64);
            }
            if (lane == 0) {
                r.acc[tau] = a;
                r.acc[r.T + tau] = g;
            }
        }
        __syncthreads();  // acc of the large tensors, for their owner threads below
        for (int32_t tau = (int32_t)threadIdx.x; tau < r.T; tau += kFinishThreads) {
            double v = 0.0, g = 0.0;
            if (r.chunk_begin[tau + 1] > r.chunk_begin[tau]) {
                v = r.acc[tau] / (double)r.K;
                g = r.acc[r.T + tau];
            }
            r.out[tau] = v;
            r.out[r.T + tau] = g;
            sa += v;
            sb += g;
        }
    }
    const Pair tot = block_sum2<kFinishThreads / 64>(sa, sb);
    if (threadIdx.x == 0) {
        int32_t status = ADPSGD_OK, p_next = p_t;
        if (r.sched && due) {
            st.p = p_t;
            // a non-finite S restarts the counter and moves nothing else
            if (!apply_sync(r.rule, r.t, r.gamma, tot.a, &st, nullptr)) status = ADPSGD_ENONFINITE;
            st.t = r.t + 1;
            *r.sched = st;
            p_next = st.p;
        }
        write_hdr(r, due ? 1 : 0, p_t, p_next, status, tot.a, tot.b, st);
    }
}

// ---------------------------------------------------------------- problem data

__global__ void __launch_bounds__(kBlock) k_init_problem(float *h, float *xs, int64_t P, RoundKeys rk,
                                                         float log_lo, float log_span, int64_t g0) {
    const int64_t g = g0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t e0 = 4 * g;
    if (e0 >= P) return;
    const u4 rh = philox10(u4{(uint32_t)g, 0u, 0u, TAG_CURVATURE}, rk);
    const f4 hv = f4{expf(fmaf(unif24(rh.x), log_span, log_lo)), expf(fmaf(unif24(rh.y), log_span, log_lo)),
                     expf(fmaf(unif24(rh.z), log_span, log_lo)), expf(fmaf(unif24(rh.w), log_span, log_lo))};
    const f4 xv = normals4(philox10(u4{(uint32_t)g, 0u, 0u, TAG_OPTIMUM}, rk));
    st4_masked(h + e0, hv, e0, 0, P);
    st4_masked(xs + e0, xv, e0, 0, P);
}

// Thread = one float4 group of one row: j = k * groups_per_row + g.
template <bool VEC>
__global__ void __launch_bounds__(kBlock) k_zero_rows(float *a, int64_t ld, int64_t P, int64_t groups_per_row,
                                                      int64_t j0, int64_t n) {
    const int64_t j = j0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= n) return;
    const int64_t k = j / groups_per_row, e0 = 4 * (j - k * groups_per_row);
    float *row = a + k * ld + e0;
    if (VEC && e0 + 4 <= P) st4<false>(row, splat(0.0f));
    else st4_masked(row, splat(0.0f), e0, 0, P);
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

// Blocks of `threads` work-items that one launch may hold (a multiple of 8).
constexpr int64_t piece_blocks(int threads) { return (kMaxLaunchItems / threads) & ~int64_t(7); }

// launch(first block, block count) over [0, n_blocks) in pieces of at most
// piece_blocks(threads) blocks.
template <class F>
hipError_t in_pieces(int64_t n_blocks, int threads, F launch) {
    const int64_t step = piece_blocks(threads);
    for (int64_t b0 = 0; b0 < n_blocks; b0 += step) {
        launch(b0, (unsigned)std::min(step, n_blocks - b0));
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// The same for the element-wise kernels: launch(first group, group count) in
// pieces of whole blocks of kBlock groups.
template <class F>
hipError_t groups_in_pieces(int64_t n, F launch) {
    const int64_t step = piece_blocks(kBlock) * kBlock;
    for (int64_t g0 = 0; g0 < n; g0 += step) {
        const int64_t m = std::min(step, n - g0);
        launch(g0, m, blocks_for(m));
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Dynamic LDS that holds a CU to `cap` resident blocks of a kernel with
// static_lds bytes of its own: each block then takes kLdsPerCU / cap bytes
// (rounded down to 512).  0 for no cap, or when the kernel's own LDS already
// allows no more.
inline int cap_lds(int cap, size_t static_lds) {
    if (cap <= 0) return 0;
    const size_t per_block = (size_t)(kLdsPerCU / cap) & ~size_t(511);
    return per_block > static_lds ? (int)(per_block - static_lds) : 0;
}

template <class Kern>
size_t static_lds_of(Kern kern) {
    hipFuncAttributes fa;
    return hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kern)) == hipSuccess ? fa.sharedSizeBytes : 0;
}

// Does the K-argument sync-tile kernel take K in this mode (else the loop
// kernel does)?  Two rows per wave up to K = 32 and four up to 64 (the last
// wave of a K that is not a multiple holds fewer): a CU holds at most two
// blocks of 9-16 waves, and several rows per wave keep more bytes in flight.
// K = 3 is the exception: one row per wave in the modes with a step, and the
// loop kernel for the separate sync (76% of peak, against 58% and 48% for
// three one-row or two two-row waves); both add the rows in row order, so the
// replicas keep the same bits.
constexpr bool any_k_kernel(int K, int mode) {
    if (K == 3) return mode != kAverage;
    return K > 0 && K <= 64;
}
constexpr int any_k_rows(int K) { return K == 3 ? 1 : (K <= 32 ? 2 : 4); }
constexpr int any_k_waves(int K) { return (K + any_k_rows(K) - 1) / any_k_rows(K); }

template <int KT, bool VEC, bool NT, int MODE, bool AVGM, int RD, bool RAGGED>
hipError_t sync_variant(const SyncParams &p, int64_t, int cap, hipStream_t st) {
    const int threads = KT > 0 ? 64 * sync_waves<KT, MODE>() : 64 * any_k_waves(p.s.K);
    int lds = 0;
    if (cap > 0) {   // (the attribute query only when it is needed: not under graph capture)
        static const size_t own = static_lds_of(k_sync_lds<KT, VEC, NT, MODE, AVGM, RD, RAGGED>);
        lds = cap_lds(cap, own);
    }
    return in_pieces(p.n_chunks, threads, [&](int64_t b0, unsigned nb) {   // a block per chunk
        SyncParams q = p;
        q.s.block0 = b0;
        k_sync_lds<KT, VEC, NT, MODE, AVGM, RD, RAGGED><<<dim3(nb), dim3(threads), lds, st>>>(q);
    });
}

template <int KT, int MODE, bool AVGM, int RD, bool RAGGED>
hipError_t sync_dispatch(const SyncParams &p, int64_t n_tiles, bool vec, bool nt, int cap, hipStream_t st) {
    if (vec && nt) return sync_variant<KT, true, true, MODE, AVGM, RD, RAGGED>(p, n_tiles, cap, st);
    if (vec) return sync_variant<KT, true, false, MODE, AVGM, RD, RAGGED>(p, n_tiles, cap, st);
    return sync_variant<KT, false, false, MODE, AVGM, RD, RAGGED>(p, n_tiles, cap, st);
}

template <int KT, int RD = 0, bool RAGGED = false>
hipError_t sync_dispatch(const SyncParams &p, int64_t n_tiles, int mode, bool avg_m, bool vec, bool nt, int cap,
                         hipStream_t st) {
    switch (mode) {
    case kAverage: return avg_m ? sync_dispatch<KT, kAverage, true, RD, RAGGED>(p, n_tiles, vec, nt, cap, st)
                                : sync_dispatch<KT, kAverage, false, RD, RAGGED>(p, n_tiles, vec, nt, cap, st);
    case kFused: return avg_m ? sync_dispatch<KT, kFused, true, RD, RAGGED>(p, n_tiles, vec, nt, cap, st)
                              : sync_dispatch<KT, kFused, false, RD, RAGGED>(p, n_tiles, vec, nt, cap, st);
    case kDevice: return avg_m ? sync_dispatch<KT, kDevice, true, RD, RAGGED>(p, n_tiles, vec, nt, cap, st)
                               : sync_dispatch<KT, kDevice, false, RD, RAGGED>(p, n_tiles, vec, nt, cap, st);
    default: return avg_m ? sync_dispatch<KT, kDeviceTrace, true, RD, RAGGED>(p, n_tiles, vec, nt, cap, st)
                          : sync_dispatch<KT, kDeviceTrace, false, RD, RAGGED>(p, n_tiles, vec, nt, cap, st);
    }
}

template <int MODE, bool AVGM>
hipError_t loop_dispatch(const SyncParams &p, int64_t n_tiles, bool vec, hipStream_t st) {
    return in_pieces(n_tiles, 64, [&](int64_t b0, unsigned nb) {
        SyncParams q = p;
        q.s.block0 = b0;
        if (vec) k_sync_loop<true, MODE, AVGM><<<dim3(nb), dim3(64), 0, st>>>(q);
        else k_sync_loop<false, MODE, AVGM><<<dim3(nb), dim3(64), 0, st>>>(q);
    });
}

hipError_t loop_dispatch(const SyncParams &p, int64_t n_tiles, int mode, bool avg_m, bool vec, hipStream_t st) {
    switch (mode) {
    case kAverage: return avg_m ? loop_dispatch<kAverage, true>(p, n_tiles, vec, st)
                                : loop_dispatch<kAverage, false>(p, n_tiles, vec, st);
    case kFused: return avg_m ? loop_dispatch<kFused, true>(p, n_tiles, vec, st)
                              : loop_dispatch<kFused, false>(p, n_tiles, vec, st);
    case kDevice: return avg_m ? loop_dispatch<kDevice, true>(p, n_tiles, vec, st)
                               : loop_dispatch<kDevice, false>(p, n_tiles, vec, st);
    default: return avg_m ? loop_dispatch<kDeviceTrace, true>(p, n_tiles, vec, st)
                          : loop_dispatch<kDeviceTrace, false>(p, n_tiles, vec, st);
    }
}

}  // namespace

int64_t local_step_blocks(int64_t n_groups, int32_t K, const StepShape &shape) {
    const int64_t chunks = (n_groups + shape.block - 1) / shape.block;
    const int64_t per = 8 * (int64_t)shape.row_chunks;  // chunks of one super-chunk
    return ((chunks + per - 1) / per) * per * (int64_t)K;
}

template <int BS>
hipError_t local_step_bs(const StepParams &p, bool vec, bool nt, const StepShape &shape, hipStream_t st) {
    // shape.lds: dynamic LDS per block that the kernel never touches (an occupancy cap)
    const int lds = shape.lds;
    return in_pieces(local_step_blocks(p.n_groups, p.K, shape), BS, [&](int64_t b0, unsigned nb) {
        StepParams q = p;
        q.row_chunks = shape.row_chunks;
        q.block0 = b0;
        const bool tail = (p.P & 3) != 0;
        if (vec && nt && tail) k_local_step<BS, true, true, true><<<dim3(nb), dim3(BS), lds, st>>>(q);
        else if (vec && nt) k_local_step<BS, true, true, false><<<dim3(nb), dim3(BS), lds, st>>>(q);
        else if (vec && tail) k_local_step<BS, true, false, true><<<dim3(nb), dim3(BS), lds, st>>>(q);
        else if (vec) k_local_step<BS, true, false, false><<<dim3(nb), dim3(BS), lds, st>>>(q);
        else k_local_step<BS, false, false, false><<<dim3(nb), dim3(BS), lds, st>>>(q);
    });
}

hipError_t launch_local_step(const StepParams &p, bool vec, bool nt, const StepShape &shape, hipStream_t st) {
    if (shape.lds < 0 || shape.lds > kMaxStepLds) return hipErrorInvalidValue;
    if (shape.row_chunks < 1 || shape.row_chunks > kMaxRowChunks) return hipErrorInvalidValue;
    if (p.n_groups <= 0) return hipSuccess;
    switch (shape.block) {
    case 64: return local_step_bs<64>(p, vec, nt, shape, st);
    case 128: return local_step_bs<128>(p, vec, nt, shape, st);
    case 256: return local_step_bs<256>(p, vec, nt, shape, st);
    default: return hipErrorInvalidValue;
    }
}

int sync_tile_waves(int K, int mode) {
    const bool avg = mode == kAverage;
    switch (K) {
    case 1: return avg ? sync_waves<1, kAverage>() : sync_waves<1, kFused>();
    case 2: return avg ? sync_waves<2, kAverage>() : sync_waves<2, kFused>();
    case 4: return avg ? sync_waves<4, kAverage>() : sync_waves<4, kFused>();
    case 8: return avg ? sync_waves<8, kAverage>() : sync_waves<8, kFused>();
    case 16: return avg ? sync_waves<16, kAverage>() : sync_waves<16, kFused>();
    case 32: return avg ? sync_waves<32, kAverage>() : sync_waves<32, kFused>();
    default: return any_k_kernel(K, mode) ? any_k_waves(K) : 0;
    }
}

hipError_t launch_tile_sync(const SyncParams &p, int64_t n_tiles, int mode, bool avg_m, bool vec, bool nt,
                            int cap, hipStream_t st) {
    if (n_tiles <= 0) return hipSuccess;
    switch (p.s.K) {
    case 1: return sync_dispatch<1>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    case 2: return sync_dispatch<2>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    case 4: return sync_dispatch<4>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    case 8: return sync_dispatch<8>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    case 16: return sync_dispatch<16>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    case 32: return sync_dispatch<32>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
    default:
        if (!any_k_kernel(p.s.K, mode)) return loop_dispatch(p, n_tiles, mode, avg_m, vec, st);
        switch (any_k_rows(p.s.K)) {
        case 1: return sync_dispatch<0, 1, false>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
        case 2:
            return p.s.K % 2 == 0 ? sync_dispatch<0, 2, false>(p, n_tiles, mode, avg_m, vec, nt, cap, st)
                                  : sync_dispatch<0, 2, true>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
        default:
            return p.s.K % 4 == 0 ? sync_dispatch<0, 4, false>(p, n_tiles, mode, avg_m, vec, nt, cap, st)
                                  : sync_dispatch<0, 4, true>(p, n_tiles, mode, avg_m, vec, nt, cap, st);
        }
    }
}

bool chunk_segments(const std::vector<Tile> &tiles, int64_t n_chunks, std::vector<int32_t> *out) {
    out->assign((size_t)n_chunks + 1, -1);
    int64_t prev = -1;
    for (size_t sgi = 0; sgi < tiles.size(); ++sgi) {
        const int64_t c = tiles[sgi].start / kTileElems;
        if (c < 0 || c >= n_chunks || c < prev) return false;
        if (c != prev) (*out)[(size_t)c] = (int32_t)sgi;
        prev = c;
    }
    (*out)[(size_t)n_chunks] = (int32_t)tiles.size();
    for (int64_t c = 0; c < n_chunks; ++c)
        if ((*out)[(size_t)c] < 0) return false;
    return true;
}

hipError_t launch_reduce(const ReduceParams &r, hipStream_t st) {
    if (r.n_chunks > 0 && !r.chunks_are_tiles) {
        const int64_t blocks = (r.n_chunks + kChunksPerBlock - 1) / kChunksPerBlock;
        const hipError_t e = in_pieces(blocks, kBlock, [&](int64_t b0, unsigned nb) {
            ReduceParams q = r;
            q.block0 = (int32_t)b0;
            k_reduce_chunks<<<dim3(nb), dim3(kBlock), 0, st>>>(q);
        });
        if (e != hipSuccess) return e;
    }
    if (r.n_windows > 0) {
        k_reduce_windows<<<dim3((unsigned)r.n_windows), dim3(kFinishThreads), 0, st>>>(r);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    k_reduce_finish<<<dim3(1), dim3(kFinishThreads), 0, st>>>(r);
    return hipGetLastError();
}

hipError_t launch_init_problem(float *h, float *xs, int64_t P, uint64_t seed, double h_lo, double h_hi,
                               hipStream_t st) {
    if (P <= 0) return hipSuccess;
    const double llo = std::log(h_lo), lhi = std::log(h_hi);
    const RoundKeys rk = round_keys(seed);
    return groups_in_pieces((P + 3) / 4, [&](int64_t g0, int64_t, unsigned nb) {
        k_init_problem<<<dim3(nb), dim3(kBlock), 0, st>>>(h, xs, P, rk, (float)llo, (float)(lhi - llo), g0);
    });
}

hipError_t launch_zero_rows(float *a, int64_t ld, int64_t P, int32_t K, bool vec, hipStream_t st) {
    if (P <= 0 || K <= 0) return hipSuccess;
    const int64_t gpr = (P + 3) / 4, n = gpr * K;
    return groups_in_pieces(n, [&](int64_t j0, int64_t, unsigned nb) {
        if (vec) k_zero_rows<true><<<dim3(nb), dim3(kBlock), 0, st>>>(a, ld, P, gpr, j0, n);
        else k_zero_rows<false><<<dim3(nb), dim3(kBlock), 0, st>>>(a, ld, P, gpr, j0, n);
    });
}

hipError_t launch_philox_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n,
                              uint32_t *out, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const RoundKeys rk = round_keys(seed);
    return groups_in_pieces(n, [&](int64_t j0, int64_t m, unsigned nb) {
        k_philox_dump<<<dim3(nb), dim3(kBlock), 0, st>>>(rk, c1, c2, c3, g0 + j0, m, out + 4 * j0);
    });
}

hipError_t launch_normal_dump(uint64_t seed, uint32_t c1, uint32_t c2, uint32_t c3, int64_t g0, int64_t n,
                              float *out, hipStream_t st) {
    if (n <= 0) return hipSuccess;
    const RoundKeys rk = round_keys(seed);
    return groups_in_pieces(n, [&](int64_t j0, int64_t m, unsigned nb) {
        k_normal_dump<<<dim3(nb), dim3(kBlock), 0, st>>>(rk, c1, c2, c3, g0 + j0, m, out + 4 * j0);
    });
}

}  // namespace adpsgd
