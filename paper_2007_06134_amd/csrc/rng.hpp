// Counter-based noise for the local steps, on the device.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy
// as 1, 2, 3", SC'11): ten rounds of two 32x32->64 multiplies by fixed odd
// multipliers, with the high halves xored into the other two counter words
// and the round key; the key advances by two Weyl constants per round.  The
// key is the 64-bit seed split into two words; it is uniform across a launch,
// so the ten round keys live in scalar registers.
//
// Gaussian noise by Box-Muller (1958) on the 24 high bits of each word.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace adpsgd {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

struct RoundKeys {
    uint32_t lo[10];
    uint32_t hi[10];
};

__host__ __device__ inline RoundKeys round_keys(uint64_t seed) {
    RoundKeys rk;
    uint32_t a = (uint32_t)seed, b = (uint32_t)(seed >> 32);
    for (int r = 0; r < 10; ++r) {
        rk.lo[r] = a;
        rk.hi[r] = b;
        a += 0x9E3779B9u;  // Weyl increments of the published key schedule
        b += 0xBB67AE85u;
    }
    return rk;
}

// Counter words (c.x, c.y, c.z, c.w) -> 4 random words.
__device__ __forceinline__ u4 philox10(u4 c, const RoundKeys &rk) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t prod_a = (uint64_t)c.x * 0xD2511F53u;
        const uint64_t prod_b = (uint64_t)c.z * 0xCD9E8D57u;
        const uint32_t y = (uint32_t)prod_b;
        const uint32_t w = (uint32_t)prod_a;
        c.x = (uint32_t)(prod_b >> 32) ^ c.y ^ rk.lo[r];
        c.z = (uint32_t)(prod_a >> 32) ^ c.w ^ rk.hi[r];
        c.y = y;
        c.w = w;
    }
    return c;
}

// Two Box-Muller normals from two words: radius sqrt(-2 ln u1) with
// u1 = (hi24(a) + 1) 2^-24 in (0, 1] (never 0, so the log is finite) and angle
// 2 pi u2 with u2 = hi24(b) 2^-24.  Both uniforms are exact in fp32.
// The gfx950 transcendental instructions fit this form directly: v_log_f32 is
// log2 (u1 >= 2^-24, so no denormal inputs), and v_sin_f32 / v_cos_f32 take
// the angle in turns, so sin(2 pi u2) needs no range reduction.  This skips
// the special-case handling of the libm-style wrappers, which this input range
// never needs.
__device__ __forceinline__ void box_muller2(uint32_t a, uint32_t b, float &z0, float &z1) {
    const float u1 = (float)((a >> 8) + 1u) * 0x1p-24f;
    const float u2 = (float)(b >> 8) * 0x1p-24f;
    constexpr float kMinus2Ln2 = -1.38629436111989061883f;   // -2 ln 2
    const float radius = __builtin_amdgcn_sqrtf(kMinus2Ln2 * __builtin_amdgcn_logf(u1));
    z0 = radius * __builtin_amdgcn_cosf(u2);
    z1 = radius * __builtin_amdgcn_sinf(u2);
}

__device__ __forceinline__ f4 normals4(u4 r) {
    float z0, z1, z2, z3;
    box_muller2(r.x, r.y, z0, z1);
    box_muller2(r.z, r.w, z2, z3);
    return f4{z0, z1, z2, z3};
}

// Uniform in [0, 1) from the 24 high bits.
__device__ __forceinline__ float unif24(uint32_t r) { return (float)(r >> 8) * 0x1p-24f; }

// Counter layout: (group g = i/4, worker k, step t, tag).
enum : uint32_t { TAG_NOISE = 0u, TAG_CURVATURE = 1u, TAG_OPTIMUM = 2u };

}  // namespace adpsgd
