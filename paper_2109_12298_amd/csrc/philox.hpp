// Counter-based Gaussian noise shared by the noise kernels.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As
// Easy as 1, 2, 3", SC'11): ten rounds of a 4x32-bit bijection keyed by the
// 64-bit seed.  Element e of parameter tensor `pidx` at step `step` takes word
// e mod 4 of the block with counter (e/4, pidx, step_lo, step_hi); the words
// (w0, w1) and (w2, w3) become normals by the Box-Muller transform.
#pragma once

#include "common.hpp"

namespace dpg {

// Philox4x32 round multipliers and Weyl key increments, as published in the
// SC'11 paper.
constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

struct Block4 {
    uint32_t w[4];
};

__device__ __forceinline__ Block4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo0 = kPhiloxM0 * c0, hi0 = __umulhi(kPhiloxM0, c0);
        const uint32_t lo1 = kPhiloxM1 * c2, hi1 = __umulhi(kPhiloxM1, c2);
        const uint32_t n0 = hi1 ^ c1 ^ k0;
        const uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    Block4 b;
    b.w[0] = c0;
    b.w[1] = c1;
    b.w[2] = c2;
    b.w[3] = c3;
    return b;
}

// Two normals from two words: u1 in (0, 1], u2 in [0, 1), both exact in fp32.
__device__ __forceinline__ void box_muller(uint32_t wa, uint32_t wb, float &za, float &zb)
{
    const float u1 = (float)((wa >> 8) + 1u) * 5.9604644775390625e-8f;  // 2^-24
    const float u2 = (float)(wb >> 8) * 5.9604644775390625e-8f;
    const float r = sqrtf(-2.0f * logf(u1));
    float s, c;
    sincospif(2.0f * u2, &s, &c);
    za = r * c;
    zb = r * s;
}

__device__ __forceinline__ void normals4(i64 q, uint32_t pidx, uint32_t s_lo, uint32_t s_hi,
                                         uint32_t k0, uint32_t k1, float z[4], uint32_t w[4])
{
    const Block4 b = philox4x32_10((uint32_t)q, pidx, s_lo, s_hi, k0, k1);
    box_muller(b.w[0], b.w[1], z[0], z[1]);
    box_muller(b.w[2], b.w[3], z[2], z[3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = b.w[i];
}

}  // namespace dpg
