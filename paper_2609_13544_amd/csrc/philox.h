// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11) for the injectors, and
// the bit rule of the bit-flip model.
#pragma once

#include "peat_internal.h"

namespace peat {

constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ULL, kPhiloxM1 = 0xCA5A826395121157ULL;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ULL, kPhiloxW1 = 0xBB67AE8584CAA73BULL;

// 64 x 64 -> 128-bit product from four 32 x 32 -> 64 multiply-adds.
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t b, uint64_t &lo, uint64_t &hi) {
    const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32);
    const uint32_t b0 = (uint32_t)b, b1 = (uint32_t)(b >> 32);
    const uint64_t p00 = (uint64_t)a0 * b0;
    const uint64_t t = (uint64_t)a1 * b0 + (p00 >> 32);
    const uint64_t u = (uint64_t)a0 * b1 + (uint32_t)t;
    lo = (u << 32) | (uint32_t)p00;
    hi = (uint64_t)a1 * b1 + (t >> 32) + (u >> 32);
}

// The block at counter (c0, c1, 0, 0) under the key (key, 0).
__device__ __forceinline__ void philox(uint64_t c0, uint64_t c1, uint64_t key, uint64_t out[4]) {
    uint64_t x0 = c0, x1 = c1, x2 = 0, x3 = 0;
    uint64_t k0 = key, k1 = 0;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t lo0, hi0, lo1, hi1;
        mulhilo64(kPhiloxM0, x0, lo0, hi0);
        mulhilo64(kPhiloxM1, x2, lo1, hi1);
        const uint64_t y0 = hi1 ^ x1 ^ k0;
        const uint64_t y2 = hi0 ^ x3 ^ k1;
        x0 = y0;
        x1 = lo1;
        x2 = y2;
        x3 = lo0;
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

// Bit toggled at element i by the bit-flip model: the j-th lowest set bit of
// the mask, j = floor(hi32(y) * popcount(mask) / 2^32), y = word 0 of the
// block at counter (i, 2, 0, 0).
__device__ __forceinline__ int chosen_bit(uint64_t seed, uint64_t mask, int popc, uint64_t i) {
    if (popc == 1) return __ffsll((long long)mask) - 1;
    uint64_t C[4];
    philox(i, 2, seed, C);
    uint64_t j = ((C[0] >> 32) * (uint64_t)popc) >> 32;
    uint64_t m = mask;
    for (uint64_t k = 0; k < j; ++k) m &= m - 1;   // drop the j lowest set bits
    return __ffsll((long long)m) - 1;
}

}  // namespace peat
