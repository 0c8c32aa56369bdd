// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) for the injectors, and
// the bit rule of the bit-flip model.
#pragma once

#include "peat_internal.h"

namespace peat {

constexpr uint32_t kPhiloxM0 = 0xD2511F53u, kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u, kPhiloxW1 = 0xBB67AE85u;

// Block number c of stream s under a 64-bit seed: the key is the seed's two
// 32-bit halves, the counter (lo32(c), hi32(c), s, 0).  Each round is two
// 32 x 32 -> 64-bit products (one v_mad_u64_u32 each) and four XORs.
__device__ __forceinline__ void philox(uint64_t c, uint32_t s, uint64_t seed, uint32_t out[4]) {
    uint32_t x0 = (uint32_t)c, x1 = (uint32_t)(c >> 32), x2 = s, x3 = 0;
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)kPhiloxM0 * x0;
        const uint64_t p1 = (uint64_t)kPhiloxM1 * x2;
        // three-input XORs as single v_bitop3_b32 (truth table 0x96)
        const uint32_t y0 = __builtin_amdgcn_bitop3_b32((uint32_t)(p1 >> 32), x1, k0, 0x96);
        const uint32_t y2 = __builtin_amdgcn_bitop3_b32((uint32_t)(p0 >> 32), x3, k1, 0x96);
        x0 = y0;
        x1 = (uint32_t)p1;
        x2 = y2;
        x3 = (uint32_t)p0;
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

// The 64-bit word h (0 or 1) of a block: words 2h (low half) and 2h + 1.
__device__ __forceinline__ uint64_t block_word64(const uint32_t B[4], uint32_t h) {
    return h ? ((uint64_t)B[2] | ((uint64_t)B[3] << 32)) : ((uint64_t)B[0] | ((uint64_t)B[1] << 32));
}

// Bit toggled at element i by the bit-flip model: the j-th lowest set bit of
// the mask, j = floor(y * popcount(mask) / 2^32), y = word 0 of block i of
// stream 2.
__device__ __forceinline__ int chosen_bit(uint64_t seed, uint64_t mask, int popc, uint64_t i) {
    if (popc == 1) return __ffsll((long long)mask) - 1;
    uint32_t C[4];
    philox(i, 2, seed, C);
    uint64_t j = ((uint64_t)C[0] * (uint64_t)popc) >> 32;
    uint64_t m = mask;
    for (uint64_t k = 0; k < j; ++k) m &= m - 1;   // drop the j lowest set bits
    return __ffsll((long long)m) - 1;
}

}  // namespace peat
