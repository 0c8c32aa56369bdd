// Random-bit-flip injector for gfx950 (the RBF error model of Section II-B,
// used by Inject() in Algorithms 1 and 2).
//
// Element i of a tensor flips iff its 64-bit uniform U_i is below
// T = floor(rate * 2^64) (every element when rate >= 1).  U_i is built from
// Philox4x64-10 (Salmon et al., SC'11) keyed by (seed, 0):
//   top byte   = byte (i mod 32) of the block at counter (i/32, 0, 0, 0)
//   low 56 bits = word (i mod 4) of the block at counter (i/4, 1, 0, 0)
// A flipped element toggles the j-th lowest set bit of the mask with
// j = floor(hi32(y) * popcount(mask) / 2^32), y = word 0 at (i, 2, 0, 0).
//
// For T < 2^56 an element can only flip when its top byte is 0, so each lane
// draws one block per 32 elements and evaluates the low bits only for the
// (1 in 256) elements whose top byte is zero.  The tensor is read and written
// only at flipped elements.
#include "peat_internal.h"

namespace peat {
namespace {

constexpr uint64_t kM0 = 0xD2E7470EE14C6C93ULL, kM1 = 0xCA5A826395121157ULL;
constexpr uint64_t kW0 = 0x9E3779B97F4A7C15ULL, kW1 = 0xBB67AE8584CAA73BULL;

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

__device__ __forceinline__ void philox(uint64_t c0, uint64_t c1, uint64_t key, uint64_t out[4]) {
    uint64_t x0 = c0, x1 = c1, x2 = 0, x3 = 0;
    uint64_t k0 = key, k1 = 0;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        uint64_t lo0, hi0, lo1, hi1;
        mulhilo64(kM0, x0, lo0, hi0);
        mulhilo64(kM1, x2, lo1, hi1);
        const uint64_t y0 = hi1 ^ x1 ^ k0;
        const uint64_t y2 = hi0 ^ x3 ^ k1;
        x0 = y0;
        x1 = lo1;
        x2 = y2;
        x3 = lo0;
        k0 += kW0;
        k1 += kW1;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

__device__ __forceinline__ int chosen_bit(const InjDesc &d, uint64_t i) {
    if (d.popc == 1) return __ffsll((long long)d.mask) - 1;
    uint64_t C[4];
    philox(i, 2, d.seed, C);
    uint64_t j = ((C[0] >> 32) * (uint64_t)d.popc) >> 32;
    uint64_t m = d.mask;
    for (uint64_t k = 0; k < j; ++k) m &= m - 1;   // drop the j lowest set bits
    return __ffsll((long long)m) - 1;
}

__device__ __forceinline__ void flip(const InjDesc &d, uint64_t i) {
    const int b = chosen_bit(d, i);
    if (d.dtype == PEAT_F32) {
        uint32_t *p = static_cast<uint32_t *>(d.x) + i;
        *p ^= 1u << b;
    } else {
        uint16_t *p = static_cast<uint16_t *>(d.x) + i;
        *p = (uint16_t)(*p ^ (1u << b));
    }
}

constexpr int kQCap = 64 + 32 * 64;   // per-wave queue: < 64 left over + one append of 32 per lane

// Low 56 bits of U_i for a queued candidate (its top byte is 0, so U_i is
// just these bits): flip the element when they are below T.
__device__ __forceinline__ uint32_t settle_candidate(const InjDesc &d, uint64_t i) {
    uint64_t B[4];
    philox(i >> 2, 1, d.seed, B);
    const uint64_t low = B[i & 3] & ((uint64_t(1) << 56) - 1);
    if (low < d.T) {
        flip(d, i);
        return 1;
    }
    return 0;
}

__global__ void __launch_bounds__(kBlock) inject_kernel(InjParams P) {
    const int64_t seg = blockIdx.x;
    const int item = P.seg_item[seg];
    const InjDesc d = P.descs[item];
    const uint64_t s0 = (uint64_t)(seg - d.first_seg) << kInjSegLog2;   // first element
    const uint64_t n = (uint64_t)d.n;
    const uint64_t len = (n - s0) < (uint64_t(1) << kInjSegLog2) ? (n - s0) : (uint64_t(1) << kInjSegLog2);
    const uint32_t ngroups = (uint32_t)((len + 31) / 32);
    const uint64_t q0 = s0 >> 5;
    const uint64_t T = d.T;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t flips = 0;

    if (!d.all && T < (uint64_t(1) << 56)) {
        // An element can flip only if the top byte of U_i is 0.  Each lane
        // draws one block per group of 32 elements; the zero-byte elements
        // go to a per-wave queue (segment-relative offsets) whose entries
        // are settled 64 at a time, one per lane.
        __shared__ uint32_t queue[kBlock / 64][kQCap];
        uint32_t qn = 0;                                   // wave-uniform
        const uint32_t iters = (ngroups + kBlock - 1) / kBlock;
        for (uint32_t k = 0; k < iters; ++k) {
            const uint32_t g = k * kBlock + threadIdx.x;
            uint32_t cand = 0;
            if (g < ngroups) {
                uint64_t A[4];
                philox(q0 + g, 0, d.seed, A);
                // exact zero-byte mask of each 32-bit half: bit 7 of a byte
                // is set iff the byte is zero; one multiply gathers bits
                // 7, 15, 23, 31 into bits 28..31 (the other partial products
                // land on distinct lower bits, so nothing carries)
#pragma unroll
                for (int w = 0; w < 8; ++w) {
                    const uint32_t v = (uint32_t)(A[w >> 1] >> (32 * (w & 1)));
                    const uint32_t z = ~(((v & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | v | 0x7F7F7F7Fu);
                    cand |= ((z * 0x00204081u) >> 28) << (4 * w);
                }
                const uint64_t rest = len - ((uint64_t)g << 5);
                if (rest < 32) cand &= (1u << (uint32_t)rest) - 1u;   // ragged end
            }
            // append this iteration's candidates, one per lane per round
            while (true) {
                const bool has = cand != 0;
                const uint64_t m = __ballot(has);
                if (m == 0) break;
                if (has) {
                    const uint32_t pos = qn + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                  __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
                    queue[wave][pos] = (g << 5) | (uint32_t)(__ffs(cand) - 1);
                    cand &= cand - 1;
                }
                qn += (uint32_t)__popcll(m);
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            while (qn >= 64) {                              // settle full batches (LIFO)
                qn -= 64;
                flips += settle_candidate(d, s0 + queue[wave][qn + lane]);
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            }
        }
        if ((uint32_t)lane < qn) flips += settle_candidate(d, s0 + queue[wave][lane]);
    } else {
        // general threshold (rate >= 2^-8) or every element
        const uint64_t Ttop = T >> 56, Tlow = T & ((uint64_t(1) << 56) - 1);
        for (uint32_t g = threadIdx.x; g < ngroups; g += kBlock) {
            const uint64_t q = q0 + g;
            uint64_t A[4];
            if (!d.all) philox(q, 0, d.seed, A);
            const uint64_t ibase = q << 5;
            const uint32_t cnt = (n - ibase) < 32 ? (uint32_t)(n - ibase) : 32u;
            for (uint32_t b = 0; b < cnt; ++b) {
                const uint64_t i = ibase + b;
                bool f = d.all;
                if (!f) {
                    const uint64_t top = (A[b >> 3] >> (8 * (b & 7))) & 0xFF;
                    if (top < Ttop) {
                        f = true;
                    } else if (top == Ttop) {
                        uint64_t B[4];
                        philox(i >> 2, 1, d.seed, B);
                        f = (B[i & 3] & ((uint64_t(1) << 56) - 1)) < Tlow;
                    }
                }
                if (f) {
                    flip(d, i);
                    ++flips;
                }
            }
        }
    }
    // block sum of the flip count (integers: any order)
    __shared__ uint32_t red[kBlock / 64];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) flips += __shfl_xor(flips, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = flips;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int w = 0; w < kBlock / 64; ++w) t += red[w];
        P.seg_counts[seg] = t;
    }
}

__global__ void __launch_bounds__(kBlock) inject_sum_kernel(InjParams P) {
    const int item = blockIdx.x;
    const InjDesc d = P.descs[item];
    uint64_t t = 0;
    for (int s = threadIdx.x; s < d.nsegs; s += kBlock) t += P.seg_counts[d.first_seg + s];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o);
    __shared__ uint64_t red[kBlock / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t s = 0;
        for (int w = 0; w < kBlock / 64; ++w) s += red[w];
        P.counts[item] = (int64_t)s;
    }
}

}  // namespace

hipError_t launch_inject(const InjParams &p, int64_t total_segs, hipStream_t s) {
    if (total_segs <= 0) return hipSuccess;
    hipLaunchKernelGGL(inject_kernel, dim3((unsigned)total_segs), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_inject_sum(const InjParams &p, hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipLaunchKernelGGL(inject_sum_kernel, dim3((unsigned)p.count), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

}  // namespace peat
