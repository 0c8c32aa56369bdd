// Random-bit-flip injector for gfx950 (the RBF error model of Section II-B,
// used by Inject() in Algorithms 1 and 2); the same decisions drive the
// random-zero and random-NaN models at a rate.
//
// Element i of a tensor flips iff its 64-bit uniform U_i is below
// T = floor(rate * 2^64) (every element when rate >= 1).  U_i is built from
// Philox4x32-10 (Salmon et al., SC'11) keyed by the seed, block c of stream s
// at counter (lo32(c), hi32(c), s, 0):
//   top byte    = byte (i mod 16) of block i/16 of stream 0
//   low 56 bits = 64-bit word (i mod 2) of block i/2 of stream 1
// A flipped element toggles the j-th lowest set bit of the mask with
// j = floor(y * popcount(mask) / 2^32), y = word 0 of block i of stream 2.
//
// For T < 2^56 an element can only flip when its top byte is 0, so each lane
// draws two blocks per 32 elements and evaluates the low bits only for the
// (1 in 256) elements whose top byte is zero.  The tensor is read and written
// only at flipped elements.
#include "philox.h"

namespace peat {
namespace {

// The chosen element's new bits: a bit flip, +0 or the type's quiet NaN.
__device__ __forceinline__ void flip(const InjDesc &d, uint64_t i) {
    if (d.model == PEAT_MODEL_BITFLIP) {
        const int b = chosen_bit(d.seed, d.mask, d.popc, i);
        if (d.dtype == PEAT_F32) {
            uint32_t *p = static_cast<uint32_t *>(d.x) + i;
            *p ^= 1u << b;
        } else {
            uint16_t *p = static_cast<uint16_t *>(d.x) + i;
            *p = (uint16_t)(*p ^ (1u << b));
        }
    } else {
        const bool nan = d.model == PEAT_MODEL_NAN;
        if (d.dtype == PEAT_F32) {
            static_cast<uint32_t *>(d.x)[i] = nan ? 0x7FC00000u : 0u;
        } else {
            static_cast<uint16_t *>(d.x)[i] = (uint16_t)(nan ? (d.dtype == PEAT_F16 ? 0x7E00u : 0x7FC0u) : 0u);
        }
    }
}

constexpr int kQCap = 64 + 32 * 64;   // per-wave queue: < 64 left over + one append of 32 per lane

// Low 56 bits of U_i for a queued candidate (its top byte is 0, so U_i is
// just these bits): flip the element when they are below T.
__device__ __forceinline__ uint32_t settle_candidate(const InjDesc &d, uint64_t i) {
    uint32_t B[4];
    philox(i >> 1, 1, d.seed, B);
    const uint64_t low = block_word64(B, (uint32_t)(i & 1)) & ((uint64_t(1) << 56) - 1);
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
                // the 32 top bytes of the group: blocks 2(q0+g) and 2(q0+g)+1
                uint32_t A[8];
                philox(2 * (q0 + g), 0, d.seed, A);
                philox(2 * (q0 + g) + 1, 0, d.seed, A + 4);
                // exact zero-byte mask of each word: bit 7 of a byte is set
                // iff the byte is zero; one multiply gathers bits 7, 15, 23,
                // 31 into bits 28..31 (the other partial products land on
                // distinct lower bits, so nothing carries)
#pragma unroll
                for (int w = 0; w < 8; ++w) {
                    const uint32_t v = A[w];
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
            uint32_t A[8];
            if (!d.all) {
                philox(2 * q, 0, d.seed, A);
                philox(2 * q + 1, 0, d.seed, A + 4);
            }
            const uint64_t ibase = q << 5;
            const uint32_t cnt = (n - ibase) < 32 ? (uint32_t)(n - ibase) : 32u;
            for (uint32_t b = 0; b < cnt; ++b) {
                const uint64_t i = ibase + b;
                bool f = d.all;
                if (!f) {
                    const uint64_t top = (A[b >> 2] >> (8 * (b & 3))) & 0xFF;
                    if (top < Ttop) {
                        f = true;
                    } else if (top == Ttop) {
                        uint32_t B[4];
                        philox(i >> 1, 1, d.seed, B);
                        f = (block_word64(B, (uint32_t)(i & 1)) & ((uint64_t(1) << 56) - 1)) < Tlow;
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
