// The random-bit-flip decisions of the injector over one span of a tensor,
// by the threads of one 256-thread block (the RBF error model of Section
// II-B, used by Inject() in Algorithms 1 and 2; the same decisions drive the
// random-zero and random-NaN models at a rate).  Shared by the injection
// kernel and by the chunk pass that injects and signs in one sweep.
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
#pragma once

#include "philox.h"

namespace peat {
namespace {

constexpr int kQCap = 64 + 32 * 64;   // per-wave queue: < 64 left over + one append of 32 per lane

// The chosen element's new bits: a bit flip, +0, the type's quiet NaN, a
// value of the tensor before the call (read from the copy d.src) or a
// uniformly random bit pattern.
// ATOMIC: the bit flip is one device-scope atomic XOR on the aligned 32-bit
// word that holds the element, performed in L2 (a 16-bit neighbour in the
// same word is XORed with zeros, so no other element can lose an update).
// The fused chunk pass reads the flipped lines right after its own flips;
// the host admits only batches whose test lines no other block reads, so no
// compute unit holds a copy of such a line from before the flip.
template <bool ATOMIC>
__device__ __forceinline__ void flip(const InjDesc &d, uint64_t i) {
    if (d.model == PEAT_MODEL_BITFLIP) {
        const int b = chosen_bit(d.seed, d.mask, d.popc, i);
        if constexpr (ATOMIC) {
            const uintptr_t a = reinterpret_cast<uintptr_t>(d.x) + i * (d.dtype == PEAT_F32 ? 4 : 2);
            const uint32_t bit = (1u << b) << ((a & 2) * 8);
            __hip_atomic_fetch_xor(reinterpret_cast<uint32_t *>(a & ~uintptr_t(3)), bit, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        } else if (d.dtype == PEAT_F32) {
            uint32_t *p = static_cast<uint32_t *>(d.x) + i;
            *p ^= 1u << b;
        } else {
            uint16_t *p = static_cast<uint16_t *>(d.x) + i;
            *p = (uint16_t)(*p ^ (1u << b));
        }
    } else {
        uint32_t v;
        if (d.model == PEAT_MODEL_VALUE || d.model == PEAT_MODEL_UNIFORM) {
            // block i of stream 4: word 0 (64 bits) picks the source, word 2
            // is the uniform bit pattern
            uint32_t V[4];
            philox(i, 4, d.seed, V);
            if (d.model == PEAT_MODEL_VALUE) {
                const uint64_t s = __umul64hi(block_word64(V, 0), (uint64_t)d.n);
                v = d.dtype == PEAT_F32 ? static_cast<const uint32_t *>(d.src)[s]
                                        : static_cast<const uint16_t *>(d.src)[s];
            } else {
                v = V[2];
            }
        } else {
            const bool nan = d.model == PEAT_MODEL_NAN;
            v = nan ? (d.dtype == PEAT_F32 ? 0x7FC00000u : (d.dtype == PEAT_F16 ? 0x7E00u : 0x7FC0u)) : 0u;
        }
        if (d.dtype == PEAT_F32)
            static_cast<uint32_t *>(d.x)[i] = v;
        else
            static_cast<uint16_t *>(d.x)[i] = (uint16_t)v;
    }
}

// Low 56 bits of U_i for a queued candidate (its top byte is 0, so U_i is
// just these bits): flip the element when they are below T.
template <bool ATOMIC>
__device__ __forceinline__ uint32_t settle_candidate(const InjDesc &d, uint64_t i) {
    uint32_t B[4];
    philox(i >> 1, 1, d.seed, B);
    const uint64_t low = block_word64(B, (uint32_t)(i & 1)) & ((uint64_t(1) << 56) - 1);
    if (low < d.T) {
        flip<ATOMIC>(d, i);
        return 1;
    }
    return 0;
}

// The flips of elements [s0, s0 + len) of tensor d (s0 a multiple of 32),
// made by the block's threads; queue is a per-wave LDS queue.  Returns the
// calling thread's share of the flip count.
template <bool ATOMIC>
__device__ uint32_t inject_span(const InjDesc &d, uint64_t s0, uint64_t len, uint32_t (*queue)[kQCap]) {
    const uint64_t n = (uint64_t)d.n;
    const uint32_t ngroups = (uint32_t)((len + 31) / 32);
    const uint64_t q0 = s0 >> 5;
    const uint64_t T = d.T;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t flips = 0;

    if (!d.all && T < (uint64_t(1) << 56)) {
        // An element can flip only if the top byte of U_i is 0.  Each lane
        // draws one block per group of 32 elements; the zero-byte elements
        // go to a per-wave queue (span-relative offsets) whose entries are
        // settled 64 at a time, one per lane.
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
                flips += settle_candidate<ATOMIC>(d, s0 + queue[wave][qn + lane]);
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            }
        }
        if ((uint32_t)lane < qn) flips += settle_candidate<ATOMIC>(d, s0 + queue[wave][lane]);
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
            const uint64_t end = s0 + len < n ? s0 + len : n;
            const uint32_t cnt = (end - ibase) < 32 ? (uint32_t)(end - ibase) : 32u;
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
                    flip<ATOMIC>(d, i);
                    ++flips;
                }
            }
        }
    }
    return flips;
}

}  // namespace
}  // namespace peat
