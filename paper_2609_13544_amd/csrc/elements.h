// Element access shared by the streaming kernels: 16-byte vectors of f32,
// f16 or bf16 bit patterns, their exact widening to binary64, and the buffer
// resource and cache policy of the streaming loads.
#pragma once

#include "peat_internal.h"

namespace peat {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte vector
typedef __attribute__((address_space(1))) const u32x4 gvec_t;
typedef __attribute__((address_space(1))) const uint32_t gu32_t;
typedef __attribute__((address_space(1))) const uint16_t gu16_t;

// Word 3 of a raw (unstrided, untyped) buffer resource on gfx9-family parts:
// 32-bit data format, default swizzle and cache policy.
constexpr int kBufFlags = 0x00020000;
// Cache-policy operand of the streaming loads: the nontemporal bit.  Each
// byte is read once, and on MI355X the hint raises the read rate of this
// access pattern from about 6.35 to 7.15 TB/s.
constexpr int kLoadNT = 2;

template <int DT> struct Tr;
template <> struct Tr<PEAT_F32>  { static constexpr int VEC = 4, W = 32; };
template <> struct Tr<PEAT_F16>  { static constexpr int VEC = 8, W = 16; };
template <> struct Tr<PEAT_BF16> { static constexpr int VEC = 8, W = 16; };

// Exact binary64 value of one element's bits.
template <int DT>
__device__ __forceinline__ double widen(uint32_t b) {
    if constexpr (DT == PEAT_F32) {
        return (double)__uint_as_float(b);
    } else if constexpr (DT == PEAT_BF16) {
        return (double)__uint_as_float(b << 16);
    } else {
        return (double)(float)__builtin_bit_cast(_Float16, (uint16_t)b);
    }
}

// Bits of element j of a 16-byte vector.
template <int DT>
__device__ __forceinline__ uint32_t lane_elem(const u32x4 &v, int j) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (Tr<DT>::W == 32) {
        return w[j];
    } else {
        return (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    }
}

// Bits of element i of a tensor (no alignment requirement beyond the type's).
template <int DT>
__device__ __forceinline__ uint32_t load_elem(const char *base, int64_t i) {
    if constexpr (Tr<DT>::W == 32) {
        return ((gu32_t *)base)[i];
    } else {
        return ((gu16_t *)base)[i];
    }
}

}  // namespace peat
