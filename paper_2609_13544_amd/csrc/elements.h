// Element access shared by the streaming kernels: lane vectors of f32, f16,
// bf16 or binary64 bit patterns, their exact widening to binary64, rounding
// to a narrower format, and the buffer resource and cache policy of the
// streaming loads.
#pragma once

#include "peat_internal.h"

namespace peat {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte vector
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) const u32x4 gvec_t;
typedef __attribute__((address_space(1))) const uint32_t gu32_t;
typedef __attribute__((address_space(1))) const uint16_t gu16_t;
typedef __attribute__((address_space(1))) const u32x2 gu32x2_t;
typedef __attribute__((address_space(1))) const uint64_t gu64_t;

// Word 3 of a raw (unstrided, untyped) buffer resource on gfx9-family parts:
// 32-bit data format, default swizzle and cache policy.
constexpr int kBufFlags = 0x00020000;
// Cache-policy operand of the streaming loads: the nontemporal bit.  Each
// byte is read once, and on MI355X the hint raises the read rate of this
// access pattern from about 6.35 to 7.15 TB/s.
constexpr int kLoadNT = 2;

template <int DT> struct Tr;
template <> struct Tr<PEAT_F32>  { static constexpr int VEC = 4, W = 32, P = 24, EMIN = -126; };
template <> struct Tr<PEAT_F16>  { static constexpr int VEC = 8, W = 16, P = 11, EMIN = -14; };
template <> struct Tr<PEAT_BF16> { static constexpr int VEC = 8, W = 16, P = 8, EMIN = -126; };
template <> struct Tr<PEAT_F64>  { static constexpr int VEC = 2, W = 64, P = 53, EMIN = -1022; };

// A golden/test type pair.  Each lane handles VEC consecutive elements per
// vector: 16 bytes of the wider side and VEC * WN / 8 bytes of the narrower
// one, so every load instruction of a wave reads one contiguous span.  The
// ULP distance of a mixed pair is counted in the narrower format.
template <int DG, int DT> struct PairTr {
    static constexpr bool SAME = DG == DT;
    static constexpr int WG = Tr<DG>::W, WT = Tr<DT>::W;
    static constexpr int VEC = 128 / (WG > WT ? WG : WT);
    static constexpr int BG = VEC * WG / 8, BT = VEC * WT / 8;     // bytes per lane vector
    static constexpr bool GOLDEN_NARROW = Tr<DG>::P <= Tr<DT>::P;
    static constexpr int DN = GOLDEN_NARROW ? DG : DT;            // the narrower format
    static constexpr int WN = Tr<DN>::W;
};

// Exact binary64 value of one element's bits.
template <int DT, typename B>
__device__ __forceinline__ double widen(B b) {
    if constexpr (DT == PEAT_F64) {
        return __longlong_as_double((long long)b);
    } else if constexpr (DT == PEAT_F32) {
        return (double)__uint_as_float((uint32_t)b);
    } else if constexpr (DT == PEAT_BF16) {
        return (double)__uint_as_float((uint32_t)b << 16);
    } else {
        return (double)(float)__builtin_bit_cast(_Float16, (uint16_t)b);
    }
}

// Exact binary32 value of one element's bits (types of at most 32 bits).
template <int DT, typename B>
__device__ __forceinline__ float widen32(B b) {
    static_assert(Tr<DT>::W <= 32, "binary32 holds f32, f16 and bf16 values exactly");
    if constexpr (DT == PEAT_F32) {
        return __uint_as_float((uint32_t)b);
    } else if constexpr (DT == PEAT_BF16) {
        return __uint_as_float((uint32_t)b << 16);
    } else {
        return (float)__builtin_bit_cast(_Float16, (uint16_t)b);
    }
}

// Bits of element j of a lane vector held in (up to) 16 bytes.
template <int DT>
__device__ __forceinline__ auto lane_elem(const u32x4 &v, int j) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (Tr<DT>::W == 64) {
        return (uint64_t)w[2 * j] | ((uint64_t)w[2 * j + 1] << 32);
    } else if constexpr (Tr<DT>::W == 32) {
        return w[j];
    } else {
        return (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    }
}

// Bits of element i of a tensor (no alignment requirement beyond the type's).
template <int DT>
__device__ __forceinline__ auto load_elem(const char *base, int64_t i) {
    if constexpr (Tr<DT>::W == 64) {
        return (uint64_t)((gu64_t *)base)[i];
    } else if constexpr (Tr<DT>::W == 32) {
        return (uint32_t)((gu32_t *)base)[i];
    } else {
        return (uint32_t)((gu16_t *)base)[i];
    }
}

// Lane vector number `idx` (B bytes each) of a tensor, through a global load.
template <int B>
__device__ __forceinline__ u32x4 load_vec(const char *base, uint32_t idx) {
    if constexpr (B == 16) {
        return ((gvec_t *)base)[idx];
    } else if constexpr (B == 8) {
        const u32x2 r = ((gu32x2_t *)base)[idx];
        return u32x4{r.x, r.y, 0u, 0u};
    } else {
        return u32x4{((gu32_t *)base)[idx], 0u, 0u, 0u};
    }
}

// B bytes through a raw buffer load (voffset in a register, soffset scalar,
// cache policy AUX).
template <int B, int AUX>
__device__ __forceinline__ u32x4 buf_load(__amdgpu_buffer_rsrc_t rs, int voff, int soff) {
    if constexpr (B == 16) {
        return __builtin_amdgcn_raw_buffer_load_b128(rs, voff, soff, AUX);
    } else if constexpr (B == 8) {
        const u32x2 r = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, AUX);
        return u32x4{r.x, r.y, 0u, 0u};
    } else {
        return u32x4{__builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, AUX), 0u, 0u, 0u};
    }
}

// Binary32 bits of x rounded to odd: the nearest binary32 toward zero, with
// its last bit set when the conversion is inexact (beyond the binary32 range:
// the largest finite value).  A second rounding of this value to a format with
// at least two fewer significand bits is the correct round-to-nearest-even of
// x (Boldo and Melquiond, "When double rounding is odd", 2005).  x is not NaN.
__device__ __forceinline__ uint32_t round_odd_f32(double x) {
    const float f = (float)x;                                 // nearest, ties to even
    uint32_t b = __float_as_uint(f);
    if ((double)f != x && !(b & 1u))                          // inexact with an even result:
        b = __builtin_fabs((double)f) > __builtin_fabs(x) ? b - 1u : b + 1u;   // its odd neighbour
    return b;
}

// Bits of x (a value of format DW, not NaN) rounded to the narrower format DN:
// nearest, ties to even, Inf beyond DN's range.
template <int DN, int DW>
__device__ __forceinline__ uint32_t narrow_bits(double x) {
    static_assert(Tr<DN>::P < Tr<DW>::P, "DN must be the narrower format");
    if constexpr (DN == PEAT_F32) {
        return __float_as_uint((float)x);
    } else {
        // binary32 value first: exact from f32, rounded to odd from binary64
        const uint32_t fb = DW == PEAT_F32 ? __float_as_uint((float)x) : round_odd_f32(x);
        if constexpr (DN == PEAT_F16) {
            return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)__uint_as_float(fb));
        } else {
            return (fb + 0x7FFFu + ((fb >> 16) & 1u)) >> 16;
        }
    }
}

// Bits of a binary32 value (bit pattern fb, not NaN) rounded to the 16-bit
// format DN: nearest, ties to even, Inf beyond DN's range.
template <int DN>
__device__ __forceinline__ uint32_t narrow_f32_bits(uint32_t fb) {
    if constexpr (DN == PEAT_F16) {
        return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)__uint_as_float(fb));
    } else {
        return (fb + 0x7FFFu + ((fb >> 16) & 1u)) >> 16;
    }
}

}  // namespace peat
