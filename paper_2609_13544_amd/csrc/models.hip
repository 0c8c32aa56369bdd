// The paper's other error models (Section II-B "Error Models"; Section III-C
// pseudo-errors; Section V-A settings) beyond the rate-driven injector:
//
//   corrupt_positions  num_pos distinct random positions (random value of the
//                      tensor or of the type, zero, NaN or bit flip), one block: positions are drawn in
//                      parallel, accepted in draw order through an LDS hash
//                      set, every source read before any position is written;
//   cast_round         the FP16 / BF16 error: round-to-nearest-even of an f32
//                      tensor to the narrower type, widened back, in place.
#include "elements.h"
#include "philox.h"

namespace peat {
namespace {

constexpr int kSet = 8192;                       // hash set of accepted positions
constexpr uint64_t kFree = ~uint64_t(0);
constexpr uint64_t kMaxDraws = uint64_t(1) << 24;   // bound of the draw loop

// High 64 bits of the 128-bit product a * b (floor(a * b / 2^64)).
__device__ __forceinline__ uint64_t mulhi64(uint64_t a, uint64_t b) { return __umul64hi(a, b); }

__device__ __forceinline__ uint32_t load_bits(const void *x, int dtype, int64_t i) {
    return dtype == PEAT_F32 ? static_cast<const uint32_t *>(x)[i] : static_cast<const uint16_t *>(x)[i];
}

__device__ __forceinline__ void store_bits(void *x, int dtype, int64_t i, uint32_t v) {
    if (dtype == PEAT_F32)
        static_cast<uint32_t *>(x)[i] = v;
    else
        static_cast<uint16_t *>(x)[i] = (uint16_t)v;
}

__global__ void __launch_bounds__(kBlock) corrupt_positions_kernel(void *x, int64_t n, int dtype, uint64_t seed,
                                                                   int model, int64_t num_pos, uint64_t mask,
                                                                   int popc, int64_t *out_pos) {
    __shared__ int64_t pos[PEAT_MAX_POSITIONS], src[PEAT_MAX_POSITIONS];
    __shared__ uint64_t set[kSet];
    __shared__ int64_t cp[kBlock], cs[kBlock];
    __shared__ uint32_t val[PEAT_MAX_POSITIONS];
    __shared__ int64_t m_sh;
    const int tid = threadIdx.x;
    for (int i = tid; i < kSet; i += kBlock) set[i] = kFree;
    if (tid == 0) m_sh = 0;
    __syncthreads();
    bool complete = false;
    for (uint64_t j0 = 0; j0 < kMaxDraws; j0 += kBlock) {
        uint32_t W[4];
        philox(j0 + tid, 3, seed, W);
        cp[tid] = (int64_t)mulhi64(block_word64(W, 0), (uint64_t)n);
        // the source index (random value) or the low bits of W1 (uniform bits)
        cs[tid] = model == PEAT_MODEL_UNIFORM ? (int64_t)(dtype == PEAT_F32 ? W[2] : (W[2] & 0xFFFFu))
                                              : (int64_t)mulhi64(block_word64(W, 1), (uint64_t)n);
        __syncthreads();
        if (tid == 0) {
            int64_t m = m_sh;
            for (int t = 0; t < kBlock && m < num_pos; ++t) {
                const uint64_t p = (uint64_t)cp[t];
                uint32_t h = (uint32_t)((p * 0x9E3779B97F4A7C15ull) >> 51);     // 13 bits
                bool fresh = false;
                while (true) {
                    if (set[h] == kFree) {
                        set[h] = p;
                        fresh = true;
                        break;
                    }
                    if (set[h] == p) break;
                    h = (h + 1) & (kSet - 1);
                }
                if (fresh) {
                    pos[m] = (int64_t)p;
                    src[m] = cs[t];
                    ++m;
                }
            }
            m_sh = m;
        }
        __syncthreads();
        complete = m_sh >= num_pos;
        __syncthreads();
        if (complete) break;
    }
    if (!complete) {                       // unreachable in practice; reported by the host
        for (int64_t m = tid; m < num_pos; m += kBlock) out_pos[m] = -1;
        return;
    }
    // every source and old value is read before any position is written
    for (int64_t m = tid; m < num_pos; m += kBlock) {
        const int64_t i = pos[m];
        uint32_t v;
        if (model == PEAT_MODEL_VALUE) {
            v = load_bits(x, dtype, src[m]);
        } else if (model == PEAT_MODEL_UNIFORM) {
            v = (uint32_t)src[m];
        } else if (model == PEAT_MODEL_ZERO) {
            v = 0;
        } else if (model == PEAT_MODEL_NAN) {
            v = dtype == PEAT_F32 ? 0x7FC00000u : (dtype == PEAT_F16 ? 0x7E00u : 0x7FC0u);
        } else {
            v = load_bits(x, dtype, i) ^ (1u << chosen_bit(seed, mask, popc, (uint64_t)i));
        }
        val[m] = v;
    }
    __syncthreads();
    for (int64_t m = tid; m < num_pos; m += kBlock) {
        store_bits(x, dtype, pos[m], val[m]);
        out_pos[m] = pos[m];
    }
}

// Round-to-nearest-even of f32 bits to binary16 (the hardware conversion,
// round-to-nearest-even mode) or bfloat16 (integer rounding on the bits),
// widened back; a NaN becomes sign | 0x7FC00000.
template <int TO>
__device__ __forceinline__ uint32_t round_bits(uint32_t b) {
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b & 0x80000000u) | 0x7FC00000u;
    if constexpr (TO == PEAT_F16) {
        return __float_as_uint((float)(_Float16)__uint_as_float(b));
    } else {
        return (b + 0x7FFFu + ((b >> 16) & 1u)) & 0xFFFF0000u;
    }
}

template <int TO>
__global__ void __launch_bounds__(kBlock) cast_round_kernel(uint32_t *x, int64_t n) {
    const int64_t nvec = ((reinterpret_cast<uintptr_t>(x) & 15) == 0) ? n / 4 : 0;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    u32x4 *v = reinterpret_cast<u32x4 *>(x);
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nvec; i += stride) {
        u32x4 a = v[i];
        a.x = round_bits<TO>(a.x);
        a.y = round_bits<TO>(a.y);
        a.z = round_bits<TO>(a.z);
        a.w = round_bits<TO>(a.w);
        v[i] = a;
    }
    for (int64_t i = nvec * 4 + (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
        x[i] = round_bits<TO>(x[i]);
}

}  // namespace

hipError_t launch_corrupt_positions(void *x, int64_t n, int dtype, uint64_t seed, int model, int64_t num_pos,
                                    uint64_t mask, int64_t *d_positions, hipStream_t s) {
    if (num_pos <= 0) return hipSuccess;
    const uint64_t m = model == PEAT_MODEL_BITFLIP ? mask : 1;
    hipLaunchKernelGGL(corrupt_positions_kernel, dim3(1), dim3(kBlock), 0, s, x, n, dtype, seed, model, num_pos, m,
                       __builtin_popcountll(m), d_positions);
    return hipGetLastError();
}

hipError_t launch_cast_round(void *x, int64_t n, int to_dtype, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t want = (n / 4 + kBlock - 1) / kBlock;
    const unsigned blocks = (unsigned)(want < 4096 ? (want > 0 ? want : 1) : 4096);
    if (to_dtype == PEAT_F16)
        hipLaunchKernelGGL(cast_round_kernel<PEAT_F16>, dim3(blocks), dim3(kBlock), 0, s, static_cast<uint32_t *>(x), n);
    else
        hipLaunchKernelGGL(cast_round_kernel<PEAT_BF16>, dim3(blocks), dim3(kBlock), 0, s, static_cast<uint32_t *>(x), n);
    return hipGetLastError();
}

}  // namespace peat
