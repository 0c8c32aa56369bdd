// Read-only streaming kernel: the device's read ceiling under the access
// pattern of the signature chunk pass (16-byte nontemporal buffer loads per
// lane, two register sets used in turn so the next step's loads are in
// flight, 256-thread blocks, one contiguous 2 MiB span per block -- the bytes
// of one 2^18-element f32 chunk pair).  A measurement aid, not a step of the
// method.
#include "peat_internal.h"

namespace peat {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSpanLog2 = 21;        // bytes per block
constexpr int kU = 8;                // 16-byte loads per lane per step
constexpr uint32_t kStep = kU * kBlock * 16u;
constexpr int kLoadNT = 2;           // nontemporal cache policy

__global__ void __launch_bounds__(kBlock) stream_read_kernel(const char *buf, int64_t bytes, uint32_t *sink) {
    const int64_t off = (int64_t)blockIdx.x << kSpanLog2;
    const int64_t rest = bytes - off;
    const uint32_t len = (uint32_t)(rest < (int64_t(1) << kSpanLog2) ? rest : (int64_t(1) << kSpanLog2));
    // the resource covers exactly this block's span
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void *)(buf + off), (short)0, (int)len, 0x00020000);
    const uint32_t lane_off = threadIdx.x * 16u;
    const uint32_t nsteps = (len / kStep) & ~1u;   // an even number of full steps
    u32x4 acc = {0u, 0u, 0u, 0u};
    auto load = [&](u32x4 (&x)[kU], uint32_t s) {
#pragma unroll
        for (int u = 0; u < kU; ++u)
            x[u] = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)lane_off, (int)(s * kStep + u * kBlock * 16u), kLoadNT);
    };
    if (nsteps > 0) {
        u32x4 a[kU], b[kU];
        const uint32_t last = nsteps - 1;
        load(a, 0);
        for (uint32_t s = 0; s < nsteps; s += 2) {
            load(b, s + 1);
#pragma unroll
            for (int u = 0; u < kU; ++u) acc ^= a[u];
            load(a, min(s + 2, last));             // a redundant in-bounds reload at the end
#pragma unroll
            for (int u = 0; u < kU; ++u) acc ^= b[u];
        }
    }
    // the rest of the span (an odd last step, a span shorter than 2 MiB)
    for (uint32_t v = nsteps * (kStep / 16u) + threadIdx.x; v < len / 16u; v += kBlock)
        acc ^= __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(v * 16u), 0, kLoadNT);
    uint32_t r = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) r ^= __shfl_xor(r, o);
    __shared__ uint32_t red[kBlock / 64];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = r;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t x = 0;
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) x ^= red[w];
        sink[blockIdx.x] = x;                  // one word per span: no atomics
    }
}

}  // namespace

hipError_t launch_stream_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t s) {
    if (bytes <= 0) return hipSuccess;
    const int64_t blocks = (bytes + (int64_t(1) << kSpanLog2) - 1) >> kSpanLog2;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                       static_cast<const char *>(buf), bytes, sink);
    return hipGetLastError();
}

}  // namespace peat
