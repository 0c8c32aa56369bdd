// Random-bit-flip injector for gfx950: one 256-thread block per 2^20-element
// segment of a tensor (the decisions are in inject_span.h), then a per-tensor
// sum of the segments' flip counts.
#include "inject_span.h"

namespace peat {
namespace {

__global__ void __launch_bounds__(kBlock) inject_kernel(InjParams P) {
    const int64_t seg = blockIdx.x;
    const int item = P.seg_item[seg];
    const InjDesc d = P.descs[item];
    const uint64_t s0 = (uint64_t)(seg - d.first_seg) << kInjSegLog2;   // first element
    const uint64_t n = (uint64_t)d.n;
    const uint64_t len = (n - s0) < (uint64_t(1) << kInjSegLog2) ? (n - s0) : (uint64_t(1) << kInjSegLog2);
    __shared__ uint32_t queue[kBlock / 64][kQCap];
    uint32_t flips = inject_span<false>(d, s0, len, queue);
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
