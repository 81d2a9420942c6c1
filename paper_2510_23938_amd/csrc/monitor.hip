// monitor.hip -- the comparison step of continuous runtime monitoring: the
// freshly computed digests of a slice of leaves against the reference digests
// recorded when the weights were first verified.  Every leaf in the slice is
// compared in full (no early exit); mismatches are counted and the lowest
// mismatching leaf number is kept, with vector atomics in global memory.
#include "hv_kernels.h"

namespace hv {
namespace {

constexpr int kThreads = 256;

template <int D>
__global__ void __launch_bounds__(kThreads) monitor_compare_kernel(const uint8_t* __restrict__ digests,
                                                                   const uint8_t* __restrict__ ref, uint64_t first,
                                                                   uint64_t k, unsigned long long* __restrict__ result) {
    constexpr int kVec = D / 16;
    for (uint64_t e = (uint64_t)blockIdx.x * kThreads + threadIdx.x; e < k; e += (uint64_t)gridDim.x * kThreads) {
        const uint4* a = reinterpret_cast<const uint4*>(digests + (uint64_t)D * e);
        const uint4* b = reinterpret_cast<const uint4*>(ref + (uint64_t)D * (first + e));
        uint32_t diff = 0;
#pragma unroll
        for (int v = 0; v < kVec; ++v) {
            const uint4 x = a[v], y = b[v];
            diff |= (x.x ^ y.x) | (x.y ^ y.y) | (x.z ^ y.z) | (x.w ^ y.w);
        }
        if (diff != 0) {
            atomicAdd(&result[0], 1ull);
            atomicMin(&result[1], (unsigned long long)(first + e));
        }
    }
}

}  // namespace

hipError_t launch_monitor_compare(const uint8_t* digests, const uint8_t* ref, uint64_t first, uint64_t k, uint32_t D,
                                  uint64_t* result, hipStream_t s) {
    if (k == 0) return hipSuccess;
    const uint64_t blocks = (k + kThreads - 1) / kThreads;
    const unsigned grid = (unsigned)(blocks < 65536 ? blocks : 65536);
    unsigned long long* r = reinterpret_cast<unsigned long long*>(result);
    if (D == 48)
        monitor_compare_kernel<48><<<grid, kThreads, 0, s>>>(digests, ref, first, k, r);
    else
        monitor_compare_kernel<32><<<grid, kThreads, 0, s>>>(digests, ref, first, k, r);
    return hipGetLastError();
}

}  // namespace hv
