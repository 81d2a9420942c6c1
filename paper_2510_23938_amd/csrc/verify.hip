// verify.hip -- root comparison (Algorithm 1's "compare root hash with
// expected value"), done on the GPU next to the root so that only a 4-byte
// flag crosses to the host.  The comparison always reads and folds every byte
// of the digest (32 for SHA-256, 48 for SHA-384) with no early exit, so its
// time does not depend on where roots differ.
#include "hv_kernels.h"

namespace hv {
namespace {

struct Expected {
    uint32_t w[12];  // the expected bytes (32 or 48), as little-endian words
};

__device__ __forceinline__ uint32_t load_le_word(const uint8_t* p) {
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) | ((uint32_t)p[3] << 24);
}

__global__ void verify_root_kernel(const uint8_t* __restrict__ root, Expected e, uint32_t nwords,
                                   uint32_t* __restrict__ flag) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    uint32_t diff = 0;
    for (uint32_t i = 0; i < nwords; ++i) diff |= load_le_word(root + 4 * i) ^ e.w[i];
    *flag = diff == 0 ? 1u : 0u;
}

// The same comparison with the expected bytes in device memory, so that a
// captured graph can check against whatever the caller last stored there.
__global__ void verify_root_dev_kernel(const uint8_t* __restrict__ root, const uint8_t* __restrict__ expected,
                                       uint32_t nwords, uint32_t* __restrict__ flag) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    uint32_t diff = 0;
    for (uint32_t i = 0; i < nwords; ++i) diff |= load_le_word(root + 4 * i) ^ load_le_word(expected + 4 * i);
    *flag = diff == 0 ? 1u : 0u;
}

__global__ void __launch_bounds__(256) compare_roots_kernel(const uint8_t* __restrict__ roots,
                                                            const uint8_t* __restrict__ expected, uint32_t n,
                                                            uint32_t nbytes, uint32_t* __restrict__ mismatch) {
    for (uint32_t r = blockIdx.x * 256 + threadIdx.x; r < n; r += gridDim.x * 256) {
        uint32_t diff = 0;
        for (uint32_t i = 0; i < nbytes; i += 4)
            diff |= load_le_word(roots + (size_t)nbytes * r + i) ^ load_le_word(expected + (size_t)nbytes * r + i);
        mismatch[r] = diff != 0 ? 1u : 0u;
    }
}

}  // namespace

hipError_t launch_verify_root(const uint8_t* root, const uint8_t* expected, uint32_t nbytes, uint32_t* flag,
                              hipStream_t s) {
    Expected e = {};
    for (uint32_t i = 0; i < nbytes && i < sizeof e.w; ++i) reinterpret_cast<uint8_t*>(e.w)[i] = expected[i];
    verify_root_kernel<<<1, 64, 0, s>>>(root, e, nbytes / 4, flag);
    return hipGetLastError();
}

hipError_t launch_verify_root_dev(const uint8_t* root, const uint8_t* expected, uint32_t nbytes, uint32_t* flag,
                                  hipStream_t s) {
    verify_root_dev_kernel<<<1, 64, 0, s>>>(root, expected, nbytes / 4, flag);
    return hipGetLastError();
}

hipError_t launch_compare_roots(const uint8_t* roots, const uint8_t* expected, uint32_t n, uint32_t nbytes,
                                uint32_t* mismatch, hipStream_t s) {
    if (n == 0) return hipSuccess;
    const uint32_t blocks = (n + 255) / 256;
    compare_roots_kernel<<<blocks < 65536 ? blocks : 65536, 256, 0, s>>>(roots, expected, n, nbytes, mismatch);
    return hipGetLastError();
}

}  // namespace hv
