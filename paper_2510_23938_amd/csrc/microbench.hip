// microbench.hip -- roofline denominators measured on the device: the issue
// rate of the SHA-256 VALU mix and of the SHA-384 mix (32-bit logic on word
// halves plus 64-bit adds), register-only SHA-256 / SHA-384 ceilings, and the
// streaming HBM read bandwidth.
#include <hip/hip_runtime.h>

#include "hv.h"
#include "hv_microbench.h"
#include "sha256_device.h"
#include "sha384_device.h"

namespace {

constexpr int kThreads = 256;
constexpr int kChains = 8;       // independent dependency chains per lane
constexpr int kOpsPerChain = 3;  // alignbit, bitop3, add3 per chain per trip

__global__ void __launch_bounds__(kThreads) valu_mix_kernel(uint32_t* __restrict__ sink, uint32_t iters,
                                                            uint32_t seed) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    uint32_t x[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) x[k] = seed ^ (tid * 0x9E3779B9u) ^ (uint32_t)(k * 0x85EBCA6Bu);
    const uint32_t y = tid ^ seed, z = tid + seed;
#pragma unroll 4
    for (uint32_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) {
            const uint32_t a = __builtin_amdgcn_alignbit(x[k], x[k], 7);
            const uint32_t b = __builtin_amdgcn_bitop3_b32(a, y, x[k], 0x96);
            x[k] = b + z + a;
        }
    }
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < kChains; ++k) r ^= x[k];
    sink[tid] = r;
}

// The SHA-384 round mix: per chain and trip, a 64-bit rotate (two
// v_alignbit_b32), a 3-input XOR on both halves (two v_bitop3_b32) and one
// 64-bit add (v_lshl_add_u64): five instructions.
constexpr int kOpsPerChain64 = 5;

__global__ void __launch_bounds__(kThreads) valu64_mix_kernel(uint32_t* __restrict__ sink, uint32_t iters,
                                                              uint32_t seed) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    uint64_t x[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k)
        x[k] = hv::pack(seed ^ (tid * 0x9E3779B9u), (uint32_t)(k * 0x85EBCA6Bu) + tid);
    const uint64_t y = hv::pack(tid ^ seed, tid + seed), z = hv::pack(tid * 3u, seed ^ 0x5bd1e995u);
#pragma unroll 4
    for (uint32_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) {
            const uint64_t a = hv::rotr64<7>(x[k]);
            x[k] = hv::bitop3_64<0x96>(a, y, z) + x[k];
        }
    }
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < kChains; ++k) r ^= hv::hi32(x[k]) ^ hv::lo32(x[k]);
    sink[tid] = r;
}

__global__ void __launch_bounds__(kThreads) hbm_read_kernel(const uint4* __restrict__ buf, uint64_t n16,
                                                            uint32_t* __restrict__ sink) {
    const uint64_t tid = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    const uint64_t stride = (uint64_t)gridDim.x * kThreads;
    uint32_t acc = 0;
    uint64_t i = tid;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const uint4 a = buf[i], b = buf[i + stride], c = buf[i + 2 * stride], d = buf[i + 3 * stride];
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
    }
    for (; i < n16; i += stride) {
        const uint4 a = buf[i];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    sink[tid] = acc;
}

// SHA-256 compressions on registers only: each lane chains `blocks`
// compressions of a block derived from its own state, with no memory traffic
// in the loop -- the ceiling the leaf kernel's arithmetic can reach.
__global__ void __launch_bounds__(kThreads) sha256_registers_kernel(uint32_t* __restrict__ sink, uint32_t blocks) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    uint32_t H[8];
    hv::init_state(H);
    uint32_t M[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) M[i] = tid * 16u + (uint32_t)i;
    for (uint32_t b = 0; b < blocks; ++b) {
        uint32_t W[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) W[i] = M[i] ^ H[i & 7];
        hv::compress(H, W);
    }
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) r ^= H[i];
    sink[tid] = r;
}

// SHA-384 compressions on registers only (section 6.4 rounds), as above.
__global__ void __launch_bounds__(kThreads) sha384_registers_kernel(uint32_t* __restrict__ sink, uint32_t blocks) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    uint64_t H[8];
    hv::init_state384(H);
    uint64_t M[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) M[i] = hv::pack(tid, (uint32_t)i);
    for (uint32_t b = 0; b < blocks; ++b) {
        uint64_t W[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) W[i] = M[i] ^ H[i & 7];
        hv::compress512(H, W);
    }
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) r ^= hv::hi32(H[i]) ^ hv::lo32(H[i]);
    sink[tid] = r;
}

}  // namespace

extern "C" {

hv_status hv_mb_valu(uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch, hipStream_t stream) {
    if (sink == nullptr || ops_per_launch == nullptr || grid == 0) return HV_ERR_INVALID_ARG;
    valu_mix_kernel<<<grid, kThreads, 0, stream>>>(sink, iters, 0x2510u);
    *ops_per_launch = (uint64_t)grid * kThreads * iters * kChains * kOpsPerChain;
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

hv_status hv_mb_sha256(uint32_t* sink, uint32_t grid, uint32_t blocks, uint64_t* blocks_per_launch,
                       hipStream_t stream) {
    if (sink == nullptr || blocks_per_launch == nullptr || grid == 0) return HV_ERR_INVALID_ARG;
    sha256_registers_kernel<<<grid, kThreads, 0, stream>>>(sink, blocks);
    *blocks_per_launch = (uint64_t)grid * kThreads * blocks;
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

hv_status hv_mb_valu64(uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch, hipStream_t stream) {
    if (sink == nullptr || ops_per_launch == nullptr || grid == 0) return HV_ERR_INVALID_ARG;
    valu64_mix_kernel<<<grid, kThreads, 0, stream>>>(sink, iters, 0x2510u);
    *ops_per_launch = (uint64_t)grid * kThreads * iters * kChains * kOpsPerChain64;
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

hv_status hv_mb_sha384(uint32_t* sink, uint32_t grid, uint32_t blocks, uint64_t* blocks_per_launch,
                       hipStream_t stream) {
    if (sink == nullptr || blocks_per_launch == nullptr || grid == 0) return HV_ERR_INVALID_ARG;
    sha384_registers_kernel<<<grid, kThreads, 0, stream>>>(sink, blocks);
    *blocks_per_launch = (uint64_t)grid * kThreads * blocks;
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

hv_status hv_mb_hbm_read(const void* buf, uint64_t nbytes, uint32_t* sink, uint32_t grid, hipStream_t stream) {
    if (buf == nullptr || sink == nullptr || grid == 0 || nbytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
        return HV_ERR_INVALID_ARG;
    hbm_read_kernel<<<grid, kThreads, 0, stream>>>(static_cast<const uint4*>(buf), nbytes / 16, sink);
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

}  // extern "C"
