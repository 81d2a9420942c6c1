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

// Issue rate of one instruction: eight independent chains per lane, four
// trips of the eight per loop iteration, written as inline assembly so that
// the compiler neither fuses (two adds into v_add3) nor splits them.
constexpr int kOpKinds = 8;  // alignbit, bitop3, add3, add, xor, lshr, perm, lshl_add_u64

#define HV_CHAIN8(S) S(0) S(1) S(2) S(3) S(4) S(5) S(6) S(7)

template <int OP>
__global__ void __launch_bounds__(kThreads) op_rate_kernel(uint32_t* __restrict__ sink, uint32_t iters) {
    const uint32_t tid = blockIdx.x * kThreads + threadIdx.x;
    uint32_t x[kChains];
    uint64_t w[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) {
        x[k] = tid * 0x9E3779B9u + (uint32_t)k;
        w[k] = hv::pack(tid, (uint32_t)k);
    }
    const uint32_t y = tid ^ 0x01234567u, z = tid + 0x5bd1e995u;
    const uint64_t y64 = hv::pack(y, z);
    for (uint32_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int rep = 0; rep < 4; ++rep) {
            if constexpr (OP == 0) {
#define S(k) asm volatile("v_alignbit_b32 %0, %0, %1, 7" : "+v"(x[k]) : "v"(y));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 1) {
#define S(k) asm volatile("v_bitop3_b32 %0, %0, %1, %2 bitop3:0x96" : "+v"(x[k]) : "v"(y), "v"(z));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 2) {
#define S(k) asm volatile("v_add3_u32 %0, %0, %1, %2" : "+v"(x[k]) : "v"(y), "v"(z));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 3) {
#define S(k) asm volatile("v_add_u32_e32 %0, %0, %1" : "+v"(x[k]) : "v"(y));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 4) {
#define S(k) asm volatile("v_xor_b32_e32 %0, %0, %1" : "+v"(x[k]) : "v"(y));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 5) {
#define S(k) asm volatile("v_lshrrev_b32_e32 %0, 3, %0" : "+v"(x[k]));
                HV_CHAIN8(S)
#undef S
            } else if constexpr (OP == 6) {
#define S(k) asm volatile("v_perm_b32 %0, %0, %1, %2" : "+v"(x[k]) : "v"(y), "v"(z));
                HV_CHAIN8(S)
#undef S
            } else {
#define S(k) asm volatile("v_lshl_add_u64 %0, %0, 0, %1" : "+v"(w[k]) : "v"(y64));
                HV_CHAIN8(S)
#undef S
            }
        }
    }
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < kChains; ++k) r ^= x[k] ^ hv::hi32(w[k]) ^ hv::lo32(w[k]);
    sink[tid] = r;
}

#undef HV_CHAIN8

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

hv_status hv_mb_op_rate(uint32_t op, uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch,
                        hipStream_t stream) {
    if (sink == nullptr || ops_per_launch == nullptr || grid == 0 || op >= (uint32_t)kOpKinds)
        return HV_ERR_INVALID_ARG;
    switch (op) {
        case 0: op_rate_kernel<0><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 1: op_rate_kernel<1><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 2: op_rate_kernel<2><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 3: op_rate_kernel<3><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 4: op_rate_kernel<4><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 5: op_rate_kernel<5><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        case 6: op_rate_kernel<6><<<grid, kThreads, 0, stream>>>(sink, iters); break;
        default: op_rate_kernel<7><<<grid, kThreads, 0, stream>>>(sink, iters); break;
    }
    *ops_per_launch = (uint64_t)grid * kThreads * iters * 4 * kChains;
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

hv_status hv_mb_hbm_read(const void* buf, uint64_t nbytes, uint32_t* sink, uint32_t grid, hipStream_t stream) {
    if (buf == nullptr || sink == nullptr || grid == 0 || nbytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
        return HV_ERR_INVALID_ARG;
    hbm_read_kernel<<<grid, kThreads, 0, stream>>>(static_cast<const uint4*>(buf), nbytes / 16, sink);
    return hipGetLastError() == hipSuccess ? HV_OK : HV_ERR_HIP;
}

}  // extern "C"
