// split_common.h -- pieces shared by the two-wave leaf kernels
// (sha256_split.hip, sha384_split.hip): global-memory pointer types and a
// barrier that orders LDS only.
#pragma once
#include <stdint.h>
#include <hip/hip_runtime.h>

namespace hv {

// Global-memory pointers: loads through them are global (not flat) loads,
// which the LDS counter does not track, so a wait for LDS leaves them in flight.
typedef const __attribute__((address_space(1))) uint32_t* gwords;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4* gquads;

// A workgroup barrier that orders LDS only: it waits for this wave's LDS
// accesses, not for its global loads, so prefetches stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }   // lgkmcnt(0)

}  // namespace hv
