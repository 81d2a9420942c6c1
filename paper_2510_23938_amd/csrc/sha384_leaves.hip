// sha384_leaves.hip -- SHA-384 of every chunk (FIPS 180-4 section 6.5), one
// chunk per lane, 64 chunks per wave: the hash of the paper's own kernel
// listings, on the same schedule and load path as the SHA-256 leaf kernel.
//
// Blocks are 128 bytes, so one LDS stage -- 128 bytes per chunk, eight
// 16-byte direct-to-LDS loads per wave, swizzled rows -- is exactly one block.
// Padding (section 5.1.2): the 0..127 tail bytes, 0x80, zeros and the 128-bit
// big-endian bit length, in one final block when the tail is at most 111
// bytes, else two.  Tail reads are aligned dwords that each hold at least one
// chunk byte, as in the SHA-256 kernel.
#include "hv_kernels.h"
#include "sha384_device.h"

namespace hv {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kStageBytes = 128;
constexpr int kRowsPerLoad = 1024 / kStageBytes;

__device__ __forceinline__ uint32_t swizzle(uint32_t c) { return (c ^ (c >> 3)) & 7u; }
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
__device__ __forceinline__ void wait_lgkm_all() { __builtin_amdgcn_s_waitcnt(0xC07F); }  // lgkmcnt(0)

__device__ __forceinline__ void block_from(const uint4 r[8], uint64_t W[16]) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        W[2 * k] = be64(r[k].x, r[k].y);
        W[2 * k + 1] = be64(r[k].z, r[k].w);
    }
}

// Whole 128-byte blocks of the wave's 64 chunks (all 16-byte aligned), staged
// through this wave's 8 KB LDS rows; nfull <= 2^30 (the chunk-size limit).
__device__ __forceinline__ void full_blocks_lds(uint64_t H[8], uint64_t src, uint32_t nfull, uint8_t* rows) {
    const uint32_t lane = threadIdx.x & 63;
    uint32_t nmax = nfull, nmin = nfull;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t a = __shfl_xor(nmax, o), b = __shfl_xor(nmin, o);
        nmax = a > nmax ? a : nmax;
        nmin = b < nmin ? b : nmin;
    }
    nmax = __builtin_amdgcn_readfirstlane(nmax);
    nmin = __builtin_amdgcn_readfirstlane(nmin);
    if (nmax == 0) return;

    const uint8_t* from[kRowsPerLoad];
    uint32_t until[kRowsPerLoad];  // blocks of the chunk this lane's slot j belongs to
#pragma unroll
    for (int j = 0; j < kRowsPerLoad; ++j) {
        const uint32_t c = kRowsPerLoad * j + (lane >> 3);
        const uint32_t slot = (lane & 7) ^ swizzle(c);
        const uint64_t s = __shfl(src, (int)c);
        from[j] = reinterpret_cast<const uint8_t*>(s) + 16 * slot;
        until[j] = __shfl(nfull, (int)c);
    }
    const bool uniform = nmin == nmax;

#pragma unroll
    for (int j = 0; j < kRowsPerLoad; ++j)
        if (0 < until[j]) __builtin_amdgcn_global_load_lds(from[j], rows + 1024 * j, 16, 0, 0);

    const uint8_t* row = rows + kStageBytes * lane;
    const uint32_t sw = swizzle(lane);
    for (uint32_t b = 0; b < nmax; ++b) {
        wait_vm_all();
        uint4 r[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) r[k] = *reinterpret_cast<const uint4*>(row + 16 * (k ^ sw));
        wait_lgkm_all();
        const uint32_t nx = b + 1;
        if (nx < nmax) {
            const uint64_t off = (uint64_t)kStageBytes * nx;
            if (uniform) {
#pragma unroll
                for (int j = 0; j < kRowsPerLoad; ++j)
                    __builtin_amdgcn_global_load_lds(from[j] + off, rows + 1024 * j, 16, 0, 0);
            } else {
#pragma unroll
                for (int j = 0; j < kRowsPerLoad; ++j)
                    if (nx < until[j]) __builtin_amdgcn_global_load_lds(from[j] + off, rows + 1024 * j, 16, 0, 0);
            }
        }
        if (b < nfull) {
            uint64_t W[16];
            block_from(r, W);
            compress512(H, W);
        }
    }
}

// Up to 128 bytes at p (any alignment) as 32 little-endian words; bytes at or
// past `valid` are undefined.  Loads only aligned dwords holding a valid byte.
__device__ __forceinline__ void gather_words(const uint8_t* p, uint32_t valid, uint32_t X[32]) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(p);
    const uint32_t sh = (uint32_t)(pa & 3);
    const uint32_t* a = reinterpret_cast<const uint32_t*>(pa - sh);
    uint32_t D[33];
#pragma unroll
    for (int k = 0; k < 33; ++k) D[k] = (uint32_t)(4 * k) < sh + valid ? a[k] : 0u;
#pragma unroll
    for (int i = 0; i < 32; ++i) X[i] = __builtin_amdgcn_alignbyte(D[i + 1], D[i], sh);
}

__device__ __forceinline__ void full_blocks_any(uint64_t H[8], const uint8_t* p, uint32_t nfull) {
    for (uint32_t b = 0; b < nfull; ++b) {
        uint32_t X[32];
        gather_words(p + 128 * (uint64_t)b, 128, X);
        uint64_t W[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) W[i] = be64(X[2 * i], X[2 * i + 1]);
        compress512(H, W);
    }
}

// Final block(s): r = 0..127 tail bytes at p, 0x80, zeros, 128-bit bit length.
__device__ __forceinline__ void final_blocks(uint64_t H[8], const uint8_t* p, uint32_t r, uint64_t total) {
    uint32_t X[32];
    gather_words(p, r, X);
#pragma unroll
    for (int i = 0; i < 32; ++i) {
        const int nv = (int)r - 4 * i;
        const uint32_t keep = nv >= 4 ? 0xffffffffu : (nv <= 0 ? 0u : (1u << (8 * nv)) - 1u);
        const uint32_t pad = (nv >= 0 && nv < 4) ? (0x80u << (8 * nv)) : 0u;
        X[i] = (X[i] & keep) | pad;
    }
    uint64_t W[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) W[i] = be64(X[2 * i], X[2 * i + 1]);
    const uint64_t bits_hi = total >> 61, bits_lo = total << 3;
    if (r <= 111) {
        W[14] = bits_hi;
        W[15] = bits_lo;
        compress512(H, W);
    } else {
        compress512(H, W);
#pragma unroll
        for (int i = 0; i < 14; ++i) W[i] = 0;
        W[14] = bits_hi;
        W[15] = bits_lo;
        compress512(H, W);
    }
}

__global__ void __launch_bounds__(kThreads) sha384_leaves_kernel(const LeafDesc* __restrict__ desc, uint64_t n_slots,
                                                                 uint64_t out_bound, uint8_t* __restrict__ digests) {
    __shared__ __attribute__((aligned(16))) uint8_t stage[kWaves][64 * kStageBytes];
    const uint64_t slot = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool live = slot < n_slots;
    LeafDesc d = {0, 0, 0};
    if (live) d = desc[slot];
    const uint8_t* p = reinterpret_cast<const uint8_t*>(d.src);
    const uint32_t nfull = (uint32_t)(d.nbytes >> 7);

    uint64_t H[8];
    init_state384(H);
    if (__all((d.src & 15) == 0)) {
        const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        full_blocks_lds(H, d.src, nfull, stage[wave]);
    } else {
        full_blocks_any(H, p, nfull);
    }
    final_blocks(H, p + ((uint64_t)nfull << 7), (uint32_t)(d.nbytes & 127), d.nbytes);
    if (live && d.out < out_bound) store_digest384(digests + 48 * d.out, H);
}

}  // namespace

hipError_t launch_sha384_leaves(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                                hipStream_t s) {
    for (uint64_t base = 0; base < n_slots; base += kMaxSlotsPerLaunch) {
        const uint64_t n = n_slots - base < kMaxSlotsPerLaunch ? n_slots - base : kMaxSlotsPerLaunch;
        sha384_leaves_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(desc + base, n, out_bound,
                                                                                          digests);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace hv
