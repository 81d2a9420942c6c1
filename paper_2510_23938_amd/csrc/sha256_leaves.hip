// sha256_leaves.hip -- SHA-256 of every chunk (Algorithm 1's per-chunk GPU
// hash), one chunk per lane, 64 chunks per wave.
//
// SHA-256 is a chain of dependent compressions (Merkle-Damgard), so a chunk
// cannot be split across lanes; parallelism is the number of chunks.  Each
// lane keeps the eight state words and a 16-word message-schedule ring in
// VGPRs and runs FIPS 180-4's padding itself (section 5.1.1): whole 64-byte
// blocks first, then one or two final blocks holding the 0..63 tail bytes,
// the 0x80 byte, zeros and the 64-bit bit length.
//
// Memory safety at tails: every load is a dword (or wider, 16-byte aligned)
// access that contains at least one byte of the chunk, so no access touches a
// page the chunk does not touch.  Bytes past the chunk end that such a load
// brings in are masked off before hashing.
#include "hv_kernels.h"
#include "sha256_device.h"

namespace hv {
namespace {

constexpr int kThreads = 256;

// Whole blocks from a 16-byte aligned chunk: four 16-byte loads per block,
// issued one block ahead of the compression that consumes them.
__device__ __forceinline__ void full_blocks_aligned(uint32_t H[8], const uint8_t* p, uint64_t nfull) {
    if (nfull == 0) return;
    const uint4* q = reinterpret_cast<const uint4*>(p);
    uint4 x0 = q[0], x1 = q[1], x2 = q[2], x3 = q[3];
    for (uint64_t b = 0; b < nfull; ++b) {
        uint32_t W[16] = {bswap(x0.x), bswap(x0.y), bswap(x0.z), bswap(x0.w), bswap(x1.x), bswap(x1.y),
                          bswap(x1.z), bswap(x1.w), bswap(x2.x), bswap(x2.y), bswap(x2.z), bswap(x2.w),
                          bswap(x3.x), bswap(x3.y), bswap(x3.z), bswap(x3.w)};
        // next block, or the current one again on the last iteration (in range)
        const uint64_t nb = b + 1 < nfull ? b + 1 : b;
        x0 = q[4 * nb]; x1 = q[4 * nb + 1]; x2 = q[4 * nb + 2]; x3 = q[4 * nb + 3];
        compress(H, W);
    }
}

// Up to 64 bytes starting at p (any alignment) as 16 little-endian words of
// the bytes p[0..63]; bytes at or past `valid` are undefined.  Loads only the
// aligned dwords that hold at least one of the first `valid` bytes.
__device__ __forceinline__ void gather_words(const uint8_t* p, uint32_t valid, uint32_t X[16]) {
    const uintptr_t pa = reinterpret_cast<uintptr_t>(p);
    const uint32_t sh = (uint32_t)(pa & 3);
    const uint32_t* a = reinterpret_cast<const uint32_t*>(pa - sh);
    uint32_t D[17];
#pragma unroll
    for (int k = 0; k < 17; ++k) D[k] = (uint32_t)(4 * k) < sh + valid ? a[k] : 0u;
#pragma unroll
    for (int i = 0; i < 16; ++i) X[i] = __builtin_amdgcn_alignbyte(D[i + 1], D[i], sh);
}

// Whole blocks from a chunk at any alignment.
__device__ __forceinline__ void full_blocks_any(uint32_t H[8], const uint8_t* p, uint64_t nfull) {
    for (uint64_t b = 0; b < nfull; ++b) {
        uint32_t W[16];
        gather_words(p + 64 * b, 64, W);
#pragma unroll
        for (int i = 0; i < 16; ++i) W[i] = bswap(W[i]);
        compress(H, W);
    }
}

// Final block(s): r = 0..63 tail bytes at p, then 0x80, zeros and the bit
// length of the whole chunk (total bytes).
__device__ __forceinline__ void final_blocks(uint32_t H[8], const uint8_t* p, uint32_t r, uint64_t total) {
    uint32_t W[16];
    gather_words(p, r, W);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int nv = (int)r - 4 * i;  // tail bytes that fall in word i
        const uint32_t keep = nv >= 4 ? 0xffffffffu : (nv <= 0 ? 0u : (1u << (8 * nv)) - 1u);
        const uint32_t pad = (nv >= 0 && nv < 4) ? (0x80u << (8 * nv)) : 0u;
        W[i] = bswap((W[i] & keep) | pad);
    }
    const uint64_t bits = total * 8;
    if (r <= 55) {
        W[14] = (uint32_t)(bits >> 32);
        W[15] = (uint32_t)bits;
        compress(H, W);
    } else {
        compress(H, W);
#pragma unroll
        for (int i = 0; i < 14; ++i) W[i] = 0;
        W[14] = (uint32_t)(bits >> 32);
        W[15] = (uint32_t)bits;
        compress(H, W);
    }
}

__global__ void __launch_bounds__(kThreads) sha256_leaves_kernel(const LeafDesc* __restrict__ desc, uint64_t n_leaves,
                                                                 uint8_t* __restrict__ digests) {
    const uint64_t slot = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool live = slot < n_leaves;
    LeafDesc d = {0, 0, 0};
    if (live) d = desc[slot];
    const uint8_t* p = reinterpret_cast<const uint8_t*>(d.src);
    const uint64_t nfull = d.nbytes >> 6;

    uint32_t H[8];
    init_state(H);
    if (__all((d.src & 15) == 0)) {
        full_blocks_aligned(H, p, nfull);
    } else {
        full_blocks_any(H, p, nfull);
    }
    final_blocks(H, p + (nfull << 6), (uint32_t)(d.nbytes & 63), d.nbytes);
    if (live && d.out < n_leaves) store_digest(digests + 32 * d.out, H);
}

}  // namespace

hipError_t launch_sha256_leaves(const LeafDesc* desc, uint64_t n_leaves, uint8_t* digests, hipStream_t s) {
    if (n_leaves == 0) return hipSuccess;
    const uint64_t blocks = (n_leaves + kThreads - 1) / kThreads;
    sha256_leaves_kernel<<<(unsigned)blocks, kThreads, 0, s>>>(desc, n_leaves, digests);
    return hipGetLastError();
}

}  // namespace hv
