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
// Load path for whole blocks (16-byte aligned chunks, the usual case): the
// wave stages its 64 chunks through LDS, 128 bytes (two blocks, one HBM line)
// per chunk per stage, with direct-to-LDS 16-byte loads
// (global_load_lds_dwordx4).  Load instruction j of a stage covers chunks
// 8j..8j+7, eight lanes per chunk, so every instruction reads eight whole
// 128-byte lines and every line is read from HBM once.  The 16-byte slots of
// a chunk's row are XOR-swizzled by chunk index so that the 64 lanes reading
// their own rows with ds_read_b128 hit distinct banks.  A stage is copied to
// VGPRs before the next stage's loads are issued into the same buffer, so
// the loads run under the two compressions of the current stage.  Chunks
// that are not 16-byte aligned take a dword-gather path instead.
//
// Memory safety at tails: the final partial block is read with aligned dword
// loads that each contain at least one byte of the chunk, so no access
// touches a page the chunk does not touch; bytes past the end are masked off.
#include "hv_kernels.h"
#include "sha256_device.h"

namespace hv {
namespace {

constexpr int kThreads = 256;                     // four waves per workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kStageBytes = 128;                  // bytes per chunk per stage
constexpr int kRowsPerLoad = 1024 / kStageBytes;  // chunks covered by one 64-lane 16-byte load

// Swizzle of a chunk's 16-byte slots within its LDS row.  Consecutive lanes
// (rows) differ in (c ^ c>>3) & 7, so the eight slots a group of lanes reads
// at once fall in different banks whether the LDS serves 8 or 16 lanes of a
// 16-byte read per cycle.
__device__ __forceinline__ uint32_t swizzle(uint32_t c) { return (c ^ (c >> 3)) & 7u; }

__device__ __forceinline__ void words_from(const uint4& x0, const uint4& x1, const uint4& x2, const uint4& x3,
                                           uint32_t W[16]) {
    W[0] = bswap(x0.x); W[1] = bswap(x0.y); W[2] = bswap(x0.z); W[3] = bswap(x0.w);
    W[4] = bswap(x1.x); W[5] = bswap(x1.y); W[6] = bswap(x1.z); W[7] = bswap(x1.w);
    W[8] = bswap(x2.x); W[9] = bswap(x2.y); W[10] = bswap(x2.z); W[11] = bswap(x2.w);
    W[12] = bswap(x3.x); W[13] = bswap(x3.y); W[14] = bswap(x3.z); W[15] = bswap(x3.w);
}

__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }   // vmcnt(0)
__device__ __forceinline__ void wait_lgkm_all() { __builtin_amdgcn_s_waitcnt(0xC07F); }  // lgkmcnt(0)

// Whole blocks of the wave's 64 chunks (every lane's chunk 16-byte aligned),
// staged through this wave's 8 KB LDS row buffer.  nfull: this lane's whole
// blocks (at most 2^31 under the library's chunk-size limit, so the block
// counts below cannot wrap).
__device__ __forceinline__ void full_blocks_lds(uint32_t H[8], uint64_t src, uint32_t nfull, uint8_t* rows) {
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
    const uint32_t stages = (nmax + 1) / 2;
    if (stages == 0) return;

    // The 16 bytes this lane moves for load j of every stage: chunk 8j + lane/8,
    // source slot (lane % 8) ^ swizzle(chunk), landing in LDS slot lane % 8.
    const uint8_t* from[kRowsPerLoad];
    uint32_t until[kRowsPerLoad];  // stages in which that slot lies in a whole block
#pragma unroll
    for (int j = 0; j < kRowsPerLoad; ++j) {
        const uint32_t c = kRowsPerLoad * j + (lane >> 3);
        const uint32_t slot = (lane & 7) ^ swizzle(c);
        const uint64_t s = __shfl(src, (int)c);
        const uint32_t nf = __shfl(nfull, (int)c);
        from[j] = reinterpret_cast<const uint8_t*>(s) + 16 * slot;
        until[j] = slot < 4 ? (nf + 1) / 2 : nf / 2;
    }
    const bool uniform = nmin == nmax;

#pragma unroll
    for (int j = 0; j < kRowsPerLoad; ++j)
        if (0 < until[j]) __builtin_amdgcn_global_load_lds(from[j], rows + 1024 * j, 16, 0, 0);

    const uint8_t* row = rows + kStageBytes * lane;
    const uint32_t sw = swizzle(lane);
    for (uint32_t st = 0; st < stages; ++st) {
        wait_vm_all();  // stage st is in LDS
        uint4 r[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) r[k] = *reinterpret_cast<const uint4*>(row + 16 * (k ^ sw));
        wait_lgkm_all();  // and in VGPRs: the buffer may be refilled
        const uint32_t nx = st + 1;
        if (nx < stages) {
            const uint32_t off = kStageBytes * nx;
            if (uniform && 2 * nx + 1 < nmax) {  // whole stage valid for every chunk
#pragma unroll
                for (int j = 0; j < kRowsPerLoad; ++j)
                    __builtin_amdgcn_global_load_lds(from[j] + off, rows + 1024 * j, 16, 0, 0);
            } else {
#pragma unroll
                for (int j = 0; j < kRowsPerLoad; ++j)
                    if (nx < until[j]) __builtin_amdgcn_global_load_lds(from[j] + off, rows + 1024 * j, 16, 0, 0);
            }
        }
        uint32_t W[16];
        if (2 * st < nfull) {
            words_from(r[0], r[1], r[2], r[3], W);
            compress(H, W);
        }
        if (2 * st + 1 < nfull) {
            words_from(r[4], r[5], r[6], r[7], W);
            compress(H, W);
        }
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
__device__ __forceinline__ void full_blocks_any(uint32_t H[8], const uint8_t* p, uint32_t nfull) {
    for (uint32_t b = 0; b < nfull; ++b) {
        uint32_t W[16];
        gather_words(p + 64 * (uint64_t)b, 64, W);
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

__global__ void __launch_bounds__(kThreads) sha256_leaves_kernel(const LeafDesc* __restrict__ desc, uint64_t n_slots,
                                                                 uint64_t out_bound, uint8_t* __restrict__ digests) {
    __shared__ __attribute__((aligned(16))) uint8_t stage[kWaves][64 * kStageBytes];
    const uint64_t slot = (uint64_t)blockIdx.x * kThreads + threadIdx.x;
    const bool live = slot < n_slots;
    LeafDesc d = {0, 0, 0};
    if (live) d = desc[slot];
    const uint8_t* p = reinterpret_cast<const uint8_t*>(d.src);
    const uint32_t nfull = (uint32_t)(d.nbytes >> 6);

    uint32_t H[8];
    init_state(H);
    if (__all((d.src & 15) == 0)) {
        const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        full_blocks_lds(H, d.src, nfull, stage[wave]);
    } else {
        full_blocks_any(H, p, nfull);
    }
    final_blocks(H, p + ((uint64_t)nfull << 6), (uint32_t)(d.nbytes & 63), d.nbytes);
    if (live && d.out < out_bound) store_digest(digests + 32 * d.out, H);
}

}  // namespace

hipError_t launch_sha256_leaves(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                                hipStream_t s) {
    for (uint64_t base = 0; base < n_slots; base += kMaxSlotsPerLaunch) {
        const uint64_t n = n_slots - base < kMaxSlotsPerLaunch ? n_slots - base : kMaxSlotsPerLaunch;
        sha256_leaves_kernel<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, s>>>(desc + base, n, out_bound,
                                                                                          digests);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace hv
