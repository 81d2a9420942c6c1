// sha384_split.hip -- SHA-384 of every chunk for small leaf counts: the
// two-wave form of the SHA-384 leaf kernel, on the scheme of the SHA-256 one
// (sha256_split.hip).
//
// A chunk is one chain of 128-byte blocks, so with fewer chunks than the chip
// has lanes its time is that chain's latency, and a lone wave issues one
// instruction per ~4.6 cycles.  A producer wave loads each block one block
// ahead, builds its 16 64-bit message words (padding of FIPS 180-4 section
// 5.1.2: tail, 0x80, zeros, 128-bit bit length) and expands them to the 80
// schedule words (section 6.4 step 1) in a double-buffered LDS area; a
// consumer wave runs only the 80 rounds and the feed-forward.  That moves
// about 1250 of the 3416 operations per block off the consumer's path.
//
// Synchronisation, exec mask and placement are as in the SHA-256 kernel: both
// waves of a pair run the same number of barriers (the workgroup's most
// blocks), one per block; the barrier orders LDS only; every lane runs every
// block (dead lanes and finished chunks on zeros or stale words) and only the
// loads, the state update and the digest store are per lane; one pair per
// workgroup up to 64 chunks per CU, two up to 128.  The schedule takes
// 80 x 8 bytes per lane per buffer: 80 KB per pair, so a two-pair workgroup
// fills the CU's 160 KB of LDS.
#include "hv_kernels.h"
#include "sha384_device.h"
#include "split_common.h"

namespace hv {
namespace {

constexpr int kGroups = 40;  // 80 schedule words, two per 16-byte LDS entry

__device__ __forceinline__ uint32_t block_valid(uint32_t nfull, uint32_t r, uint32_t b) {
    return b < nfull ? 128u : (b == nfull ? r : 0u);
}

// Block b's bytes into D, as in the SHA-256 kernel: kAligned (16-byte aligned
// chunk) loads the 16-byte granules holding chunk bytes into D[0..31] (D[32]
// is left as it is: with sh = 0 it does not enter the words), otherwise the
// aligned dwords holding chunk bytes into D[0..32]; the others are zero.  An
// aligned granule or dword holding a chunk byte lies in that byte's page.
template <bool kAligned>
__device__ __forceinline__ void load_block(uint64_t src, uint32_t valid, uint32_t b, uint32_t D[33]) {
    if constexpr (kAligned) {
        const gquads q = reinterpret_cast<gquads>(src + 128 * (uint64_t)b);
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if ((uint32_t)(16 * g) < valid) v = q[g];
            D[4 * g] = v.x; D[4 * g + 1] = v.y; D[4 * g + 2] = v.z; D[4 * g + 3] = v.w;
        }
    } else {
        const uint32_t sh = (uint32_t)(src & 3);
        const gwords w = reinterpret_cast<gwords>(src + 128 * (uint64_t)b - sh);
#pragma unroll
        for (int k = 0; k < 33; ++k) D[k] = (uint32_t)(4 * k) < sh + valid ? w[k] : 0u;
    }
}

// The 16 message words of a whole block.
__device__ __forceinline__ void whole_block_words(const uint32_t D[33], uint32_t sh, uint64_t W[16]) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
        W[i] = be64(__builtin_amdgcn_alignbyte(D[2 * i + 1], D[2 * i], sh),
                    __builtin_amdgcn_alignbyte(D[2 * i + 2], D[2 * i + 1], sh));
}

// The 16 message words of block b of a chunk of `total` bytes with nfull
// whole blocks and r tail bytes: a whole block, the tail block (and the bit
// length when r <= 111), or the length-only block after a longer tail.
__device__ __forceinline__ void block_words(const uint32_t D[33], uint32_t sh, uint64_t total, uint32_t nfull,
                                            uint32_t r, uint32_t b, uint64_t W[16]) {
    const uint32_t valid = block_valid(nfull, r, b);
    uint32_t X[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
        const uint32_t x = __builtin_amdgcn_alignbyte(D[i + 1], D[i], sh);
        const int nv = (int)valid - 4 * i;  // bytes of the chunk in dword i
        const uint32_t keep = nv >= 4 ? 0xffffffffu : (nv <= 0 ? 0u : (1u << (8 * nv)) - 1u);
        const uint32_t pad = (b == nfull && nv >= 0 && nv < 4) ? (0x80u << (8 * nv)) : 0u;
        X[i] = (x & keep) | pad;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) W[i] = be64(X[2 * i], X[2 * i + 1]);
    if (b == nfull + (r <= 111 ? 0u : 1u)) {
        W[14] = total >> 61;
        W[15] = total << 3;
    }
}

// Two 64-bit words as one 16-byte LDS entry, and back.
__device__ __forceinline__ uint4 entry(uint64_t w0, uint64_t w1) {
    return make_uint4(lo32(w0), hi32(w0), lo32(w1), hi32(w1));
}

// Producer: issue block b + 1's loads into `nxt`, build block b's 80
// schedule words from `cur` into `buf` (16 message words, then four trips of
// 16 expanded words), meet the consumer at the barrier.
template <bool kAligned>
__device__ __forceinline__ void produce(uint32_t b, uint64_t src, uint64_t total, uint32_t nfull, uint32_t r,
                                        uint32_t nblk, uint32_t nfull_min, uint32_t lane, uint4 (*buf)[64],
                                        const uint32_t cur[33], uint32_t nxt[33]) {
    const uint32_t sh = kAligned ? 0u : (uint32_t)(src & 3);
    // `cur` has landed (its loads were issued one block ago); waiting here,
    // before the next loads, keeps the compiler from waiting for those too
    wait_vmem();
    if (b + 1 < nblk) load_block<kAligned>(src, block_valid(nfull, r, b + 1), b + 1, nxt);
    uint64_t W[16];
    if (b < nfull_min)  // wave-uniform: a whole block on every lane
        whole_block_words(cur, sh, W);
    else
        block_words(cur, sh, total, nfull, r, b, W);
#pragma unroll
    for (int g = 0; g < 8; ++g) buf[g][lane] = entry(W[2 * g], W[2 * g + 1]);
#pragma nounroll
    for (int trip = 1; trip < 5; ++trip) {
#pragma unroll
        for (int i = 0; i < 16; ++i)
            W[i] = small_sigma1_512(W[(i + 14) & 15]) + W[(i + 9) & 15] + small_sigma0_512(W[(i + 1) & 15]) + W[i];
#pragma unroll
        for (int g = 0; g < 8; ++g) buf[8 * trip + g][lane] = entry(W[2 * g], W[2 * g + 1]);
    }
    lds_barrier();  // block b's words are in buf
}

template <bool kAligned>
__device__ __forceinline__ void produce_all(uint64_t src, uint64_t total, uint32_t nfull, uint32_t r, uint32_t nblk,
                                            uint32_t nmax, uint32_t nfull_min, uint32_t lane,
                                            uint4 (*sched)[kGroups][64]) {
    uint32_t A[33], B[33];
#pragma unroll
    for (int k = 0; k < 33; ++k) A[k] = B[k] = 0;
    if (0 < nblk) load_block<kAligned>(src, block_valid(nfull, r, 0), 0, A);
    for (uint32_t b = 0; b < nmax; b += 2) {
        produce<kAligned>(b, src, total, nfull, r, nblk, nfull_min, lane, sched[0], A, B);
        if (b + 1 < nmax) produce<kAligned>(b + 1, src, total, nfull, r, nblk, nfull_min, lane, sched[1], B, A);
    }
}

template <int kPairs>
__global__ void __launch_bounds__(128 * kPairs) sha384_split_kernel(const LeafDesc* __restrict__ desc,
                                                                    uint64_t n_slots, uint64_t out_bound,
                                                                    uint8_t* __restrict__ digests) {
    // [pair][buffer][entry of two words][lane]
    __shared__ uint4 sched[kPairs][2][kGroups][64];
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t pair = wave >> 1;
    const uint64_t base = (uint64_t)blockIdx.x * (64 * kPairs);
    const uint64_t slot = base + 64 * pair + lane;
    const bool live = slot < n_slots;
    LeafDesc d = {0, 0, 0};
    if (live) d = desc[slot];
    const uint32_t nfull = (uint32_t)(d.nbytes >> 7);
    const uint32_t r = (uint32_t)(d.nbytes & 127);
    const uint32_t nblk = live ? nfull + (r <= 111 ? 1u : 2u) : 0u;
    // every wave of the workgroup runs the same number of barriers: the most
    // blocks of any of its chunks
    uint32_t nmax = nblk;
    const uint64_t other = base + 64 * (pair ^ 1) + lane;
    if (kPairs == 2 && other < n_slots) {
        const uint64_t ob = desc[other].nbytes;
        const uint32_t on = (uint32_t)(ob >> 7) + ((ob & 127) <= 111 ? 1u : 2u);
        nmax = on > nmax ? on : nmax;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t x = __shfl_xor(nmax, o);
        nmax = x > nmax ? x : nmax;
    }
    nmax = __builtin_amdgcn_readfirstlane(nmax);

    if ((wave & 1) == 0) {
        uint32_t nfull_min = live ? nfull : 0xffffffffu;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const uint32_t x = __shfl_xor(nfull_min, o);
            nfull_min = x < nfull_min ? x : nfull_min;
        }
        nfull_min = __builtin_amdgcn_readfirstlane(nfull_min);
        if (__all((d.src & 15) == 0))
            produce_all<true>(d.src, d.nbytes, nfull, r, nblk, nmax, nfull_min, lane, sched[pair]);
        else
            produce_all<false>(d.src, d.nbytes, nfull, r, nblk, nmax, nfull_min, lane, sched[pair]);
    } else {
        uint64_t H[8];
        init_state384(H);
        for (uint32_t b = 0; b < nmax; ++b) {
            lds_barrier();  // block b's words are in buffer b % 2
            uint4(*buf)[64] = sched[pair][b & 1];
            uint64_t s[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) s[i] = H[i];
            // the words in five groups of 16 (eight entries): group j + 1's
            // reads are issued before group j's rounds; the scheduling barrier
            // keeps the compiler from moving each read next to its use, where
            // its latency would stall the rounds
            uint4 q[2][8];
#pragma unroll
            for (int e = 0; e < 8; ++e) q[0][e] = buf[e][lane];
#pragma unroll
            for (int j = 0; j < kGroups / 8; ++j) {
                if (j + 1 < kGroups / 8) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) q[(j + 1) & 1][e] = buf[8 * (j + 1) + e][lane];
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint64_t w2[2] = {pack(q[j & 1][e].y, q[j & 1][e].x), pack(q[j & 1][e].w, q[j & 1][e].z)};
#pragma unroll
                    for (int k = 0; k < 2; ++k) {
                        const int t = 16 * j + 2 * e + k;
                        round512(s[(8 - t) & 7], s[(9 - t) & 7], s[(10 - t) & 7], s[(11 - t) & 7],
                                 s[(12 - t) & 7], s[(13 - t) & 7], s[(14 - t) & 7], s[(15 - t) & 7], kRound512[t],
                                 w2[k]);
                    }
                }
            }
            const bool on = b < nblk;
#pragma unroll
            for (int i = 0; i < 8; ++i) H[i] = on ? H[i] + s[i] : H[i];
        }
        if (live && d.out < out_bound) store_digest384(digests + 48 * d.out, H);
    }
}

}  // namespace

hipError_t launch_sha384_auto(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                              hipStream_t s, bool background) {
    const int k = leaf_kernel_for(n_slots, background);  // the same rule as SHA-256's
    if (k == 1) return launch_sha384_leaves(desc, n_slots, out_bound, digests, s);
    return launch_sha384_split(desc, n_slots, out_bound, digests, k == 3, s);
}

hipError_t launch_sha384_split(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                               bool two_pairs, hipStream_t s) {
    for (uint64_t base = 0; base < n_slots; base += kMaxSlotsPerLaunch) {
        const uint64_t n = n_slots - base < kMaxSlotsPerLaunch ? n_slots - base : kMaxSlotsPerLaunch;
        if (!two_pairs)
            sha384_split_kernel<1><<<(unsigned)((n + 63) / 64), 128, 0, s>>>(desc + base, n, out_bound, digests);
        else
            sha384_split_kernel<2><<<(unsigned)((n + 127) / 128), 256, 0, s>>>(desc + base, n, out_bound, digests);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace hv
