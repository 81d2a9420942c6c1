// sha256_split.hip -- SHA-256 of every chunk for small leaf counts: two waves
// per 64 chunks, so that one chunk's chain of blocks runs faster.
//
// With fewer chunks than the chip has lanes, the leaf kernel is latency-bound:
// a chunk is one sequential chain of compressions on one lane, and a lone wave
// issues about one instruction every four cycles.  Here the message schedule
// (48 words x 10 operations per block, FIPS 180-4 section 6.2.2 step 1) moves
// to a second wave: wave 0 builds each block's 64 schedule words -- message
// words, padding (section 5.1.1) and expansion -- into LDS, and wave 1 runs
// only the 64 rounds and the feed-forward, reading the words from LDS.  The
// rounds' dependent path per block shrinks from about 1400 to about 900
// instructions, while wave 0 prepares the next block on another SIMD.
//
// Synchronisation: the two waves hold the same 64 descriptors and compute the
// same block count (the wave maximum), and each executes exactly one barrier
// per block: wave 0 after writing block b's words into buffer b % 2, wave 1
// before reading them.  Wave 0 refills buffer b % 2 only after the barrier
// of block b + 1, which wave 1 reaches after its last read of block b.
// Wave 0 loads each block's bytes one block ahead, so the load latency runs
// under the previous block's expansion and the barrier wait.
//
// Exec mask: on gfx950 a wave whose rounds run with most lanes masked off is
// much slower per instruction than a full one (measured: 16 or fewer active
// lanes take about 1.6x as long per block as 32 or 64).  So every lane runs
// every block's expansion and rounds, also dead lanes and lanes past their
// last block (on zeros or stale words); only the loads, the state update
// (a select) and the digest store are per lane.
#include "hv_kernels.h"
#include "sha256_device.h"
#include "split_common.h"

#include <atomic>

namespace hv {
namespace {

// A workgroup holds kPairs producer/consumer pairs (1 or 2): waves 2p build
// schedules, waves 2p + 1 run rounds.  Up to 64 chunks per CU one pair per
// workgroup is slightly faster (a two-wave barrier); up to 128 two pairs keep
// one workgroup, and so one wave per SIMD, on each CU.
constexpr int kMaxPairs = 2;
constexpr int kMaxDevices = 64;

// The aligned dwords under block b of a chunk at p with nfull whole blocks and
// r tail bytes: only those holding at least one byte of the chunk are loaded
// (the others are zero), so no access leaves the pages the chunk touches.
// sh = p & 3, the same for every block of the chunk.
__device__ __forceinline__ uint32_t block_valid(uint32_t nfull, uint32_t r, uint32_t b) {
    return b < nfull ? 64u : (b == nfull ? r : 0u);
}

// Block b's bytes into D.  kAligned (the chunk starts on a 16-byte boundary):
// the 16-byte granules that hold chunk bytes, with four 16-byte loads, into
// D[0..15] (D[16] is left as it is: with sh = 0 it does not enter the words).
// Otherwise the aligned dwords that hold chunk bytes, into D[0..16].  The
// others are zero.  An aligned granule or dword holding a chunk byte lies in
// the same page as that byte, so no access leaves the pages the chunk touches.
template <bool kAligned>
__device__ __forceinline__ void load_block(uint64_t src, uint32_t valid, uint32_t b, uint32_t D[17]) {
    if constexpr (kAligned) {
        const gquads q = reinterpret_cast<gquads>(src + 64 * (uint64_t)b);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if ((uint32_t)(16 * g) < valid) v = q[g];
            D[4 * g] = v.x; D[4 * g + 1] = v.y; D[4 * g + 2] = v.z; D[4 * g + 3] = v.w;
        }
    } else {
        const uint32_t sh = (uint32_t)(src & 3);
        const gwords w = reinterpret_cast<gwords>(src + 64 * (uint64_t)b - sh);
#pragma unroll
        for (int k = 0; k < 17; ++k) D[k] = (uint32_t)(4 * k) < sh + valid ? w[k] : 0u;
    }
}

// The 16 message words (big-endian) of block b from its dwords: a whole
// block, the tail block (tail, 0x80, zeros, and the bit length when r <= 55),
// or the length-only block that follows a tail of more than 55 bytes.
__device__ __forceinline__ void block_words(const uint32_t D[17], uint32_t sh, uint64_t total, uint32_t nfull,
                                            uint32_t r, uint32_t b, uint32_t W[16]) {
    const uint32_t valid = block_valid(nfull, r, b);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const uint32_t x = __builtin_amdgcn_alignbyte(D[i + 1], D[i], sh);
        const int nv = (int)valid - 4 * i;  // bytes of the chunk in word i
        const uint32_t keep = nv >= 4 ? 0xffffffffu : (nv <= 0 ? 0u : (1u << (8 * nv)) - 1u);
        const uint32_t pad = (b == nfull && nv >= 0 && nv < 4) ? (0x80u << (8 * nv)) : 0u;
        W[i] = bswap((x & keep) | pad);
    }
    const bool last = b == nfull + (r <= 55 ? 0u : 1u);
    if (last) {
        const uint64_t bits = total * 8;
        W[14] = (uint32_t)(bits >> 32);
        W[15] = (uint32_t)bits;
    }
}

// The words of a whole block (no padding, no length).
__device__ __forceinline__ void whole_block_words(const uint32_t D[17], uint32_t sh, uint32_t W[16]) {
#pragma unroll
    for (int i = 0; i < 16; ++i) W[i] = bswap(__builtin_amdgcn_alignbyte(D[i + 1], D[i], sh));
}

// Wave 0's work for block b: issue the loads of block b + 1 into `nxt`, build
// block b's 64 schedule words from `cur` into `buf`, then meet wave 1 at the
// barrier.
template <bool kAligned>
__device__ __forceinline__ void produce(uint32_t b, uint64_t src, uint64_t total, uint32_t nfull, uint32_t r,
                                        uint32_t nblk, uint32_t nfull_min, uint32_t lane, uint4 (*buf)[64],
                                        const uint32_t cur[17], uint32_t nxt[17]) {
    const uint32_t sh = kAligned ? 0u : (uint32_t)(src & 3);
    // `cur` has landed (its loads were issued one block ago); waiting here, on
    // every path and before the next loads, keeps the compiler from placing a
    // wait for them where it would also wait for the loads issued below
    wait_vmem();
    if (b + 1 < nblk) load_block<kAligned>(src, block_valid(nfull, r, b + 1), b + 1, nxt);
    {  // every lane, also past its last block: see the kernel's comment on exec
        uint32_t W[16];
        if (b < nfull_min)  // wave-uniform: a whole block on every lane
            whole_block_words(cur, sh, W);
        else
            block_words(cur, sh, total, nfull, r, b, W);
#pragma unroll
        for (int g = 0; g < 4; ++g) buf[g][lane] = make_uint4(W[4 * g], W[4 * g + 1], W[4 * g + 2], W[4 * g + 3]);
#pragma unroll
        for (int g = 4; g < 16; ++g) {
            uint32_t x[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int t = 4 * g + k;
                const uint32_t w = small_sigma1(W[(t - 2) & 15]) + W[(t - 7) & 15] + small_sigma0(W[(t - 15) & 15]) +
                                   W[t & 15];
                W[t & 15] = w;
                x[k] = w;
            }
            buf[g][lane] = make_uint4(x[0], x[1], x[2], x[3]);
        }
    }
    lds_barrier();  // block b's words are in buf
}

// All of wave 0's blocks.  Two register sets take turns: block b + 1 loads
// into one while block b is built from the other, so the loads run under the
// expansion and the barrier wait, and no copy waits on them.
template <bool kAligned>
__device__ __forceinline__ void produce_all(uint64_t src, uint64_t total, uint32_t nfull, uint32_t r, uint32_t nblk,
                                            uint32_t nmax, uint32_t nfull_min, uint32_t lane, uint4 (*sched)[16][64]) {
    uint32_t A[17], B[17];
#pragma unroll
    for (int k = 0; k < 17; ++k) A[k] = B[k] = 0;
    if (0 < nblk) load_block<kAligned>(src, block_valid(nfull, r, 0), 0, A);
    for (uint32_t b = 0; b < nmax; b += 2) {
        produce<kAligned>(b, src, total, nfull, r, nblk, nfull_min, lane, sched[0], A, B);
        if (b + 1 < nmax) produce<kAligned>(b + 1, src, total, nfull, r, nblk, nfull_min, lane, sched[1], B, A);
    }
}

// The 64 rounds of one block on its schedule words q (FIPS 180-4 section
// 6.2.2 steps 2-4); the feed-forward only where `on` (the lane still has
// blocks).
__device__ __forceinline__ void rounds(uint32_t H[8], const uint4 q[16], bool on) {
    uint32_t s[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = H[i];
#pragma unroll
    for (int g = 0; g < 16; ++g) {
        const uint32_t w4[4] = {q[g].x, q[g].y, q[g].z, q[g].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int t = 4 * g + k;
            uint32_t& a = s[(8 - t) & 7];
            uint32_t& bb = s[(9 - t) & 7];
            uint32_t& c = s[(10 - t) & 7];
            uint32_t& dd = s[(11 - t) & 7];
            uint32_t& e = s[(12 - t) & 7];
            uint32_t& f = s[(13 - t) & 7];
            uint32_t& gg = s[(14 - t) & 7];
            uint32_t& h = s[(15 - t) & 7];
            const uint32_t t1 = h + kRound[t] + w4[k] + big_sigma1(e) + choose(e, f, gg);
            const uint32_t t2 = big_sigma0(a) + majority(a, bb, c);
            dd += t1;     // the new e
            h = t1 + t2;  // the new a
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) H[i] = on ? H[i] + s[i] : H[i];
}

// The consumer's work for block b: pass the barrier of block b + 1 and issue
// the reads of its words into `nxt`, then run block b's rounds on `cur`, so
// the reads land under the rounds.
__device__ __forceinline__ void consume(uint32_t b, uint32_t nmax, uint32_t nblk, uint32_t lane,
                                        uint4 (*sched)[16][64], uint32_t H[8], const uint4 cur[16], uint4 nxt[16]) {
    // `cur` has landed (read one block ago); waiting here, on every path and
    // before the next reads, keeps the compiler from placing a wait for it
    // where it would also wait for the reads issued below
    wait_lds();
    if (b + 1 < nmax) {
        lds_barrier();  // block b + 1's words are in buffer (b + 1) % 2
#pragma unroll
        for (int g = 0; g < 16; ++g) nxt[g] = sched[(b + 1) & 1][g][lane];
    }
    rounds(H, cur, b < nblk);
}

template <int kPairs>
__global__ void __launch_bounds__(128 * kPairs) sha256_split_kernel(const LeafDesc* __restrict__ desc,
                                                                    uint64_t n_slots, uint64_t out_bound,
                                                                    uint8_t* __restrict__ digests) {
    // [pair][buffer][group of four words][lane]: lane-consecutive 16-byte entries
    __shared__ uint4 sched[kPairs][2][16][64];
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t pair = wave >> 1;
    const uint64_t base = (uint64_t)blockIdx.x * (64 * kPairs);
    const uint64_t slot = base + 64 * pair + lane;
    const bool live = slot < n_slots;
    LeafDesc d = {0, 0, 0};
    if (live) d = desc[slot];
    const uint32_t nfull = (uint32_t)(d.nbytes >> 6);
    const uint32_t r = (uint32_t)(d.nbytes & 63);
    const uint32_t nblk = live ? nfull + (r <= 55 ? 1u : 2u) : 0u;
    // every wave of the workgroup runs the same number of barriers: the most
    // blocks of any of its 128 chunks
    const uint64_t other = base + 64 * (pair ^ 1) + lane;
    uint32_t nmax = nblk;
    if (kPairs == 2 && other < n_slots) {
        const uint64_t ob = desc[other].nbytes;
        const uint32_t on = (uint32_t)(ob >> 6) + ((ob & 63) <= 55 ? 1u : 2u);
        nmax = on > nmax ? on : nmax;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t x = __shfl_xor(nmax, o);
        nmax = x > nmax ? x : nmax;
    }
    nmax = __builtin_amdgcn_readfirstlane(nmax);

    if ((wave & 1) == 0) {
        // the fewest whole blocks of any live lane of the wave (wave-uniform)
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
        uint32_t H[8];
        init_state(H);
        // two register sets take turns: block b + 1's words are read into one
        // while block b's rounds run on the other
        uint4 A[16], B[16];
        if (nmax > 0) {
            lds_barrier();  // block 0's words are in buffer 0
#pragma unroll
            for (int g = 0; g < 16; ++g) A[g] = sched[pair][0][g][lane];
        }
        for (uint32_t b = 0; b < nmax; b += 2) {
            consume(b, nmax, nblk, lane, sched[pair], H, A, B);
            if (b + 1 < nmax) consume(b + 1, nmax, nblk, lane, sched[pair], H, B, A);
        }
        if (live && d.out < out_bound) store_digest(digests + 32 * d.out, H);
    }
}

}  // namespace

// Compute units of the current device, queried once per device.
uint32_t device_cus() {
    static std::atomic<int> cus[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
        cus[dev].store(n, std::memory_order_relaxed);
    }
    return (uint32_t)n;
}

int leaf_kernel_for(uint64_t n_slots, bool background) {
    const int choice = leaf_kernel_choice();
    const uint64_t cus = device_cus();
    // the two-wave kernel while every CU holds one workgroup at most (two
    // pairs: four waves on the CU's four SIMDs); with more, a CU's SIMDs would
    // each run two waves and the one-wave kernel is faster.  Background work
    // keeps the one-wave kernel: the two-wave kernel spends two waves per 64
    // chunks to shorten each chain, about 1.3x the CU time per byte.
    if (choice == 1 || (choice == 0 && (background || n_slots > 64 * kMaxPairs * cus))) return 1;
    return choice == 3 || n_slots > 64 * cus ? 3 : 2;
}

hipError_t launch_sha256_auto(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                              hipStream_t s, bool background) {
    const int k = leaf_kernel_for(n_slots, background);
    if (k == 1) return launch_sha256_leaves(desc, n_slots, out_bound, digests, s);
    return launch_sha256_split(desc, n_slots, out_bound, digests, k == 3, s);
}

hipError_t launch_sha256_split(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                               bool two_pairs, hipStream_t s) {
    for (uint64_t base = 0; base < n_slots; base += kMaxSlotsPerLaunch) {
        const uint64_t n = n_slots - base < kMaxSlotsPerLaunch ? n_slots - base : kMaxSlotsPerLaunch;
        if (!two_pairs)
            sha256_split_kernel<1><<<(unsigned)((n + 63) / 64), 128, 0, s>>>(desc + base, n, out_bound, digests);
        else
            sha256_split_kernel<2><<<(unsigned)((n + 127) / 128), 256, 0, s>>>(desc + base, n, out_bound, digests);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace hv
