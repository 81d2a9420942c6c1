// merkle.hip -- segmented RFC 6962 Merkle Tree Hash, bottom-up, on the GPU
// (Algorithm 1's "construct Merkle tree from leaf_hashes using GPU").
//
// RFC 6962 section 2.1 defines MTH recursively, splitting n entries at the
// largest power of two below n.  Built bottom-up that is: level 0 holds the
// leaf hashes SHA-256(0x00 || d_i); each level pairs neighbours (2i, 2i+1)
// into SHA-256(0x01 || left || right) and moves an unpaired last node up
// unchanged.  (Node i of level j then covers entries [i*2^j, min((i+1)*2^j, n)),
// so the root's two children split exactly where the recursion splits.)
//
// A workgroup reduces a tile of up to 512 = 2^9 consecutive nodes of one
// segment by nine levels, to one node.  Tiles start at multiples of 512, so no
// pair ever straddles two tiles, and the tile's last unpaired node at any level
// is the segment's last node there -- the same promotion the whole tree
// makes.  One launch therefore takes every segment nine levels up; the host
// chains ceil(depth / 9) launches, the first of which also forms the leaf
// hashes as it loads the entries.  Level 1 is formed in registers from the
// two entries a thread loads; higher levels go through LDS, with idle waves
// waiting at the barriers.
#include "hv_kernels.h"
#include "sha256_device.h"

namespace hv {
namespace {

constexpr int kThreads = kTileNodes / 2;  // 256: each thread owns one pair of level 0

// SHA-256(0x00 || d): 33 bytes, one block.  d as big-endian words.
__device__ __forceinline__ void leaf_hash(const uint32_t d[8], uint32_t out[8]) {
    uint32_t W[16];
    W[0] = d[0] >> 8;
#pragma unroll
    for (int i = 1; i < 8; ++i) W[i] = (d[i - 1] << 24) | (d[i] >> 8);
    W[8] = (d[7] << 24) | 0x00800000u;
#pragma unroll
    for (int i = 9; i < 15; ++i) W[i] = 0;
    W[15] = 33 * 8;
    init_state(out);
    compress(out, W);
}

// SHA-256(0x01 || L || R): 65 bytes, two blocks.
__device__ __forceinline__ void node_hash(const uint32_t L[8], const uint32_t R[8], uint32_t out[8]) {
    uint32_t W[16];
    W[0] = 0x01000000u | (L[0] >> 8);
#pragma unroll
    for (int i = 1; i < 8; ++i) W[i] = (L[i - 1] << 24) | (L[i] >> 8);
    W[8] = (L[7] << 24) | (R[0] >> 8);
#pragma unroll
    for (int i = 1; i < 8; ++i) W[8 + i] = (R[i - 1] << 24) | (R[i] >> 8);
    init_state(out);
    compress(out, W);
    W[0] = (R[7] << 24) | 0x00800000u;
#pragma unroll
    for (int i = 1; i < 15; ++i) W[i] = 0;
    W[15] = 65 * 8;
    compress(out, W);
}

// SHA-256 of the empty string: the root of an empty segment.
__device__ __forceinline__ void empty_hash(uint32_t out[8]) {
    uint32_t W[16];
    W[0] = 0x80000000u;
#pragma unroll
    for (int i = 1; i < 16; ++i) W[i] = 0;
    init_state(out);
    compress(out, W);
}

__device__ __forceinline__ uint32_t find_segment(const uint64_t* __restrict__ tile_off, uint32_t n_seg, uint64_t tile) {
    uint32_t lo = 0, hi = n_seg;  // tile_off[lo] <= tile < tile_off[hi]
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (tile_off[mid] <= tile) lo = mid; else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(kThreads) merkle_tile_kernel(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                                               const uint64_t* __restrict__ in_off,
                                                               const uint64_t* __restrict__ tile_off, uint32_t n_seg,
                                                               uint64_t n_tiles, int leaf_mode) {
    __shared__ uint32_t lds[8][kThreads];  // word-major: node i's word w at lds[w][i]
    const uint32_t i = threadIdx.x;
    for (uint64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const uint32_t s = find_segment(tile_off, n_seg, tile);
        const uint64_t t = tile - tile_off[s];
        const uint64_t c = in_off[s + 1] - in_off[s];
        const uint64_t first = t * kTileNodes;
        const uint32_t cnt = c > first ? (uint32_t)(c - first < (uint64_t)kTileNodes ? c - first : kTileNodes) : 0u;
        const uint8_t* base = in + 32 * (in_off[s] + first);

        uint32_t P[8];
        uint32_t n;  // nodes held in lds after the first level
        if (cnt == 0) {  // empty segment (only ever a first-launch tile)
            if (i == 0) empty_hash(P);
            n = 1;
        } else {
            const bool hasA = 2 * i < cnt, hasB = 2 * i + 1 < cnt;
            uint32_t A[8], B[8];
            if (hasA) {
                load_digest(base + 64 * i, A);
                if (leaf_mode) { uint32_t T[8]; leaf_hash(A, T); for (int w = 0; w < 8; ++w) A[w] = T[w]; }
            }
            if (hasB) {
                load_digest(base + 64 * i + 32, B);
                if (leaf_mode) { uint32_t T[8]; leaf_hash(B, T); for (int w = 0; w < 8; ++w) B[w] = T[w]; }
                node_hash(A, B, P);
            } else if (hasA) {
                for (int w = 0; w < 8; ++w) P[w] = A[w];  // unpaired last node moves up
            }
            n = (cnt + 1) / 2;
        }
        if (i < n) for (int w = 0; w < 8; ++w) lds[w][i] = P[w];
        __syncthreads();
        while (n > 1) {
            const uint32_t m = (n + 1) / 2;
            if (i < m) {
                uint32_t L[8];
                for (int w = 0; w < 8; ++w) L[w] = lds[w][2 * i];
                if (2 * i + 1 < n) {
                    uint32_t R[8];
                    for (int w = 0; w < 8; ++w) R[w] = lds[w][2 * i + 1];
                    node_hash(L, R, P);
                } else {
                    for (int w = 0; w < 8; ++w) P[w] = L[w];
                }
            }
            __syncthreads();
            if (i < m) for (int w = 0; w < 8; ++w) lds[w][i] = P[w];
            __syncthreads();
            n = m;
        }
        if (i == 0) {
            uint32_t R[8];
            for (int w = 0; w < 8; ++w) R[w] = lds[w][0];
            store_digest(out + 32 * tile, R);
        }
        __syncthreads();  // lds is reused by the next tile
    }
}

}  // namespace

hipError_t launch_merkle_tiles(const uint8_t* in, uint8_t* out, const uint64_t* in_off, const uint64_t* tile_off,
                               uint32_t n_seg, uint64_t n_tiles, int leaf_mode, hipStream_t s) {
    if (n_tiles == 0) return hipSuccess;
    const uint64_t cap = 1u << 20;
    const unsigned grid = (unsigned)(n_tiles < cap ? n_tiles : cap);
    merkle_tile_kernel<<<grid, kThreads, 0, s>>>(in, out, in_off, tile_off, n_seg, n_tiles, leaf_mode);
    return hipGetLastError();
}

}  // namespace hv
