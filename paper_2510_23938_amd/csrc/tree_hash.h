// tree_hash.h -- RFC 6962 node hashes (section 2.1) for the Merkle kernels,
// as policies over the hash: SHA-256 (32-byte nodes; an interior node is two
// blocks) and SHA-384 (48-byte nodes; leaf and interior nodes are one
// 128-byte block each).  A policy gives the node size (kWords big-endian
// 32-bit words, kBytes bytes), the leaf node H(0x00 || d), the interior node
// H(0x01 || L || R) (also in a form fed by a table in LDS, for kernels that
// stage it), the hash of the empty string (the root of an empty tree), and
// 16-byte-aligned loads and stores of a node.
#pragma once
#include "sha256_device.h"
#include "sha384_device.h"

namespace hv {

// The second block of a SHA-256 interior node holds one byte of data (the
// last byte of R), then the 0x80 pad byte, zeros and the bit length 520
// (FIPS 180-4 section 5.1.1), so its 64 expanded message words (section
// 6.2.2, step 1) depend on that byte alone.  In unrolled code words 16..30
// fold to a few operations; words 31..63, about a third of that block's
// VALU work, are taken from this table: word 31 + k for byte value v sits at
// w[k * 256 + v] (word-major, so a wave's 64 lookups of one word fall within
// one 1 KB row of LDS).  The table is built at compile time from the
// definition of the schedule.
struct NodeTailTable {
    static constexpr int kFirst = 31;
    static constexpr int kWords = (64 - kFirst) * 256;
    alignas(16) uint32_t w[kWords];
};

constexpr uint32_t tail_rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

constexpr NodeTailTable make_node_tail_table() {
    NodeTailTable t{};
    for (uint32_t v = 0; v < 256; ++v) {
        uint32_t W[64] = {};
        W[0] = (v << 24) | 0x00800000u;
        W[15] = 65 * 8;
        for (int i = 16; i < 64; ++i) {
            const uint32_t x = W[i - 15], y = W[i - 2];
            const uint32_t s0 = tail_rotr(x, 7) ^ tail_rotr(x, 18) ^ (x >> 3);
            const uint32_t s1 = tail_rotr(y, 17) ^ tail_rotr(y, 19) ^ (y >> 10);
            W[i] = s1 + W[i - 7] + s0 + W[i - 16];
        }
        for (int k = 0; k < 64 - NodeTailTable::kFirst; ++k) t.w[k * 256 + v] = W[NodeTailTable::kFirst + k];
    }
    return t;
}

__device__ constexpr NodeTailTable kNodeTail = make_node_tail_table();

struct Sha256Tree {
    static constexpr int kWords = 8;
    static constexpr int kBytes = 32;
    // SHA-256(0x00 || d): 33 bytes, one block.  d as big-endian words.
    static __device__ __forceinline__ void leaf_hash(const uint32_t d[8], uint32_t out[8]) {
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

    // Words of LDS a kernel sets aside for the node-tail table, and the copy
    // into them: every thread of the block takes part; the caller then
    // synchronises the block before the first node_hash with the table.
    static constexpr int kTableWords = NodeTailTable::kWords;
    static __device__ __forceinline__ void stage_table(uint32_t* lds) {
        const uint4* src = reinterpret_cast<const uint4*>(kNodeTail.w);
        uint4* dst = reinterpret_cast<uint4*>(lds);
        for (int i = threadIdx.x; i < kTableWords / 4; i += blockDim.x) dst[i] = src[i];
    }

    // SHA-256(0x01 || L || R) with the second block's schedule words 31..63
    // from the node-tail table in LDS (`tab`, staged by stage_table).
    static __device__ __forceinline__ void node_hash(const uint32_t L[8], const uint32_t R[8], uint32_t out[8],
                                                     const uint32_t* tab) {
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
        const uint32_t* col = tab + (R[7] & 0xffu);
        constexpr int F = NodeTailTable::kFirst;
        uint32_t a = out[0], b = out[1], c = out[2], d = out[3];
        uint32_t e = out[4], f = out[5], g = out[6], h = out[7];
#pragma unroll
        for (int t = 0; t < 64; ++t) {
            uint32_t w;
            if (t < 16) {
                w = W[t];
            } else if (t < F) {
                w = small_sigma1(W[(t - 2) & 15]) + W[(t - 7) & 15] + small_sigma0(W[(t - 15) & 15]) + W[t & 15];
                W[t & 15] = w;
            } else {
                w = col[(t - F) * 256];
            }
            const uint32_t t1 = h + kRound[t] + w + big_sigma1(e) + choose(e, f, g);
            const uint32_t t2 = big_sigma0(a) + majority(a, b, c);
            h = g; g = f; f = e; e = d + t1;
            d = c; c = b; b = a; a = t1 + t2;
        }
        out[0] += a; out[1] += b; out[2] += c; out[3] += d;
        out[4] += e; out[5] += f; out[6] += g; out[7] += h;
    }

    // SHA-256(0x01 || L || R): 65 bytes, two blocks.
    static __device__ __forceinline__ void node_hash(const uint32_t L[8], const uint32_t R[8], uint32_t out[8]) {
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
    static __device__ __forceinline__ void empty_hash(uint32_t out[8]) {
        uint32_t W[16];
        W[0] = 0x80000000u;
#pragma unroll
        for (int i = 1; i < 16; ++i) W[i] = 0;
        init_state(out);
        compress(out, W);
    }

    static __device__ __forceinline__ void load(const uint8_t* p, uint32_t D[8]) { load_digest(p, D); }
    static __device__ __forceinline__ void store(uint8_t* p, const uint32_t D[8]) { store_digest(p, D); }
};

// SHA-384 nodes (48 bytes): both SHA-384(0x00 || d) (49 bytes) and
// SHA-384(0x01 || L || R) (97 bytes) fit in one 128-byte block.
struct Sha384Tree {
    static constexpr int kWords = 12;
    static constexpr int kBytes = 48;
    // One block from 26 big-endian message words (the rest zero) and the bit
    // length of `len` bytes; the state's first six words as 12 digest words.
    static __device__ __forceinline__ void one_block(const uint32_t w32[26], uint32_t len, uint32_t out[12]) {
        uint64_t W[16];
#pragma unroll
        for (int k = 0; k < 13; ++k) W[k] = pack(w32[2 * k], w32[2 * k + 1]);
        W[13] = 0;
        W[14] = 0;
        W[15] = (uint64_t)len * 8;
        uint64_t H[8];
        init_state384(H);
        compress512(H, W);
#pragma unroll
        for (int i = 0; i < 6; ++i) {
            out[2 * i] = hi32(H[i]);
            out[2 * i + 1] = lo32(H[i]);
        }
    }
    static __device__ __forceinline__ void leaf_hash(const uint32_t d[12], uint32_t out[12]) {
        uint32_t w[26];
        w[0] = d[0] >> 8;
#pragma unroll
        for (int i = 1; i < 12; ++i) w[i] = (d[i - 1] << 24) | (d[i] >> 8);
        w[12] = (d[11] << 24) | 0x00800000u;
#pragma unroll
        for (int i = 13; i < 26; ++i) w[i] = 0;
        one_block(w, 49, out);
    }
    static __device__ __forceinline__ void node_hash(const uint32_t L[12], const uint32_t R[12], uint32_t out[12]) {
        uint32_t w[26];
        w[0] = 0x01000000u | (L[0] >> 8);
#pragma unroll
        for (int i = 1; i < 12; ++i) w[i] = (L[i - 1] << 24) | (L[i] >> 8);
        w[12] = (L[11] << 24) | (R[0] >> 8);
#pragma unroll
        for (int i = 1; i < 12; ++i) w[12 + i] = (R[i - 1] << 24) | (R[i] >> 8);
        w[24] = (R[11] << 24) | 0x00800000u;
        w[25] = 0;
        one_block(w, 97, out);
    }
    // No table: both SHA-384 node forms are one block of data-dependent words.
    static constexpr int kTableWords = 4;
    static __device__ __forceinline__ void stage_table(uint32_t*) {}
    static __device__ __forceinline__ void node_hash(const uint32_t L[12], const uint32_t R[12], uint32_t out[12],
                                                     const uint32_t*) {
        node_hash(L, R, out);
    }
    static __device__ __forceinline__ void empty_hash(uint32_t out[12]) {
        uint32_t w[26];
        w[0] = 0x80000000u;
#pragma unroll
        for (int i = 1; i < 26; ++i) w[i] = 0;
        one_block(w, 0, out);
    }
    static __device__ __forceinline__ void load(const uint8_t* p, uint32_t D[12]) { load_digest384(p, D); }
    static __device__ __forceinline__ void store(uint8_t* p, const uint32_t D[12]) {
        uint4* q = reinterpret_cast<uint4*>(p);
#pragma unroll
        for (int i = 0; i < 3; ++i)
            q[i] = make_uint4(bswap(D[4 * i]), bswap(D[4 * i + 1]), bswap(D[4 * i + 2]), bswap(D[4 * i + 3]));
    }
};

}  // namespace hv
