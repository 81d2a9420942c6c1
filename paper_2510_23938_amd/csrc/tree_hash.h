// tree_hash.h -- RFC 6962 node hashes (section 2.1) for the Merkle kernels,
// as policies over the hash: SHA-256 (32-byte nodes; an interior node is two
// blocks) and SHA-384 (48-byte nodes; leaf and interior nodes are one
// 128-byte block each).  A policy gives the node size (kWords big-endian
// 32-bit words, kBytes bytes), the leaf node H(0x00 || d), the interior node
// H(0x01 || L || R), the hash of the empty string (the root of an empty
// tree), and 16-byte-aligned loads and stores of a node.
#pragma once
#include "sha256_device.h"
#include "sha384_device.h"

namespace hv {

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
