// sha256_device.h -- SHA-256 compression for gfx950 (CDNA4), one message per lane.
//
// FIPS 180-4 section 6.2.2 on 32-bit VALU operations only (this is not a dense
// contraction, so no matrix cores):
//   ROTR           -> v_alignbit_b32 (x, x, n)
//   Sigma/sigma    -> two or three alignbits, one v_bitop3_b32 (3-input XOR, 0x96)
//   Ch (e, f, g)   -> one v_bitop3_b32 (truth table 0xCA)
//   Maj (a, b, c)  -> one v_bitop3_b32 (truth table 0xE8)
//   sums           -> v_add3_u32 (the compiler fuses a + b + c)
// The bitop3 truth-table index of inputs (x, y, z) is x<<2 | y<<1 | z.
// The round constants are literals in fully unrolled code, so they sit in
// SGPRs (VOP3 has no literal operand on gfx950) and cost no VALU op.
#pragma once
#include <stdint.h>
#include <hip/hip_runtime.h>

namespace hv {

// FIPS 180-4 section 4.2.2: first 32 bits of the fractional parts of the cube
// roots of the first 64 primes.
__device__ constexpr uint32_t kRound[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u, 0xab1c5ed5u,
    0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u,
    0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u,
    0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u,
    0xa2bfe8a1u, 0xa81a664bu, 0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u,
};

// FIPS 180-4 section 5.3.3: first 32 bits of the fractional parts of the square
// roots of the first 8 primes.
__device__ constexpr uint32_t kInit[8] = {
    0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au, 0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u,
};

__device__ __forceinline__ uint32_t rotr(uint32_t x, uint32_t n) { return __builtin_amdgcn_alignbit(x, x, n); }
__device__ __forceinline__ uint32_t xor3(uint32_t x, uint32_t y, uint32_t z) {
    return __builtin_amdgcn_bitop3_b32(x, y, z, 0x96);
}
__device__ __forceinline__ uint32_t choose(uint32_t e, uint32_t f, uint32_t g) {
    return __builtin_amdgcn_bitop3_b32(e, f, g, 0xCA);
}
__device__ __forceinline__ uint32_t majority(uint32_t a, uint32_t b, uint32_t c) {
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0xE8);
}
__device__ __forceinline__ uint32_t big_sigma0(uint32_t a) { return xor3(rotr(a, 2), rotr(a, 13), rotr(a, 22)); }
__device__ __forceinline__ uint32_t big_sigma1(uint32_t e) { return xor3(rotr(e, 6), rotr(e, 11), rotr(e, 25)); }
__device__ __forceinline__ uint32_t small_sigma0(uint32_t x) { return xor3(rotr(x, 7), rotr(x, 18), x >> 3); }
__device__ __forceinline__ uint32_t small_sigma1(uint32_t x) { return xor3(rotr(x, 17), rotr(x, 19), x >> 10); }

__device__ __forceinline__ uint32_t bswap(uint32_t x) { return __builtin_bswap32(x); }

__device__ __forceinline__ void init_state(uint32_t H[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) H[i] = kInit[i];
}

// One block: H <- H + rounds(H, W).  W holds the 16 big-endian message words
// and is used as the ring for the message schedule (overwritten).
__device__ __forceinline__ void compress(uint32_t H[8], uint32_t W[16]) {
    uint32_t a = H[0], b = H[1], c = H[2], d = H[3];
    uint32_t e = H[4], f = H[5], g = H[6], h = H[7];
#pragma unroll
    for (int t = 0; t < 64; ++t) {
        uint32_t w;
        if (t < 16) {
            w = W[t];
        } else {
            w = small_sigma1(W[(t - 2) & 15]) + W[(t - 7) & 15] + small_sigma0(W[(t - 15) & 15]) + W[t & 15];
            W[t & 15] = w;
        }
        const uint32_t hkw = h + kRound[t] + w;
        const uint32_t t1 = hkw + big_sigma1(e) + choose(e, f, g);
        const uint32_t t2 = big_sigma0(a) + majority(a, b, c);
        h = g; g = f; f = e; e = d + t1;
        d = c; c = b; b = a; a = t1 + t2;
    }
    H[0] += a; H[1] += b; H[2] += c; H[3] += d;
    H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

// Digest bytes are the state words in big-endian order; store them as two
// 16-byte writes (dst must be 16-byte aligned).
__device__ __forceinline__ void store_digest(uint8_t* dst, const uint32_t H[8]) {
    uint4* p = reinterpret_cast<uint4*>(dst);
    p[0] = make_uint4(bswap(H[0]), bswap(H[1]), bswap(H[2]), bswap(H[3]));
    p[1] = make_uint4(bswap(H[4]), bswap(H[5]), bswap(H[6]), bswap(H[7]));
}

// Digest as 8 big-endian words from its 32 stored bytes (16-byte aligned).
__device__ __forceinline__ void load_digest(const uint8_t* src, uint32_t D[8]) {
    const uint4* p = reinterpret_cast<const uint4*>(src);
    const uint4 x = p[0], y = p[1];
    D[0] = bswap(x.x); D[1] = bswap(x.y); D[2] = bswap(x.z); D[3] = bswap(x.w);
    D[4] = bswap(y.x); D[5] = bswap(y.y); D[6] = bswap(y.z); D[7] = bswap(y.w);
}

}  // namespace hv
