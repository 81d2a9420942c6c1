// sha384_device.h -- SHA-384 compression for gfx950, one message per lane.
//
// FIPS 180-4 section 6.5: the SHA-512 computation of section 6.4 (80 rounds
// on 64-bit words, 1024-bit blocks) from SHA-384's own initial value, with
// the digest truncated to the first six state words.  gfx950's VALU is 32
// bits wide, so each 64-bit word is a pair of 32-bit halves:
//   ROTR^n          -> two v_alignbit_b32 (the halves swap roles for n >= 32)
//   3-input XOR     -> one v_bitop3_b32 per half (truth table 0x96)
//   Ch / Maj        -> one v_bitop3_b32 per half (0xCA / 0xE8)
//   addition mod 2^64 -> the compiler's 64-bit add (carry between halves)
#pragma once
#include <stdint.h>
#include <hip/hip_runtime.h>

namespace hv {

// FIPS 180-4 section 4.2.3: first 64 bits of the fractional parts of the cube
// roots of the first 80 primes.
__device__ constexpr uint64_t kRound512[80] = {
    0x428a2f98d728ae22ull, 0x7137449123ef65cdull, 0xb5c0fbcfec4d3b2full, 0xe9b5dba58189dbbcull,
    0x3956c25bf348b538ull, 0x59f111f1b605d019ull, 0x923f82a4af194f9bull, 0xab1c5ed5da6d8118ull,
    0xd807aa98a3030242ull, 0x12835b0145706fbeull, 0x243185be4ee4b28cull, 0x550c7dc3d5ffb4e2ull,
    0x72be5d74f27b896full, 0x80deb1fe3b1696b1ull, 0x9bdc06a725c71235ull, 0xc19bf174cf692694ull,
    0xe49b69c19ef14ad2ull, 0xefbe4786384f25e3ull, 0x0fc19dc68b8cd5b5ull, 0x240ca1cc77ac9c65ull,
    0x2de92c6f592b0275ull, 0x4a7484aa6ea6e483ull, 0x5cb0a9dcbd41fbd4ull, 0x76f988da831153b5ull,
    0x983e5152ee66dfabull, 0xa831c66d2db43210ull, 0xb00327c898fb213full, 0xbf597fc7beef0ee4ull,
    0xc6e00bf33da88fc2ull, 0xd5a79147930aa725ull, 0x06ca6351e003826full, 0x142929670a0e6e70ull,
    0x27b70a8546d22ffcull, 0x2e1b21385c26c926ull, 0x4d2c6dfc5ac42aedull, 0x53380d139d95b3dfull,
    0x650a73548baf63deull, 0x766a0abb3c77b2a8ull, 0x81c2c92e47edaee6ull, 0x92722c851482353bull,
    0xa2bfe8a14cf10364ull, 0xa81a664bbc423001ull, 0xc24b8b70d0f89791ull, 0xc76c51a30654be30ull,
    0xd192e819d6ef5218ull, 0xd69906245565a910ull, 0xf40e35855771202aull, 0x106aa07032bbd1b8ull,
    0x19a4c116b8d2d0c8ull, 0x1e376c085141ab53ull, 0x2748774cdf8eeb99ull, 0x34b0bcb5e19b48a8ull,
    0x391c0cb3c5c95a63ull, 0x4ed8aa4ae3418acbull, 0x5b9cca4f7763e373ull, 0x682e6ff3d6b2b8a3ull,
    0x748f82ee5defb2fcull, 0x78a5636f43172f60ull, 0x84c87814a1f0ab72ull, 0x8cc702081a6439ecull,
    0x90befffa23631e28ull, 0xa4506cebde82bde9ull, 0xbef9a3f7b2c67915ull, 0xc67178f2e372532bull,
    0xca273eceea26619cull, 0xd186b8c721c0c207ull, 0xeada7dd6cde0eb1eull, 0xf57d4f7fee6ed178ull,
    0x06f067aa72176fbaull, 0x0a637dc5a2c898a6ull, 0x113f9804bef90daeull, 0x1b710b35131c471bull,
    0x28db77f523047d84ull, 0x32caab7b40c72493ull, 0x3c9ebe0a15c9bebcull, 0x431d67c49c100d4cull,
    0x4cc5d4becb3e42b6ull, 0x597f299cfc657e2aull, 0x5fcb6fab3ad6faecull, 0x6c44198c4a475817ull,
};

// FIPS 180-4 section 5.3.4: first 64 bits of the fractional parts of the square
// roots of the ninth through sixteenth primes.
__device__ constexpr uint64_t kInit384[8] = {
    0xcbbb9d5dc1059ed8ull, 0x629a292a367cd507ull, 0x9159015a3070dd17ull, 0x152fecd8f70e5939ull,
    0x67332667ffc00b31ull, 0x8eb44a8768581511ull, 0xdb0c2e0d64f98fa7ull, 0x47b5481dbefa4fa4ull,
};

__device__ __forceinline__ uint32_t hi32(uint64_t x) { return (uint32_t)(x >> 32); }
__device__ __forceinline__ uint32_t lo32(uint64_t x) { return (uint32_t)x; }
// A 64-bit word from its halves, built as a bit cast of a two-dword vector so
// that it stays one register pair: written as (hi << 32) | lo, the compiler
// splits later 64-bit additions into a zero-extended low part and a shifted
// high part (two v_lshl_add_u64 and a v_mov where one add suffices), about a
// quarter more VALU work per block.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint64_t pack(uint32_t hi, uint32_t lo) {
    const u32x2 v = {lo, hi};
    return __builtin_bit_cast(uint64_t, v);
}

template <int N>
__device__ __forceinline__ uint64_t rotr64(uint64_t x) {
    static_assert(N > 0 && N < 64 && N != 32, "rotate amount");
    const uint32_t h = hi32(x), l = lo32(x);
    if (N < 32) return pack(__builtin_amdgcn_alignbit(l, h, N), __builtin_amdgcn_alignbit(h, l, N));
    return pack(__builtin_amdgcn_alignbit(h, l, N - 32), __builtin_amdgcn_alignbit(l, h, N - 32));
}

template <int N>
__device__ __forceinline__ uint64_t shr64(uint64_t x) {
    static_assert(N > 0 && N < 32, "shift amount");
    return pack(hi32(x) >> N, __builtin_amdgcn_alignbit(hi32(x), lo32(x), N));
}

template <int TT>
__device__ __forceinline__ uint64_t bitop3_64(uint64_t x, uint64_t y, uint64_t z) {
    return pack(__builtin_amdgcn_bitop3_b32(hi32(x), hi32(y), hi32(z), TT),
                __builtin_amdgcn_bitop3_b32(lo32(x), lo32(y), lo32(z), TT));
}

__device__ __forceinline__ uint64_t big_sigma0_512(uint64_t a) {
    return bitop3_64<0x96>(rotr64<28>(a), rotr64<34>(a), rotr64<39>(a));
}
__device__ __forceinline__ uint64_t big_sigma1_512(uint64_t e) {
    return bitop3_64<0x96>(rotr64<14>(e), rotr64<18>(e), rotr64<41>(e));
}
__device__ __forceinline__ uint64_t small_sigma0_512(uint64_t x) {
    return bitop3_64<0x96>(rotr64<1>(x), rotr64<8>(x), shr64<7>(x));
}
__device__ __forceinline__ uint64_t small_sigma1_512(uint64_t x) {
    return bitop3_64<0x96>(rotr64<19>(x), rotr64<61>(x), shr64<6>(x));
}

__device__ __forceinline__ void init_state384(uint64_t H[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) H[i] = kInit384[i];
}

// One round on the rotating state (the caller renames a..h between rounds).
__device__ __forceinline__ void round512(uint64_t a, uint64_t b, uint64_t c, uint64_t& d, uint64_t e, uint64_t f,
                                         uint64_t g, uint64_t& h, uint64_t k, uint64_t w) {
    const uint64_t t1 = h + k + w + big_sigma1_512(e) + bitop3_64<0xCA>(e, f, g);
    const uint64_t t2 = big_sigma0_512(a) + bitop3_64<0xE8>(a, b, c);
    d += t1;       // the new e
    h = t1 + t2;   // the new a
}

// Sixteen rounds starting at round r0 (a multiple of 16), so that after them
// the eight state variables are back in their named places.  With SCHED the
// message schedule word of each round is computed in the 16-word ring first.
template <bool SCHED>
__device__ __forceinline__ void sixteen_rounds(uint64_t s[8], uint64_t W[16], const uint64_t* k) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        if (SCHED)
            W[i] = small_sigma1_512(W[(i + 14) & 15]) + W[(i + 9) & 15] + small_sigma0_512(W[(i + 1) & 15]) + W[i];
        // round i works on s rotated by i: a = s[(8 - i) & 7], ..., h = s[(15 - i) & 7]
        round512(s[(8 - i) & 7], s[(9 - i) & 7], s[(10 - i) & 7], s[(11 - i) & 7], s[(12 - i) & 7],
                 s[(13 - i) & 7], s[(14 - i) & 7], s[(15 - i) & 7], k[i], W[i]);
    }
}

// One 1024-bit block: H <- H + rounds(H, W); W holds the 16 big-endian
// message words and is used as the schedule ring (overwritten).  Rounds 0-15
// use W directly; rounds 16-79 run as four trips of sixteen, the round
// constants for a trip coming from kRound512 through scalar loads.
__device__ __forceinline__ void compress512(uint64_t H[8], uint64_t W[16]) {
    uint64_t s[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = H[i];
    sixteen_rounds<false>(s, W, kRound512);
#pragma nounroll
    for (int r = 16; r < 80; r += 16) sixteen_rounds<true>(s, W, kRound512 + r);
#pragma unroll
    for (int i = 0; i < 8; ++i) H[i] += s[i];
}

// Big-endian 64-bit message word from two little-endian dwords as loaded.
__device__ __forceinline__ uint64_t be64(uint32_t first, uint32_t second) {
    return pack(__builtin_bswap32(first), __builtin_bswap32(second));
}

// The 48 digest bytes (H0..H5 big-endian) as three 16-byte stores (16-byte aligned).
__device__ __forceinline__ void store_digest384(uint8_t* dst, const uint64_t H[8]) {
    uint4* p = reinterpret_cast<uint4*>(dst);
#pragma unroll
    for (int i = 0; i < 3; ++i)
        p[i] = make_uint4(__builtin_bswap32(hi32(H[2 * i])), __builtin_bswap32(lo32(H[2 * i])),
                          __builtin_bswap32(hi32(H[2 * i + 1])), __builtin_bswap32(lo32(H[2 * i + 1])));
}

// A 48-byte digest as 12 big-endian 32-bit words (16-byte aligned source).
__device__ __forceinline__ void load_digest384(const uint8_t* src, uint32_t D[12]) {
    const uint4* p = reinterpret_cast<const uint4*>(src);
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const uint4 x = p[i];
        D[4 * i] = __builtin_bswap32(x.x);
        D[4 * i + 1] = __builtin_bswap32(x.y);
        D[4 * i + 2] = __builtin_bswap32(x.z);
        D[4 * i + 3] = __builtin_bswap32(x.w);
    }
}

}  // namespace hv
