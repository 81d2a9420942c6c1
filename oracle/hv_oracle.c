/*
 * hv_oracle.c -- plain, slow, obviously-correct CPU reference for the
 * chunk-hash / Merkle / verify path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the tests, the package's smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no source, header, table
 * or helper with the HIP library, and it never reads anything the HIP library
 * produced.
 *
 * What it computes (from the paper, arXiv 2510.23938):
 *   - Algorithm 1 ("Streaming Model Verification for Large Models", Discussion,
 *     Memory Scalability Considerations): a model M is cut into
 *     ceil(|M| / C) chunks, each chunk gets its own hash H_i, the H_i are the
 *     leaves of a Merkle tree, and the root is compared with an expected value.
 *   - The per-chunk hash is SHA-256 (the hash the paper names as the standard
 *     verification hash in its Introduction and threat model, citing
 *     FIPS 180-4).  Implemented here exactly as FIPS 180-4 defines it:
 *     padding (section 5.1.1), parsing (5.2.1), initial value (5.3.3),
 *     constants (4.2.2), functions (4.1.2) and the hash computation (6.2.2).
 *   - The Merkle construction follows RFC 6962 section 2.1, which the paper
 *     cites for its Merkle tree (Introduction, GPU-Native Security
 *     Architecture): MTH({}) = SHA-256(""), MTH({d}) = SHA-256(0x00 || d),
 *     MTH(D[0:n]) = SHA-256(0x01 || MTH(D[0:k]) || MTH(D[k:n])) with k the
 *     largest power of two smaller than n.  It is written recursively, as the
 *     RFC states it -- deliberately not the bottom-up order a GPU uses.
 *   - SHA-384 (FIPS 180-4 section 6.5, the SHA-512 computation of 6.4 with its
 *     own initial value, truncated) -- the hash of the paper's own kernel
 *     listings (Implementation, the vectorized SHA-384 kernel) and the
 *     48-byte digest of its C ABI; the same chunking and RFC 6962 tree apply
 *     with 48-byte entries.
 *   - Hierarchy (Introduction, "Hierarchical Integrity Verification"): one
 *     root per tensor or shard file, then a manifest root over those roots in
 *     caller order.  That composition is done by the Python driver from the
 *     primitives below.
 *
 * Readings of points the paper leaves open (chunk tails are simply shorter,
 * C must be a multiple of 64 or 0 = whole message, an empty message has no
 * chunks) are listed with the design notes; the functions below implement
 * those readings literally.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* FIPS 180-4 section 4.2.2: the 64 SHA-256 round constants.                */
static const uint32_t K256[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u, 0xab1c5ed5u,
    0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u,
    0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u,
    0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u,
    0xa2bfe8a1u, 0xa81a664bu, 0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u,
};

/* FIPS 180-4 section 5.3.3: the initial hash value H(0). */
static const uint32_t H256_INIT[8] = {
    0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
    0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u,
};

/* FIPS 180-4 section 4.1.2 functions, section 3.2 ROTR / SHR. */
static uint32_t ROTR(uint32_t x, unsigned n) { return (x >> n) | (x << (32u - n)); }
static uint32_t SHR(uint32_t x, unsigned n) { return x >> n; }
static uint32_t Ch(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (~x & z); }
static uint32_t Maj(uint32_t x, uint32_t y, uint32_t z) { return (x & y) ^ (x & z) ^ (y & z); }
static uint32_t BSIG0(uint32_t x) { return ROTR(x, 2) ^ ROTR(x, 13) ^ ROTR(x, 22); }
static uint32_t BSIG1(uint32_t x) { return ROTR(x, 6) ^ ROTR(x, 11) ^ ROTR(x, 25); }
static uint32_t SSIG0(uint32_t x) { return ROTR(x, 7) ^ ROTR(x, 18) ^ SHR(x, 3); }
static uint32_t SSIG1(uint32_t x) { return ROTR(x, 17) ^ ROTR(x, 19) ^ SHR(x, 10); }

typedef struct {
    uint32_t H[8];
    uint8_t block[64];
    size_t used;        /* bytes currently held in block[] */
    uint64_t total;     /* message length so far, in bytes */
} sha256_ctx;

/* FIPS 180-4 section 6.2.2, steps 1-4, for one 512-bit block M(i). */
static void sha256_compress(uint32_t H[8], const uint8_t M[64]) {
    uint32_t W[64];
    for (int t = 0; t < 16; ++t)   /* section 5.2.1: big-endian 32-bit words */
        W[t] = ((uint32_t)M[4 * t] << 24) | ((uint32_t)M[4 * t + 1] << 16) |
               ((uint32_t)M[4 * t + 2] << 8) | (uint32_t)M[4 * t + 3];
    for (int t = 16; t < 64; ++t)
        W[t] = SSIG1(W[t - 2]) + W[t - 7] + SSIG0(W[t - 15]) + W[t - 16];

    uint32_t a = H[0], b = H[1], c = H[2], d = H[3];
    uint32_t e = H[4], f = H[5], g = H[6], h = H[7];
    for (int t = 0; t < 64; ++t) {
        uint32_t T1 = h + BSIG1(e) + Ch(e, f, g) + K256[t] + W[t];
        uint32_t T2 = BSIG0(a) + Maj(a, b, c);
        h = g; g = f; f = e; e = d + T1;
        d = c; c = b; b = a; a = T1 + T2;
    }
    H[0] += a; H[1] += b; H[2] += c; H[3] += d;
    H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

static void sha256_init(sha256_ctx* s) {
    memcpy(s->H, H256_INIT, sizeof s->H);
    s->used = 0;
    s->total = 0;
}

static void sha256_update(sha256_ctx* s, const uint8_t* p, uint64_t n) {
    s->total += n;
    while (n > 0) {
        size_t take = 64 - s->used;
        if (take > n) take = (size_t)n;
        memcpy(s->block + s->used, p, take);
        s->used += take;
        p += take;
        n -= take;
        if (s->used == 64) {
            sha256_compress(s->H, s->block);
            s->used = 0;
        }
    }
}

/* Section 5.1.1: append bit '1', then k zero bits with l + 1 + k = 448 mod 512,
 * then the 64-bit big-endian bit length l.  Section 6.2.2: the digest is
 * H0 || ... || H7, each big-endian. */
static void sha256_final(sha256_ctx* s, uint8_t out[32]) {
    uint64_t bits = s->total * 8u;
    uint8_t one = 0x80, zero = 0x00;
    uint64_t saved_total = s->total;
    sha256_update(s, &one, 1);
    while (s->used != 56) sha256_update(s, &zero, 1);
    uint8_t len_be[8];
    for (int i = 0; i < 8; ++i) len_be[i] = (uint8_t)(bits >> (56 - 8 * i));
    sha256_update(s, len_be, 8);
    s->total = saved_total;
    for (int i = 0; i < 8; ++i) {
        out[4 * i] = (uint8_t)(s->H[i] >> 24);
        out[4 * i + 1] = (uint8_t)(s->H[i] >> 16);
        out[4 * i + 2] = (uint8_t)(s->H[i] >> 8);
        out[4 * i + 3] = (uint8_t)s->H[i];
    }
}

/* ------------------------------------------------------------------------ */
/* Exported primitives (loaded through ctypes by the Python driver).        */

void oracle_constants(uint32_t K_out[64], uint32_t H0_out[8]) {
    memcpy(K_out, K256, sizeof K256);
    memcpy(H0_out, H256_INIT, sizeof H256_INIT);
}

/* SHA-256(m[0:n]). */
void oracle_sha256(const uint8_t* m, uint64_t n, uint8_t out[32]) {
    sha256_ctx s;
    sha256_init(&s);
    sha256_update(&s, m, n);
    sha256_final(&s, out);
}

/* SHA-256(p || m[0:n]) for a one-byte prefix p (RFC 6962 domain separation). */
static void sha256_prefixed(uint8_t p, const uint8_t* m, uint64_t n, uint8_t out[32]) {
    sha256_ctx s;
    sha256_init(&s);
    sha256_update(&s, &p, 1);
    sha256_update(&s, m, n);
    sha256_final(&s, out);
}

/* Algorithm 1: chunk_count = ceil(|M| / C); C = 0 means "one chunk = whole
 * message" (even when the message is empty).  Returns UINT64_MAX for a chunk
 * size that is not a multiple of 64. */
uint64_t oracle_chunk_count(uint64_t len, uint64_t C) {
    if (C == 0) return 1;
    if (C % 64 != 0) return UINT64_MAX;
    return len / C + (len % C != 0);
}

/* Chunk i covers bytes [i*C, min((i+1)*C, len)); the last one is simply
 * shorter -- no zero padding to C (SHA-256 pads on its own). */
void oracle_chunk_digests(const uint8_t* m, uint64_t len, uint64_t C, uint8_t* out) {
    uint64_t n = oracle_chunk_count(len, C);
    if (C == 0) { oracle_sha256(m, len, out); return; }
    for (uint64_t i = 0; i < n; ++i) {
        uint64_t lo = i * C;
        uint64_t hi = lo + C < len ? lo + C : len;
        oracle_sha256(m + lo, hi - lo, out + 32 * i);
    }
}

/* RFC 6962 section 2.1, recursively. entries: n 32-byte values. */
void oracle_mth(const uint8_t* entries, uint64_t n, uint8_t out[32]) {
    if (n == 0) { oracle_sha256(NULL, 0, out); return; }
    if (n == 1) { sha256_prefixed(0x00, entries, 32, out); return; }
    uint64_t k = 1;
    while (k * 2 < n) k *= 2;          /* largest power of two < n */
    uint8_t lr[64];
    oracle_mth(entries, k, lr);
    oracle_mth(entries + 32 * k, n - k, lr + 32);
    sha256_prefixed(0x01, lr, 64, out);
}

/* Root of one message: MTH over its chunk digests. */
void oracle_seg_root(const uint8_t* m, uint64_t len, uint64_t C, uint8_t out[32]) {
    uint64_t n = oracle_chunk_count(len, C);
    uint8_t* d = (uint8_t*)malloc(n ? 32 * n : 1);
    oracle_chunk_digests(m, len, C, d);
    oracle_mth(d, n, out);
    free(d);
}


/* ------------------------------------------------------------------------ */
/* SHA-384 (FIPS 180-4 section 6.5): the SHA-512 computation of section 6.4 */
/* with its own initial value (5.3.4), truncated to the first 384 bits.     */

/* Section 4.2.3: first 64 bits of the fractional parts of the cube roots of
 * the first 80 primes. */
static const uint64_t K512[80] = {
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

/* Section 5.3.4: first 64 bits of the fractional parts of the square roots of
 * the ninth through sixteenth primes. */
static const uint64_t H384_INIT[8] = {
    0xcbbb9d5dc1059ed8ull, 0x629a292a367cd507ull, 0x9159015a3070dd17ull, 0x152fecd8f70e5939ull,
    0x67332667ffc00b31ull, 0x8eb44a8768581511ull, 0xdb0c2e0d64f98fa7ull, 0x47b5481dbefa4fa4ull,
};

/* Section 4.1.3 functions on 64-bit words. */
static uint64_t ROTR64(uint64_t x, unsigned n) { return (x >> n) | (x << (64u - n)); }
static uint64_t Ch64(uint64_t x, uint64_t y, uint64_t z) { return (x & y) ^ (~x & z); }
static uint64_t Maj64(uint64_t x, uint64_t y, uint64_t z) { return (x & y) ^ (x & z) ^ (y & z); }
static uint64_t BSIG0_64(uint64_t x) { return ROTR64(x, 28) ^ ROTR64(x, 34) ^ ROTR64(x, 39); }
static uint64_t BSIG1_64(uint64_t x) { return ROTR64(x, 14) ^ ROTR64(x, 18) ^ ROTR64(x, 41); }
static uint64_t SSIG0_64(uint64_t x) { return ROTR64(x, 1) ^ ROTR64(x, 8) ^ (x >> 7); }
static uint64_t SSIG1_64(uint64_t x) { return ROTR64(x, 19) ^ ROTR64(x, 61) ^ (x >> 6); }

typedef struct {
    uint64_t H[8];
    uint8_t block[128];
    size_t used;
    uint64_t total;
} sha512_ctx;

/* Section 6.4.2 steps 1-4 for one 1024-bit block. */
static void sha512_compress(uint64_t H[8], const uint8_t M[128]) {
    uint64_t W[80];
    for (int t = 0; t < 16; ++t) {  /* section 5.2.2: big-endian 64-bit words */
        uint64_t w = 0;
        for (int b = 0; b < 8; ++b) w = (w << 8) | M[8 * t + b];
        W[t] = w;
    }
    for (int t = 16; t < 80; ++t) W[t] = SSIG1_64(W[t - 2]) + W[t - 7] + SSIG0_64(W[t - 15]) + W[t - 16];
    uint64_t a = H[0], b = H[1], c = H[2], d = H[3], e = H[4], f = H[5], g = H[6], h = H[7];
    for (int t = 0; t < 80; ++t) {
        uint64_t T1 = h + BSIG1_64(e) + Ch64(e, f, g) + K512[t] + W[t];
        uint64_t T2 = BSIG0_64(a) + Maj64(a, b, c);
        h = g; g = f; f = e; e = d + T1;
        d = c; c = b; b = a; a = T1 + T2;
    }
    H[0] += a; H[1] += b; H[2] += c; H[3] += d;
    H[4] += e; H[5] += f; H[6] += g; H[7] += h;
}

static void sha384_init(sha512_ctx* s) {
    memcpy(s->H, H384_INIT, sizeof s->H);
    s->used = 0;
    s->total = 0;
}

static void sha512_update(sha512_ctx* s, const uint8_t* p, uint64_t n) {
    s->total += n;
    while (n > 0) {
        size_t take = 128 - s->used;
        if (take > n) take = (size_t)n;
        memcpy(s->block + s->used, p, take);
        s->used += take;
        p += take;
        n -= take;
        if (s->used == 128) {
            sha512_compress(s->H, s->block);
            s->used = 0;
        }
    }
}

/* Section 5.1.2: bit '1', zeros to 896 mod 1024, then the 128-bit big-endian
 * bit length.  Section 6.5: the digest is H0..H5, big-endian. */
static void sha384_final(sha512_ctx* s, uint8_t out[48]) {
    const uint64_t total = s->total;
    uint8_t len_be[16];
    const uint64_t hi = total >> 61, lo = total << 3;
    for (int i = 0; i < 8; ++i) {
        len_be[i] = (uint8_t)(hi >> (56 - 8 * i));
        len_be[8 + i] = (uint8_t)(lo >> (56 - 8 * i));
    }
    uint8_t one = 0x80, zero = 0x00;
    sha512_update(s, &one, 1);
    while (s->used != 112) sha512_update(s, &zero, 1);
    sha512_update(s, len_be, 16);
    s->total = total;
    for (int i = 0; i < 6; ++i)
        for (int b = 0; b < 8; ++b) out[8 * i + b] = (uint8_t)(s->H[i] >> (56 - 8 * b));
}

void oracle_constants512(uint64_t K_out[80], uint64_t H384_out[8]) {
    memcpy(K_out, K512, sizeof K512);
    memcpy(H384_out, H384_INIT, sizeof H384_INIT);
}

void oracle_sha384(const uint8_t* m, uint64_t n, uint8_t out[48]) {
    sha512_ctx s;
    sha384_init(&s);
    sha512_update(&s, m, n);
    sha384_final(&s, out);
}

static void sha384_prefixed(uint8_t p, const uint8_t* m, uint64_t n, uint8_t out[48]) {
    sha512_ctx s;
    sha384_init(&s);
    sha512_update(&s, &p, 1);
    sha512_update(&s, m, n);
    sha384_final(&s, out);
}

/* RFC 6962 section 2.1 with SHA-384 as the hash: 48-byte entries and nodes. */
void oracle_mth384(const uint8_t* entries, uint64_t n, uint8_t out[48]) {
    if (n == 0) { oracle_sha384(NULL, 0, out); return; }
    if (n == 1) { sha384_prefixed(0x00, entries, 48, out); return; }
    uint64_t k = 1;
    while (k * 2 < n) k *= 2;
    uint8_t lr[96];
    oracle_mth384(entries, k, lr);
    oracle_mth384(entries + 48 * k, n - k, lr + 48);
    sha384_prefixed(0x01, lr, 96, out);
}

/* ------------------------------------------------------------------------ */
/* Threaded driver: the same chunk digests, spread over POSIX threads.  Each
 * thread takes whole chunks from a shared counter and hashes them with the
 * single-threaded routine above; nothing is reordered inside a chunk.  Used
 * to keep full-size parity runs and the CPU baseline within wall-clock
 * limits. */

typedef struct {
    int alg;                      /* 0: SHA-256 (32-byte digests), 1: SHA-384 (48-byte digests) */
    const uint8_t* const* msgs;
    const uint64_t* lens;
    const uint64_t* first_leaf;   /* leaf index of each message's chunk 0 */
    uint32_t n_msgs;
    uint64_t C;
    uint8_t* out;
    uint64_t n_leaves;
    uint64_t next;                /* next leaf to take (guarded by lock) */
    uint64_t grab;                /* leaves a thread takes at a time */
    pthread_mutex_t lock;
} mt_job;

static void* mt_worker(void* arg) {
    mt_job* j = (mt_job*)arg;
    uint32_t m = 0;
    for (;;) {
        pthread_mutex_lock(&j->lock);
        uint64_t leaf = j->next;
        uint64_t take = j->grab;
        if (leaf + take > j->n_leaves) take = j->n_leaves - leaf;
        j->next = leaf + take;
        pthread_mutex_unlock(&j->lock);
        if (take == 0) break;
        for (uint64_t L = leaf; L < leaf + take; ++L) {
            /* find the message holding leaf L (leaves are message-major) */
            while (m + 1 < j->n_msgs && j->first_leaf[m + 1] <= L) ++m;
            uint64_t i = L - j->first_leaf[m];
            const uint8_t* p = j->msgs[m];
            uint64_t len = j->lens[m];
            uint64_t lo = 0, hi = len;
            if (j->C != 0) {
                lo = i * j->C;
                hi = lo + j->C < len ? lo + j->C : len;
            }
            if (j->alg == 1) oracle_sha384(p + lo, hi - lo, j->out + 48 * L);
            else oracle_sha256(p + lo, hi - lo, j->out + 32 * L);
        }
    }
    return NULL;
}

/* Leaf digests of n_msgs messages, message-major and chunk-ascending, written
 * to out (n_leaves * 32 bytes for SHA-256, * 48 for SHA-384; C must then be a
 * multiple of the algorithm's 64- or 128-byte block).  Returns the number of leaves, or UINT64_MAX
 * on a bad chunk size.  Each thread only ever moves forward through the leaf
 * list, so its message cursor m only moves forward too. */
uint64_t oracle_leaf_digests_alg_mt(int alg, const uint8_t* const* msgs, const uint64_t* lens, uint32_t n_msgs,
                                    uint64_t C, uint8_t* out, int nthreads) {
    if (C != 0 && C % (alg == 1 ? 128 : 64) != 0) return UINT64_MAX;
    uint64_t* first = (uint64_t*)malloc(sizeof(uint64_t) * (n_msgs ? n_msgs : 1));
    uint64_t total = 0;
    for (uint32_t m = 0; m < n_msgs; ++m) {
        first[m] = total;
        total += oracle_chunk_count(lens[m], C);
    }
    mt_job j;
    j.alg = alg;
    j.msgs = msgs; j.lens = lens; j.first_leaf = first; j.n_msgs = n_msgs; j.C = C;
    j.out = out; j.n_leaves = total; j.next = 0;
    if (nthreads < 1) nthreads = 1;
    /* about eight grabs per thread, 1..64 leaves each, so that few large
     * chunks still spread over every thread */
    j.grab = total / ((uint64_t)nthreads * 8);
    if (j.grab < 1) j.grab = 1;
    if (j.grab > 64) j.grab = 64;
    pthread_mutex_init(&j.lock, NULL);
    pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
    /* Workers drain the shared counter, so the result is complete even if
     * fewer threads than asked for could be started. */
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
        if (pthread_create(&th[t], NULL, mt_worker, &j) != 0) break;
        ++started;
    }
    if (started == 0) mt_worker(&j);
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    pthread_mutex_destroy(&j.lock);
    free(th);
    free(first);
    return total;
}

/* SHA-256 leaf digests (32 bytes each): the threaded driver with alg 0. */
uint64_t oracle_leaf_digests_mt(const uint8_t* const* msgs, const uint64_t* lens, uint32_t n_msgs, uint64_t C,
                                uint8_t* out, int nthreads) {
    return oracle_leaf_digests_alg_mt(0, msgs, lens, n_msgs, C, out, nthreads);
}
