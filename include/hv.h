/*
 * hv.h -- C ABI of the device-resident model-integrity path: chunked SHA-256
 * of weight bytes already in GPU memory, Merkle reduction of the chunk
 * digests to per-tensor roots and a manifest root, and comparison of a root
 * with its expected value.  One AMD Instinct MI355X (gfx950), HIP streams.
 *
 * The operations follow arXiv 2510.23938:
 *   - Algorithm 1 ("Streaming Model Verification for Large Models",
 *     Discussion): a model is cut into ceil(|M| / C) chunks, each chunk is
 *     hashed on the GPU, the chunk hashes are the leaves of a Merkle tree
 *     built on the GPU, and the root is compared with the expected value;
 *   - the Merkle tree is the one of RFC 6962 section 2.1 (cited for the
 *     paper's Merkle construction, Introduction), the chunk hash is SHA-256
 *     (FIPS 180-4, the standard hash the paper names);
 *   - roots are hierarchical (Introduction, "Hierarchical Integrity
 *     Verification"): per tensor or shard file, then over those roots;
 *   - the hash runs where the weights live, on the exact device bytes the
 *     model executes from, so nothing crosses PCIe (Problem Statement,
 *     TOCTOU discussion);
 *   - a status plus caller-provided outputs, as the paper's own C ABI does
 *     (Implementation, the extern "C" verification entry point).
 *
 * Conventions for every call:
 *   - Device pointers are caller-owned (typically torch tensor storage).  The
 *     library never allocates device memory: scratch comes from a
 *     caller-provided workspace of the size the *_workspace_bytes call gives
 *     (hv_hash_chunks_noalloc alone uses a static array of the library's).
 *   - Calls are asynchronous on `stream` unless marked "synchronous".  Input
 *     bytes must stay valid and unmodified until the stream work completes.
 *     Host arrays a call takes (message tables, offset, leaf and dirty lists,
 *     expected roots) are an exception: they are read, and uploaded where the
 *     device needs them, before the call returns, whatever memory they are in
 *     (pageable or pinned); such a call returns once `stream` has reached and
 *     finished its uploads.
 *   - All argument checks happen before any kernel is queued; on a non-OK
 *     status no kernel was launched (except HV_ERR_HIP, which reports a failed
 *     launch or copy) and hv_last_error() describes the problem.  (A large
 *     descriptor table may already have been copied into the workspace,
 *     which is scratch: hv_hash_chunks starts that upload while it checks.)
 *   - A root mismatch is not an error: hv_verify_root returns HV_OK, *match=0.
 *   - No global state except a thread-local error string (and the static
 *     scratch of hv_hash_chunks_noalloc).  Concurrent calls on different
 *     streams with different workspaces are safe; calls that share a
 *     workspace must be ordered by the caller.
 */
#ifndef HV_H
#define HV_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HV_OK = 0,
    HV_ERR_INVALID_ARG = 1, /* bad pointer, size, chunk size or offsets     */
    HV_ERR_WORKSPACE = 2,   /* workspace NULL or smaller than required       */
    HV_ERR_HIP = 3          /* a HIP launch or copy failed                   */
} hv_status;

/* One message: `nbytes` bytes at device address `data` (any alignment).
 * `data` may be NULL only when nbytes == 0. */
typedef struct {
    const void* data;
    uint64_t nbytes;
} hv_msg;

enum { HV_DIGEST_BYTES = 32 };

/* Hash of a call.  The plain entry points use SHA-256 (FIPS 180-4 6.2: 32-byte
 * digests, 64-byte blocks).  The *_alg entry points also take SHA-384 (FIPS
 * 180-4 6.5: 48-byte digests, 128-byte blocks) -- the hash of the paper's own
 * kernel listings and the 48-byte digest of its C ABI (Implementation).  With
 * SHA-384 every digest, Merkle node and root is 48 bytes, the tree is RFC 6962
 * with SHA-384 as its hash, and chunk_bytes must be 0 or a multiple of 128. */
typedef int32_t hv_alg; /* an int, not an enum: any value a caller passes is well defined, and rejected if unknown */
enum { HV_SHA256 = 0, HV_SHA384 = 1 };

/* Leaf layout (synchronous, host only, touches no device memory).
 * Chunking (Algorithm 1): a message of L bytes with chunk size C > 0 has
 * ceil(L / C) leaves (none when L == 0); chunk i covers bytes
 * [i*C, min((i+1)*C, L)) -- the last chunk is simply shorter.  C == 0 means
 * one leaf per message, the whole message (also when L == 0).  C must be 0 or
 * a multiple of 64 (so every chunk but the last is whole SHA-256 blocks).
 * Leaves are numbered message-major, chunk-ascending.
 *   seg_offsets: optional (may be NULL), n_msgs + 1 entries: seg_offsets[0] = 0,
 *                seg_offsets[m+1] - seg_offsets[m] = leaves of message m.
 *   n_leaves:    required, total leaves.
 * A single chunk may hold at most 2^37 bytes (128 GiB), and one call at most
 * 2^31 leaves (every call of this library that takes a message set or a
 * segmented node array rejects more).
 * Errors: HV_ERR_INVALID_ARG for msgs == NULL with n_msgs > 0, a NULL data
 * pointer with nbytes > 0, a bad C, a chunk over the size limit, a NULL
 * n_leaves, or a count overflow. */
hv_status hv_leaf_layout(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                         uint64_t* seg_offsets, uint64_t* n_leaves);

/* Workspace bytes hv_hash_chunks needs for n_msgs messages with n_leaves
 * leaves in total (from hv_leaf_layout); 0 (and hv_last_error set) for more
 * than 2^31 leaves. */
size_t hv_hash_workspace_bytes(uint32_t n_msgs, uint64_t n_leaves);

/* Chunk digests (Algorithm 1's per-chunk GPU hash): leaf_digests[j] =
 * SHA-256(chunk j) per FIPS 180-4, 32 bytes each in the standard big-endian
 * byte order, leaves numbered as in hv_leaf_layout.
 *   msgs:         host array of n_msgs device messages (read during the call;
 *                 the descriptors are copied to the workspace).
 *   chunk_bytes:  0 or a multiple of 64.
 *   leaf_digests: device, n_leaves * 32 bytes, 16-byte aligned, caller-owned,
 *                 written.
 *   workspace:    device, >= hv_hash_workspace_bytes(n_msgs, n_leaves) bytes,
 *                 256-byte aligned; contents are scratch.
 * Errors: as hv_leaf_layout, plus leaf_digests == NULL with n_leaves > 0,
 * HV_ERR_WORKSPACE, HV_ERR_HIP. */
hv_status hv_hash_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                         uint8_t* leaf_digests, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* Workspace bytes hv_merkle_reduce needs for n_nodes entries in n_seg
 * segments; 0 (and hv_last_error set) for more than 2^31 entries. */
size_t hv_merkle_workspace_bytes(uint64_t n_nodes, uint32_t n_seg);

/* Segmented Merkle Tree Hash (RFC 6962 section 2.1; Algorithm 1's "construct
 * Merkle tree from leaf_hashes"): for every segment s,
 *   roots[s] = MTH(nodes[seg_offsets[s] .. seg_offsets[s+1]))
 * with MTH({}) = SHA-256(""), MTH({d}) = SHA-256(0x00 || d) and
 * MTH(D[0:n]) = SHA-256(0x01 || MTH(D[0:k]) || MTH(D[k:n])), k the largest
 * power of two below n.  Entries are 32-byte values (chunk digests, or
 * segment roots for a manifest over tensors -- the hierarchical roots).
 *   nodes:       device, seg_offsets[n_seg] * 32 bytes, 16-byte aligned, read only.
 *   seg_offsets: host, n_seg + 1 entries, seg_offsets[0] == 0, non-decreasing.
 *   roots:       device, n_seg * 32 bytes, 16-byte aligned, written.
 *   workspace:   device, >= hv_merkle_workspace_bytes(seg_offsets[n_seg], n_seg).
 * The host plans ceil(depth / 9) launches from seg_offsets and uploads that
 * plan before returning (so the call returns once the stream has reached it).
 * Errors: HV_ERR_INVALID_ARG for n_seg == 0, NULL or misaligned pointers,
 * offsets that do not start at 0 or decrease, more than 2^31 entries;
 * HV_ERR_WORKSPACE; HV_ERR_HIP. */
hv_status hv_merkle_reduce(const uint8_t* nodes, const uint64_t* seg_offsets, uint32_t n_seg,
                           uint8_t* roots, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* Workspace bytes hv_verify_root needs (a few bytes for the device flag). */
size_t hv_verify_workspace_bytes(void);

/* Root comparison (Algorithm 1's last step), synchronous on `stream`:
 * *match = 1 when the 32 device bytes at `root` equal `expected`, else 0.
 * The comparison runs on the GPU over all 32 bytes without an early exit;
 * only the 4-byte flag crosses to the host.
 *   root:     device, 32 bytes.   expected: host, 32 bytes.   match: host.
 *   workspace: device, >= hv_verify_workspace_bytes() bytes, 4-byte aligned.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers; HV_ERR_WORKSPACE for a
 * missing, short or misaligned workspace; HV_ERR_HIP. */
hv_status hv_verify_root(const uint8_t* root, const uint8_t expected[32], int* match,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Per-entry comparison for localising a mismatch (asynchronous):
 * mismatch[i] = 1 when roots[i] (32 bytes) differs from expected[i], else 0.
 *   roots, expected: device, n * 32 bytes.   mismatch: device, n uint32.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers with n > 0; HV_ERR_HIP. */
hv_status hv_compare_roots(const uint8_t* roots, const uint8_t* expected, uint32_t n,
                           uint32_t* mismatch, hipStream_t stream);

/* The same four operations with an explicit hash (hv_alg).  Digest, node and
 * root sizes are 32 bytes for HV_SHA256 and 48 for HV_SHA384 (all arrays
 * [n][32] or [n][48]); `expected` holds that many bytes.  Semantics, layout
 * and errors are those of the SHA-256 calls above, plus HV_ERR_INVALID_ARG
 * for an unknown algorithm or (SHA-384) a chunk size that is not a multiple
 * of 128.  The workspace sizes of hv_hash_workspace_bytes and
 * hv_verify_workspace_bytes serve both hashes; hv_merkle_workspace_bytes_alg
 * returns 0 (and sets hv_last_error) for an unknown algorithm. */
hv_status hv_hash_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                             uint8_t* leaf_digests, void* workspace, size_t workspace_bytes, hipStream_t stream);
size_t hv_merkle_workspace_bytes_alg(hv_alg alg, uint64_t n_nodes, uint32_t n_seg);
hv_status hv_merkle_reduce_alg(hv_alg alg, const uint8_t* nodes, const uint64_t* seg_offsets, uint32_t n_seg,
                               uint8_t* roots, void* workspace, size_t workspace_bytes, hipStream_t stream);
hv_status hv_verify_root_alg(hv_alg alg, const uint8_t* root, const uint8_t* expected, int* match, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);
hv_status hv_compare_roots_alg(hv_alg alg, const uint8_t* roots, const uint8_t* expected, uint32_t n,
                               uint32_t* mismatch, hipStream_t stream);

/* Chunk digests without allocation, for callers that cannot allocate device
 * memory or pass a workspace (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same operation, digests, layout,
 * argument checks and errors as hv_hash_chunks_alg with the same arguments;
 * only the workspace differs: the scheduler's scratch (16 B per message for
 * the descriptors, 32 B per message for counts and offsets, a 32 KiB tail
 * histogram and 24 B per leaf for the leaf table, each region rounded up to
 * 256 B) lives in a static device array of HV_NOALLOC_SCRATCH_BYTES (64 MiB)
 * inside the library, one per GPU, held from the first call on that GPU until
 * the process ends.  That covers, e.g., one message of up to 2,794,794 leaves,
 * or the 723 tensors and 2,153,249 leaves of a 70B-shaped weight set with
 * 64 KiB chunks.  The call makes no hipMalloc, hipFree or other allocation;
 * it runs on the GPU that owns `stream`, and, like hv_hash_chunks, uploads
 * the descriptors before it returns.
 * Every call on one GPU shares that GPU's array, and each call rewrites what
 * it reads there: calls whose work may overlap on one GPU (other streams,
 * other threads) race and must be ordered by the caller.  The leaf-kernel
 * timing of hv_set_kernel_timing is not recorded.
 * Errors: those of hv_hash_chunks_alg, and HV_ERR_INVALID_ARG, before any
 * work is queued, when the message set needs more scratch than the array
 * holds (hv_last_error() gives both sizes). */
enum { HV_NOALLOC_SCRATCH_BYTES = 64 << 20 };
hv_status hv_hash_chunks_noalloc(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                 uint8_t* leaf_digests, hipStream_t stream);

/* Detail string for the last non-OK status returned on this thread. */
const char* hv_last_error(void);

/* Kernel timing for measurement.  When enabled (per thread), hv_hash_chunks
 * records HIP events on `stream` around its leaf kernel (SHA-256, or SHA-384
 * for hv_hash_chunks_alg), and
 * hv_leaf_kernel_ms() waits for the last such pair and returns the elapsed
 * milliseconds.  Off by default; costs two event records per call when on.
 * Errors: HV_ERR_INVALID_ARG if no timed call was made on this thread. */
hv_status hv_set_kernel_timing(int enable);
hv_status hv_leaf_kernel_ms(float* ms);

#ifdef __cplusplus
}
#endif

#endif /* HV_H */
