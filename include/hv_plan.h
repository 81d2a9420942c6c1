/*
 * hv_plan.h -- the whole verification path prepared once and run many times.
 *
 * Algorithm 1 verifies one model; a server re-verifies the same resident
 * weights again and again (at load, after updates, at an interval).  A plan
 * binds one message set -- its addresses, lengths, chunk size and hash -- and
 * does the host-side work once: the message table and the Merkle launch
 * tables are uploaded and the scheduler builds the leaf table (longest chunks
 * first) in plan memory.  A run then only queues kernels: chunk digests, the
 * per-message (or single) RFC 6962 tree, the manifest root over the message
 * roots (Introduction, hierarchical integrity verification) and, if asked,
 * the comparison with an expected root held in device memory.  A run makes
 * no upload, no host wait, no memset and no allocation, so it can be
 * captured once in a HIP graph and replayed.
 */
#ifndef HV_PLAN_H
#define HV_PLAN_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { HV_PLAN_MAX_LAUNCHES = 8 };

/* Host handle of a plan (caller-owned POD).  `device` points into caller-owned
 * device memory that must outlive every run; the messages must stay at their
 * addresses (their bytes may change: that is what a run checks). */
typedef struct {
    void* device;          /* plan memory: message table, leaf table, Merkle tables, scratch */
    size_t bytes;          /* size of the plan memory in use */
    hv_alg alg;
    int manifest;          /* 1: a root per message, then the manifest root over them; 0: one root over all leaves */
    uint32_t n_msgs;
    uint32_t n_seg;        /* segments of the first tree: n_msgs (manifest) or 1 */
    uint64_t chunk_bytes;
    uint64_t n_leaves;
    uint32_t launches[2];  /* Merkle launches of the first tree and of the manifest */
    uint64_t tiles[2][HV_PLAN_MAX_LAUNCHES];  /* output nodes of each launch */
} hv_verify_plan;

/* Device bytes of a plan for these messages; 0 (with hv_last_error set) for
 * arguments hv_plan_init would reject. */
size_t hv_plan_bytes(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest);

/* Build a plan.  Uploads the host tables before returning (so it returns once the
 * stream has reached them) and queues the scheduling kernels on `stream`.
 *   msgs: host, n_msgs entries (device addresses), as hv_hash_chunks_alg.
 *   plan_memory: device, >= hv_plan_bytes(...), 256-byte aligned.
 *   plan: host, filled on HV_OK.
 * Errors: HV_ERR_INVALID_ARG as hv_hash_chunks_alg, or a NULL plan;
 * HV_ERR_WORKSPACE for missing or short plan memory; HV_ERR_HIP. */
hv_status hv_plan_init(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest,
                       void* plan_memory, size_t plan_bytes, hv_verify_plan* plan, hipStream_t stream);

/* One pass of the path, asynchronous on `stream` (kernels only).
 *   leaf_digests: device, [n_leaves][D] (D = 32 or 48), 16-byte aligned.
 *   roots: device, [n_seg][D], 16-byte aligned (n_seg >= 1 or NULL).
 *   root: device, [1][D], 16-byte aligned: the manifest root (manifest
 *         plans; ignored otherwise, where roots[0] is the root).
 *   expected, match: both NULL (no comparison), or expected = device D
 *         bytes and match = device uint32 that receives 1 when the root
 *         equals expected, else 0.
 * With hv_set_kernel_timing on, events are recorded around the leaf kernel
 * (leave timing off while capturing a graph).
 * Errors: HV_ERR_INVALID_ARG for a NULL or uninitialised plan, NULL or
 * misaligned outputs, or only one of expected / match; HV_ERR_HIP. */
hv_status hv_plan_run(const hv_verify_plan* plan, uint8_t* leaf_digests, uint8_t* roots, uint8_t* root,
                      const uint8_t* expected, uint32_t* match, hipStream_t stream);

/* Result of hv_verify_model: the paper's verification result (Implementation,
 * Rust FFI Bridge: a verified flag, the digest and the time taken), with the
 * root of this path in place of a whole-file digest. */
typedef struct {
    int integrity_verified;         /* 1 when the root equals `expected`, else 0 (0 when no expected root) */
    uint32_t root_bytes;            /* 32 (SHA-256) or 48 (SHA-384) */
    uint8_t root[48];               /* the root, its first root_bytes bytes */
    uint64_t verification_time_ns;  /* host wall time of the call */
} hv_result;

/* Device workspace bytes hv_verify_model needs; 0 (hv_last_error set) for
 * arguments it would reject. */
size_t hv_verify_model_workspace_bytes(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                       int manifest);

/* One call for one verification (synchronous): plan, chunk digests, per-message
 * roots and the manifest root (manifest = 1; Introduction, hierarchical
 * integrity verification) or one root over all chunks (manifest = 0), the
 * comparison with `expected` on the GPU, and the root copied to the host.
 *   msgs: host array of device messages, as hv_hash_chunks_alg.
 *   expected: host, 32 or 48 bytes (the hash's digest size), or NULL to only
 *             compute the root.
 *   workspace: device, >= hv_verify_model_workspace_bytes(...), 256-byte
 *             aligned (holds the plan, digests and roots; nothing is kept).
 *   result: host, filled on HV_OK.
 * A mismatch is not an error: HV_OK with integrity_verified = 0.
 * Errors: as hv_plan_init; HV_ERR_INVALID_ARG for a NULL result; HV_ERR_HIP. */
hv_status hv_verify_model(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest,
                          const uint8_t* expected, void* workspace, size_t workspace_bytes, hv_result* result,
                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HV_PLAN_H */
