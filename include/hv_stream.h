/*
 * hv_stream.h -- chunk digests of host-resident messages, streamed through GPU
 * memory: the load / hash / free loop of Algorithm 1 ("Streaming Model
 * Verification for Large Models", Discussion), for models larger than HBM or
 * not yet on the GPU.  The digests are exactly those hv_hash_chunks gives for
 * the same bytes resident on the device; the Merkle and verify calls of hv.h
 * then apply unchanged.
 */
#ifndef HV_STREAM_H
#define HV_STREAM_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes hv_hash_host_chunks needs: two staging buffers of
 * batch_bytes plus the descriptors and scheduler scratch of the batch plan.
 * Returns 0 when the arguments are invalid (hv_last_error() says why). */
size_t hv_stream_workspace_bytes(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t batch_bytes);

/* leaf_digests[j] = SHA-256(chunk j) for messages in host memory, numbered as
 * in hv_leaf_layout.  Synchronous: returns after every digest is written.
 *   msgs:        host array; msgs[m].data are HOST addresses (pinned memory,
 *                e.g. hipHostMalloc or torch pin_memory, lets copies overlap
 *                hashing; pageable memory works but copies synchronously).
 *   chunk_bytes: 0 or a multiple of 64.
 *   batch_bytes: staging size per batch, a multiple of 256, at least the
 *                longest chunk (with chunk_bytes 0: the longest message).
 *   leaf_digests: device, n_leaves * 32 bytes, 16-byte aligned, written.
 *   workspace:   device, >= hv_stream_workspace_bytes(...), 256-byte aligned.
 *   copy_stream, hash_stream: host-to-device copies run on the first, hashing
 *                on the second (they may be the same stream: no overlap).
 * Errors: as hv_hash_chunks, plus HV_ERR_INVALID_ARG for a batch_bytes that is
 * not a multiple of 256 or is smaller than a chunk. */
hv_status hv_hash_host_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint8_t* leaf_digests,
                              uint64_t batch_bytes, void* workspace, size_t workspace_bytes, hipStream_t copy_stream,
                              hipStream_t hash_stream);

/* The same with an explicit hash (hv_alg, as hv_hash_chunks_alg): with
 * HV_SHA384 the digests are 48 bytes (leaf_digests n_leaves * 48 bytes) and
 * chunk_bytes must be 0 or a multiple of 128.  The workspace size of
 * hv_stream_workspace_bytes serves both hashes. */
hv_status hv_hash_host_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                  uint8_t* leaf_digests, uint64_t batch_bytes, void* workspace, size_t workspace_bytes,
                                  hipStream_t copy_stream, hipStream_t hash_stream);

#ifdef __cplusplus
}
#endif

#endif /* HV_STREAM_H */
