/*
 * hv_incremental.h -- incremental re-verification after a model update.
 *
 * The paper's lifecycle argument (Introduction and Problem Statement: model
 * lifecycle complexity; Discussion: version management, differential
 * verification and incremental hash updates) is that fine-tuning changes a
 * subset of the weights, so re-measurement should rehash only the changed
 * chunks and recompute only the Merkle branches above them.  These calls do
 * that on the device:
 *   hv_rehash_chunks  -- recompute leaf_digests[j] for a listed set of leaves;
 *   hv_tree_build     -- keep every level of every segment's RFC 6962 tree;
 *   hv_tree_update    -- recompute only the nodes above listed leaves:
 *                        O(k log n) node hashes for k changed leaves.
 * Results equal a full recompute (hv_hash_chunks + hv_merkle_reduce) of the
 * updated bytes.  Conventions are those of hv.h.
 */
#ifndef HV_INCREMENTAL_H
#define HV_INCREMENTAL_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Device bytes of the persistent tree for these segments (as hv_merkle_reduce
 * takes them): every level's nodes plus the level offset table.  Returns 0
 * for invalid offsets. */
size_t hv_tree_bytes(const uint64_t* seg_offsets, uint32_t n_seg);

/* Builds the tree from leaf digests (device [seg_offsets[n_seg]][32]) into
 * `tree` (device, >= hv_tree_bytes, 256-byte aligned, caller-owned, kept
 * between calls) and writes roots[s] = MTH of segment s (as hv_merkle_reduce).
 * Errors: as hv_merkle_reduce. */
hv_status hv_tree_build(const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg, void* tree,
                        size_t tree_bytes, uint8_t* roots, hipStream_t stream);

/* Workspace bytes hv_tree_update needs for n_dirty listed leaves. */
size_t hv_tree_update_workspace_bytes(uint32_t n_dirty);

/* After leaf_digests[dirty[i]] changed (i < n_dirty): recomputes the leaf
 * nodes of the listed leaves and every ancestor of them, in place in `tree`
 * (built by hv_tree_build with the same seg_offsets), and rewrites roots[].
 *   dirty: host, strictly increasing leaf numbers below seg_offsets[n_seg].
 * Errors: as hv_tree_build, plus HV_ERR_INVALID_ARG for an unsorted or
 * out-of-range list; HV_ERR_WORKSPACE. */
hv_status hv_tree_update(const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg, void* tree,
                         size_t tree_bytes, const uint64_t* dirty, uint32_t n_dirty, uint8_t* roots, void* workspace,
                         size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes hv_rehash_chunks needs for n_msgs messages and n_listed leaves. */
size_t hv_rehash_workspace_bytes(uint32_t n_msgs, uint32_t n_listed);

/* leaf_digests[leaves[i]] = SHA-256(chunk leaves[i]) for i < n_listed, with
 * chunks and leaf numbers as in hv_hash_chunks; other digests are untouched.
 *   leaves: host, strictly increasing leaf numbers below the message set's
 *           leaf count.
 * Errors: as hv_hash_chunks, plus HV_ERR_INVALID_ARG for an unsorted or
 * out-of-range list. */
hv_status hv_rehash_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, const uint64_t* leaves,
                           uint32_t n_listed, uint8_t* leaf_digests, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* The four calls above with an explicit hash (hv_alg, as the *_alg calls of
 * hv.h): with HV_SHA384 every digest and node is 48 bytes (the tree holds
 * 48-byte nodes, so hv_tree_bytes_alg sizes it for the hash) and the chunk
 * size of a rehash must be 0 or a multiple of 128.  The plain calls are the
 * HV_SHA256 case.  A tree must be updated with the hash it was built with.
 * hv_tree_bytes_alg returns 0 for an unknown algorithm; the others fail with
 * HV_ERR_INVALID_ARG. */
size_t hv_tree_bytes_alg(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg);
hv_status hv_tree_build_alg(hv_alg alg, const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg,
                            void* tree, size_t tree_bytes, uint8_t* roots, hipStream_t stream);
hv_status hv_tree_update_alg(hv_alg alg, const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg,
                             void* tree, size_t tree_bytes, const uint64_t* dirty, uint32_t n_dirty, uint8_t* roots,
                             void* workspace, size_t workspace_bytes, hipStream_t stream);
hv_status hv_rehash_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                               const uint64_t* leaves, uint32_t n_listed, uint8_t* leaf_digests, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HV_INCREMENTAL_H */
