/*
 * hv_inspect.h -- inspection entry points for tests: the chunk scheduler's
 * leaf table, the leaf-kernel choice and the Merkle launch plan.
 *
 * hv_leaf_schedule runs the same device-side scheduling hv_hash_chunks runs
 * (Algorithm 1's chunking: ceil(|M| / C) chunks per message, the last one
 * shorter) and copies the resulting leaf table to the host, so a test can
 * check that every chunk appears exactly once, with the right source range
 * and output slot, in non-increasing order of SHA-256 block count.  It does
 * not hash.  Synchronous on `stream`.
 *
 *   msgs, n_msgs, chunk_bytes, workspace, workspace_bytes: as hv_hash_chunks.
 *   table: host, n_leaves * 3 uint64 values, written in schedule order as
 *          {source device address, byte length, leaf index} per leaf.
 * Errors: as hv_hash_chunks (HV_ERR_INVALID_ARG for a NULL table with
 * n_leaves > 0).
 */
#ifndef HV_INSPECT_H
#define HV_INSPECT_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

hv_status hv_leaf_schedule(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t* table,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Leaf-kernel choice for tests and measurements, per calling thread:
 * 0 = automatic (calls with at most 128 leaves per compute unit of
 * the current device -- 32768 on MI355X -- use the two-wave kernel, which
 * moves the message schedule to a second wave and shortens each chunk's chain
 * of blocks; others use the one-wave kernel), 1 = always the
 * one-wave kernel, 2 = always the two-wave kernel, 3 = always the two-wave
 * kernel with two producer/consumer pairs per workgroup (the layout it takes
 * above 64 leaves per compute unit).  Monitor scans (hv_monitor.h) take the
 * one-wave kernel under the automatic choice.  The same choice applies to
 * SHA-384's two leaf kernels.  The digests do not depend on it.
 * Errors: HV_ERR_INVALID_ARG for another value. */
hv_status hv_set_leaf_kernel(int choice);

/* The leaf kernel a hash call over n_leaves leaves would run on the current
 * device under this thread's choice: *kernel = 1 (one-wave), 2 (two-wave, one
 * producer/consumer pair per workgroup) or 3 (two-wave, two pairs).  Monitor
 * scans take the one-wave kernel under the automatic choice.
 * Errors: HV_ERR_INVALID_ARG for a NULL kernel. */
hv_status hv_leaf_kernel_for(uint64_t n_leaves, int* kernel);

/* The launches hv_merkle_reduce_alg makes for these segments on a device of
 * `cus` compute units, or on the current device when cus = 0 (RFC 6962
 * section 2.1's tree, built level by level; Algorithm 1's
 * "construct Merkle tree from leaf_hashes using GPU"), for tests and
 * measurements: *launches (at most 8), and per launch k < *launches
 * kind[k] = 1 for a group launch (8 entries of a segment reduced by three
 * levels in registers) or 2 for a tile launch (512 entries, nine levels),
 * units[k] = the groups or tiles it reduces, and one_lane[k] = the groups a
 * group launch gives one lane each; its remaining units[k] - one_lane[k]
 * groups, the launch's last ones, take four lanes each (0 for a tile
 * launch).  kind, units and one_lane: host arrays of at least 8 entries.
 * Host only; no kernel runs, and with cus > 0 no device is needed.
 * Errors: HV_ERR_INVALID_ARG as hv_merkle_reduce_alg's checks of alg and
 * seg_offsets, or for a NULL output; HV_ERR_HIP if cus = 0 and the current
 * device cannot be queried. */
hv_status hv_merkle_launches(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg, uint32_t cus, int* launches,
                             int* kind, uint64_t* units, uint64_t* one_lane);

#ifdef __cplusplus
}
#endif

#endif /* HV_INSPECT_H */
