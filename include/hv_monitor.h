/*
 * hv_monitor.h -- continuous runtime monitoring of resident weights.
 *
 * The paper asks whether co-locating verification with the GPU makes
 * continuous integrity monitoring during pipeline execution practical,
 * without a large cost to that execution (GPU-Native Model Integrity
 * Overview, Research Questions and Objectives: continuous verification), and
 * its command-line integration re-verifies a running model at a fixed
 * interval (Implementation, Atlas CLI Integration: the runtime-monitoring
 * command).  Here a monitor
 * re-verifies the weights slice by slice while other work runs on the GPU:
 * each scan rehashes a contiguous range of leaves (the chunks of Algorithm 1,
 * numbered as by hv_leaf_layout) and compares every fresh digest with the
 * reference digest recorded when the weights were first verified against
 * their expected root.  If every leaf digest equals its reference, the root
 * over them equals the verified root, so a full sweep of scans is a full
 * re-verification; a mismatch names the changed chunk.
 *
 * The slice length is the monitor's budget: a scan of k leaves occupies
 * about k / 64 waves for the time one chunk takes to hash, so short slices
 * leave most of the chip to the co-running work.  Scans are asynchronous,
 * allocate nothing and wait for nothing on the host, so they can be issued
 * on their own stream (default priority) between or beside inference work.
 */
#ifndef HV_MONITOR_H
#define HV_MONITOR_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The device-resident description of a message set, made once by
 * hv_monitor_init and read by every scan.  Host struct, caller-owned;
 * `device` points into caller-owned device memory that must stay allocated,
 * and the messages must stay at the same addresses (their bytes may change:
 * that is what a scan detects). */
typedef struct {
    void* device;          /* plan memory (device): message table and leaf offsets */
    hv_alg alg;            /* hash of the leaves */
    uint32_t n_msgs;
    uint64_t chunk_bytes;  /* C, as for hv_hash_chunks_alg */
    uint64_t n_leaves;     /* leaves of the whole set */
} hv_monitor_plan;

/* Device bytes hv_monitor_init needs for n_msgs messages. */
size_t hv_monitor_plan_bytes(uint32_t n_msgs);

/* Build a plan: uploads the message table before returning (so this returns
 * once the stream has reached the upload) and queues the per-message leaf
 * offsets on `stream`.
 *   msgs: host, n_msgs entries (device addresses, as hv_hash_chunks_alg).
 *   plan_memory: device, >= hv_monitor_plan_bytes(n_msgs), 256-byte aligned.
 *   plan: host, filled on HV_OK.
 * Errors: HV_ERR_INVALID_ARG as hv_hash_chunks_alg (bad algorithm, chunk
 * size, NULL message data) or NULL plan; HV_ERR_WORKSPACE for missing or
 * short plan memory; HV_ERR_HIP. */
hv_status hv_monitor_init(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, void* plan_memory,
                          size_t plan_bytes, hv_monitor_plan* plan, hipStream_t stream);

/* Scratch bytes of a scan of up to max_slice leaves; 0 (and hv_last_error
 * set) for an unknown algorithm or more than 2^31 leaves. */
size_t hv_monitor_scan_workspace_bytes(hv_alg alg, uint64_t max_slice);

/* One scan (asynchronous on `stream`; no host synchronisation, no upload,
 * no allocation): rehash leaves [first_leaf, first_leaf + n_slice) of the
 * plan's message set and compare each digest with ref_digests[leaf].
 *   ref_digests: device, [plan->n_leaves][D] (D = 32 or 48), 16-byte aligned:
 *                the reference digests of the whole set, message-major.
 *   slice_digests: device, [n_slice][D], 16-byte aligned, or NULL; when
 *                given, the fresh digests are also left there.
 *   result: device, 2 uint64, 8-byte aligned, overwritten by the scan:
 *                result[0] = number of leaves in the slice whose digest
 *                differs from its reference; result[1] = the lowest such
 *                leaf number, or UINT64_MAX when none does.
 *   workspace: device, >= hv_monitor_scan_workspace_bytes(plan->alg,
 *                n_slice), 256-byte aligned; reused by the next scan on the
 *                same stream, so scans sharing a workspace must share a
 *                stream.
 * Errors: HV_ERR_INVALID_ARG for a NULL plan or result, a range past
 * plan->n_leaves, NULL or misaligned digests; HV_ERR_WORKSPACE; HV_ERR_HIP. */
hv_status hv_monitor_scan(const hv_monitor_plan* plan, uint64_t first_leaf, uint64_t n_slice,
                          const uint8_t* ref_digests, uint8_t* slice_digests, uint64_t* result, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/* Spatial partitioning for a monitor: a stream whose kernels run only on the
 * listed compute units (HIP's CU-masked streams), at the default priority.
 * Giving the monitor a few CUs and the co-running work a stream masked to
 * the others bounds the monitor's cost to the CUs it takes; sharing CUs
 * instead slows a co-running kernel by more than the monitor's share, since
 * that kernel waits for its tiles on the shared CUs.
 *   mask: host, n_words 32-bit words; bit i of word w selects CU 32*w + i
 *         in the runtime's numbering (bits at or past the device's CU count
 *         are ignored).
 *   stream: host, receives the new stream; release it with hv_stream_destroy.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers, n_words == 0, or a mask that
 * selects none of the device's CUs (work on such a stream could never run);
 * HV_ERR_HIP. */
hv_status hv_stream_create_cu_masked(const uint32_t* mask, uint32_t n_words, hipStream_t* stream);

/* The CU mask of a stream (n_words words written to mask, host).
 * Errors: HV_ERR_INVALID_ARG for NULL pointers or n_words == 0; HV_ERR_HIP. */
hv_status hv_stream_cu_mask(hipStream_t stream, uint32_t* mask, uint32_t n_words);

/* Wait for a stream made by hv_stream_create_cu_masked, then destroy it.
 * No event recorded on the stream may be queried, waited on or destroyed
 * afterwards (the runtime's events refer to their stream), so a stream that
 * other libraries have recorded events on should live until the process ends.
 * Errors: HV_ERR_INVALID_ARG for a NULL stream; HV_ERR_HIP. */
hv_status hv_stream_destroy(hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HV_MONITOR_H */
