/*
 * hv_microbench.h -- microbenchmarks for the two roofline denominators of the
 * hashing path on the GPU it runs on: the integer-VALU issue rate and the HBM
 * read bandwidth.  The hashing path itself is bound by 32-bit VALU work
 * (about 1400 ops per 64-byte SHA-256 block); these kernels measure what the
 * chip sustains for that instruction mix and for a plain streaming read, so
 * the hash kernel's fraction of peak can be stated against measured, not only
 * published, peaks.  Asynchronous on `stream`; time them with events on the
 * same stream.
 */
#ifndef HV_MICROBENCH_H
#define HV_MICROBENCH_H

#include "hv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Independent chains of v_alignbit_b32, v_bitop3_b32 and v_add3_u32 (the
 * SHA-256 round mix), `iters` loop trips per lane, `grid` blocks of 256 lanes.
 *   sink: device, grid * 256 uint32 (written; keeps the work alive).
 *   ops_per_launch: host, receives the number of 32-bit lane-ops one launch
 *                   issues in its loop (grid * 256 * iters * ops per trip).
 * Errors: HV_ERR_INVALID_ARG for NULL pointers or grid == 0; HV_ERR_HIP. */
hv_status hv_mb_valu(uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch, hipStream_t stream);

/* SHA-256 compressions chained on registers only (FIPS 180-4 section 6.2.2
 * rounds, no loads or stores in the loop): `blocks` per lane, `grid` blocks
 * of 256 lanes.  The rate of this kernel is the ceiling of the leaf kernel's
 * arithmetic on this chip at the clock it holds.
 *   sink: device, grid * 256 uint32 (written).
 *   blocks_per_launch: host, receives grid * 256 * blocks.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers or grid == 0; HV_ERR_HIP. */
hv_status hv_mb_sha256(uint32_t* sink, uint32_t grid, uint32_t blocks, uint64_t* blocks_per_launch,
                       hipStream_t stream);

/* Streaming read of `nbytes` (a multiple of 16) at `buf` with 16-byte loads,
 * grid-stride, folded to one word per lane.
 *   buf: device, 16-byte aligned.   sink: device, grid * 256 uint32.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers, misalignment, grid == 0;
 * HV_ERR_HIP. */
hv_status hv_mb_hbm_read(const void* buf, uint64_t nbytes, uint32_t* sink, uint32_t grid, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HV_MICROBENCH_H */
