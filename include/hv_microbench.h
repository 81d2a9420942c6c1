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

/* The SHA-384 mix (FIPS 180-4 section 6.4 on 32-bit lanes): independent
 * chains of a 64-bit rotate (two v_alignbit_b32), a 3-input XOR of 64-bit
 * words (two v_bitop3_b32) and a 64-bit add (one v_lshl_add_u64), `iters`
 * trips per lane.  Its rate against hv_mb_valu's shows whether the 64-bit
 * add issues at the 32-bit rate.  Arguments and errors as hv_mb_valu;
 * ops_per_launch counts five instructions per chain and trip. */
hv_status hv_mb_valu64(uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch, hipStream_t stream);

/* SHA-384 compressions chained on registers only (section 6.4 rounds on
 * 1024-bit blocks, SHA-384's initial value), as hv_mb_sha256: the ceiling of
 * the SHA-384 leaf kernel's arithmetic.  Arguments and errors as hv_mb_sha256. */
hv_status hv_mb_sha384(uint32_t* sink, uint32_t grid, uint32_t blocks, uint64_t* blocks_per_launch,
                       hipStream_t stream);

/* Issue rate of one VALU instruction: eight independent chains per lane of
 *   op 0 v_alignbit_b32, 1 v_bitop3_b32, 2 v_add3_u32, 3 v_add_u32,
 *   4 v_xor_b32, 5 v_lshrrev_b32, 6 v_perm_b32, 7 v_lshl_add_u64,
 * 32 instructions per loop trip (four of each of the eight chains), `iters`
 * trips, `grid` blocks of 256 lanes.  Some of these issue
 * two per quad-cycle when two waves of a SIMD offer them together; comparing
 * the rates shows which.
 *   ops_per_launch: host, receives grid * 256 * iters * 32.
 * Errors: HV_ERR_INVALID_ARG for NULL pointers, grid == 0 or op > 7; HV_ERR_HIP. */
hv_status hv_mb_op_rate(uint32_t op, uint32_t* sink, uint32_t grid, uint32_t iters, uint64_t* ops_per_launch,
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
