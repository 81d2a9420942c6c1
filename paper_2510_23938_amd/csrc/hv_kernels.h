// hv_kernels.h -- launchers shared between the kernel sources and the C ABI.
// Every launcher queues work on `stream` and returns the launch status; it
// trusts its arguments (the C ABI validates them first).
#pragma once
#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime.h>

namespace hv {

// Hash algorithm of a call: SHA-256 (32-byte digests, 64-byte blocks) or
// SHA-384 (48-byte digests, 128-byte blocks).
constexpr int kAlgSha256 = 0;
constexpr int kAlgSha384 = 1;

// One leaf as the hash kernel sees it.
struct LeafDesc {
    uint64_t src;     // device address of the chunk's first byte
    uint64_t nbytes;  // chunk length in bytes
    uint64_t out;     // leaf index: the digest goes to leaf_digests + 32 * out
};

// Message descriptor as uploaded (same layout as hv_msg).
struct MsgDesc {
    uint64_t data;
    uint64_t nbytes;
};

// Per-message counts / offsets: x = full chunks, y = tail leaves (0 or 1).
using Pair = ulonglong2;

constexpr int kSortBuckets = 4096;   // block-count classes of the tail sort

// Leaf launchers split a call into launches of at most this many leaf-table
// slots, so a grid stays below a dispatch's 2^32 work-items at two lanes per
// slot (the two-wave kernels).
constexpr uint64_t kMaxSlotsPerLaunch = (uint64_t)1 << 30;

// Scheduler (sched.hip).
hipError_t launch_fill_u64(uint64_t* p, size_t n, uint64_t v, hipStream_t s);
hipError_t launch_sched_count(const MsgDesc* msgs, uint32_t n, uint64_t C, Pair* cnt, hipStream_t s);
size_t scan_partials_count(size_t n);
hipError_t launch_scan_pairs(const Pair* in, Pair* out, size_t n, Pair* partials, hipStream_t s);
hipError_t launch_sched_full(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                             LeafDesc* desc, hipStream_t s);
hipError_t launch_sched_tails(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                              uint64_t* hist, LeafDesc* desc, hipStream_t s);

// SHA-384 of the n_slots leaves of a leaf table (sha384_leaves.hip): 48-byte
// digests at digests + 48 * desc.out for desc.out < out_bound.
hipError_t launch_sha384_leaves(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                                hipStream_t s);

// Leaf table for a sorted list of leaf numbers (sched.hip): desc[e] is leaf
// leaves[e], located through the per-message offsets `off` (first leaf of
// message m = off[m].x + off[m].y).
hipError_t launch_sched_select(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, const uint64_t* leaves,
                               uint64_t k, LeafDesc* desc, hipStream_t s);

// SHA-256 of the n_slots leaves of a leaf table (sha256_leaves.hip); digests
// go to digests + 32 * desc.out for desc.out < out_bound.
// Leaf table of leaves [first, first + k) into desc[0..k) (digest slot e for
// leaf first + e); also resets reset[0] = 0, reset[1] = ~0 when reset != NULL.
hipError_t launch_sched_range(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t first,
                              uint64_t k, LeafDesc* desc, uint64_t* reset, hipStream_t s);
// Monitor comparison: for e < k, digest e (D bytes at digests + D*e) against
// reference leaf first + e (ref + D*(first + e)); result[0] += mismatches,
// result[1] = min(result[1], lowest mismatching leaf number).  D is 32 or 48.
hipError_t launch_monitor_compare(const uint8_t* digests, const uint8_t* ref, uint64_t first, uint64_t k, uint32_t D,
                                  uint64_t* result, hipStream_t s);
// The two-wave SHA-256 leaf kernel (sha256_split.hip; same contract as
// launch_sha256_leaves), with one or two producer/consumer pairs per
// workgroup.  The automatic choice takes it for up to 128 leaves per compute
// unit of the current device (32768 on a 256-CU device).
hipError_t launch_sha256_split(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                               bool two_pairs, hipStream_t s);
// The two-wave SHA-384 leaf kernel (sha384_split.hip; same contract as
// launch_sha384_leaves), one or two pairs per workgroup.
hipError_t launch_sha384_split(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                               bool two_pairs, hipStream_t s);
// SHA-384 leaf digests with the kernel the choice selects (the callers' entry),
// by the same rules as launch_sha256_auto.
hipError_t launch_sha384_auto(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                              hipStream_t s, bool background = false);
// The leaf kernel a call over n_slots leaves takes under this thread's choice
// on the current device: 1 one-wave, 2 two-wave with one pair per workgroup,
// 3 two-wave with two pairs (both hashes use this rule).
int leaf_kernel_for(uint64_t n_slots, bool background);
// Compute units of the current device (queried once per device; 0 if the
// query fails, which makes the automatic choices take the one-wave kernels).
uint32_t device_cus();
// Leaf-kernel choice of the calling thread (hv_set_leaf_kernel): 0 automatic,
// 1 one-wave kernel, 2 two-wave kernel, 3 two-wave kernel with two pairs per
// workgroup.
int leaf_kernel_choice();
// SHA-256 leaf digests with the kernel that choice selects (the callers' entry).
// background: work that shares the chip with other work (monitor scans);
// under the automatic choice it takes the one-wave kernel, which hashes a byte
// in the least CU time, rather than the one with the shortest chains.
hipError_t launch_sha256_auto(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                              hipStream_t s, bool background = false);
hipError_t launch_sha256_leaves(const LeafDesc* desc, uint64_t n_slots, uint64_t out_bound, uint8_t* digests,
                                hipStream_t s);

// Merkle tiles (merkle.hip).  One launch reduces every segment by up to
// kTileLevels levels: tile t covers up to 2^kTileLevels consecutive nodes of
// one segment and writes one node.
constexpr int kTileLevels = 9;
constexpr int kTileNodes = 1 << kTileLevels;
hipError_t launch_merkle_tiles(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                               const uint64_t* tile_off, uint32_t n_seg, uint64_t n_tiles, int leaf_mode,
                               hipStream_t s);
// Merkle groups (merkle.hip), the launches over the widest levels: group g
// -- up to 2^kGroupLevels consecutive nodes of one segment, starting at a
// multiple of that -- is reduced to one node in registers, by one lane for
// g < n_main and by four lanes (two entries each, then two shuffle levels)
// for the launch's last groups, g >= n_main.
constexpr int kGroupLevels = 3;
constexpr int kGroupNodes = 1 << kGroupLevels;
constexpr int kGroupQuad = 4;  // lanes per group beyond n_main
hipError_t launch_merkle_groups(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                const uint64_t* grp_off, uint32_t n_seg, uint64_t n_groups, uint64_t n_main,
                                int leaf_mode, hipStream_t s);

// Persistent tree for incremental updates (tree.hip).
hipError_t launch_tree_leaf_level(int alg, const uint8_t* digests, uint64_t n, uint8_t* level0, hipStream_t s);
hipError_t launch_tree_build_level(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                   const uint64_t* out_off, uint32_t n_seg, uint64_t n_out, hipStream_t s);
hipError_t launch_tree_locate(const uint64_t* dirty, uint32_t k, const uint64_t* seg_off, uint32_t n_seg,
                              uint32_t* seg_of, uint64_t* local, hipStream_t s);
hipError_t launch_tree_update_leaves(int alg, const uint8_t* digests, const uint64_t* dirty, uint32_t k,
                                     uint8_t* level0, hipStream_t s);
hipError_t launch_tree_update_level(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                    const uint64_t* out_off, const uint32_t* seg_of, const uint64_t* local, uint32_t k,
                                    uint32_t shift, hipStream_t s);
hipError_t launch_tree_roots(int alg, const uint8_t* top, const uint64_t* top_off, uint32_t n_seg, uint8_t* roots,
                             hipStream_t s);

// Verification (verify.hip).
// nbytes: 32 or 48 (the digest size of the call's hash).
hipError_t launch_verify_root(const uint8_t* root, const uint8_t* expected, uint32_t nbytes, uint32_t* flag,
                              hipStream_t s);
// As launch_verify_root with `expected` (nbytes) in device memory.
hipError_t launch_verify_root_dev(const uint8_t* root, const uint8_t* expected, uint32_t nbytes, uint32_t* flag,
                                  hipStream_t s);
hipError_t launch_compare_roots(const uint8_t* roots, const uint8_t* expected, uint32_t n, uint32_t nbytes,
                                uint32_t* mismatch, hipStream_t s);

}  // namespace hv
