// hv_kernels.h -- launchers shared between the kernel sources and the C ABI.
// Every launcher queues work on `stream` and returns the launch status; it
// trusts its arguments (the C ABI validates them first).
#pragma once
#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime.h>

namespace hv {

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

// Scheduler (sched.hip).
hipError_t launch_fill_u64(uint64_t* p, size_t n, uint64_t v, hipStream_t s);
hipError_t launch_sched_count(const MsgDesc* msgs, uint32_t n, uint64_t C, Pair* cnt, hipStream_t s);
size_t scan_partials_count(size_t n);
hipError_t launch_scan_pairs(const Pair* in, Pair* out, size_t n, Pair* partials, hipStream_t s);
hipError_t launch_sched_full(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                             LeafDesc* desc, hipStream_t s);
hipError_t launch_sched_tails(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                              uint64_t* hist, LeafDesc* desc, hipStream_t s);

// SHA-256 of every leaf (sha256_leaves.hip).
hipError_t launch_sha256_leaves(const LeafDesc* desc, uint64_t n_leaves, uint8_t* digests, hipStream_t s);

// Merkle tiles (merkle.hip).  One launch reduces every segment by up to
// kTileLevels levels: tile t covers up to 2^kTileLevels consecutive nodes of
// one segment and writes one node.
constexpr int kTileLevels = 9;
constexpr int kTileNodes = 1 << kTileLevels;
hipError_t launch_merkle_tiles(const uint8_t* in, uint8_t* out, const uint64_t* in_off, const uint64_t* tile_off,
                               uint32_t n_seg, uint64_t n_tiles, int leaf_mode, hipStream_t s);

// Verification (verify.hip).
hipError_t launch_verify_root(const uint8_t* root, const uint32_t expected_le[8], uint32_t* flag, hipStream_t s);
hipError_t launch_compare_roots(const uint8_t* roots, const uint8_t* expected, uint32_t n, uint32_t* mismatch,
                                hipStream_t s);

}  // namespace hv
