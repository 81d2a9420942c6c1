// hv_host.h -- host-side internals shared by the C-ABI sources: argument
// errors, workspace carving and the scheduling launch sequence.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "hv.h"
#include "hv_kernels.h"

namespace hvh {

constexpr size_t kAlign = 256;
inline size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Largest leaf (or tree entry) count one call accepts.  It keeps the kernels'
// 32-bit grid-stride indices below 2^32 and is far above what fits in HBM
// (every leaf takes a 24-byte table entry and its digest besides its bytes).
constexpr uint64_t kMaxLeaves = (uint64_t)1 << 31;
// Largest chunk: the leaf kernels count a chunk's 64-byte blocks, padding
// blocks included, in 32 bits; 2^31 whole blocks leave room for the padding
// and for the kernels' rounding of block counts to pairs.
constexpr uint64_t kMaxChunkBytes = (uint64_t)1 << 37;

// Carves consecutive 256-byte-aligned regions out of a workspace.
struct Carver {
    uint8_t* base;
    size_t used = 0;
    explicit Carver(void* b) : base(static_cast<uint8_t*>(b)) {}
    template <typename T>
    T* take(size_t count) {
        T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
        used += round_up(count * sizeof(T));
        return p;
    }
};

struct HashLayout {
    hv::MsgDesc* msgs;
    hv::Pair* cnt;
    hv::Pair* off;
    hv::Pair* partials;
    uint64_t* hist;
    hv::LeafDesc* desc;
    size_t bytes;
};

HashLayout hash_layout(void* ws, uint32_t n_msgs, uint64_t n_leaves);

// Records a detail string for hv_last_error() and returns st.
hv_status fail(hv_status st, const char* fmt, ...);
hv_status hip_fail(hipError_t e, const char* what);

// Leaf counts of a message list (validation included); fills seg_offsets when given.
hv_status layout(const hv_msg* msgs, uint32_t n_msgs, uint64_t C, uint64_t* seg_offsets, uint64_t* n_leaves,
                 uint64_t* n_full);

// The body of hv_hash_chunks_alg over a given workspace (validation, descriptor
// upload, scheduling, leaf kernel).  With `events` the call may create and use
// HIP events: a large descriptor table is then uploaded asynchronously while
// the host validates it, and the leaf kernel is timed when
// hv_set_kernel_timing is on; without, it creates no runtime object.
hv_status hash_chunks_into(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                           uint8_t* leaf_digests, void* workspace, size_t workspace_bytes, bool events,
                           hipStream_t stream);

// Scheduling kernels over device-resident descriptors into L (leaf table in L.desc).
hv_status queue_schedule(const hv::MsgDesc* msgs_dev, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t n_full,
                         uint64_t n_leaves, const HashLayout& L, hipStream_t stream);

// Segmented Merkle reductions chain launches.  A launch whose input has at
// least kGroupMinNodes entries is a group launch (3 levels in registers, one
// lane per group of 8 entries: every lane busy on the widest levels); every
// other launch takes 9 levels (512-node tiles).  Up to 2^31 entries (the
// per-call limit) that is at most 5 group launches and 2 tile launches.
constexpr int kMaxMerkleLaunches = 8;
constexpr uint64_t kGroupMinNodes = (uint64_t)1 << 18;
inline bool merkle_grouped(uint64_t n_nodes) { return n_nodes >= kGroupMinNodes; }
// Entries one output node of a launch over n_nodes entries covers.
inline uint64_t merkle_width(uint64_t n_nodes) {
    return merkle_grouped(n_nodes) ? (uint64_t)hv::kGroupNodes : (uint64_t)hv::kTileNodes;
}

// Host plan of a segmented Merkle reduction over validated segment offsets:
// `table` gets rows of n_seg + 1 offsets -- row 0 the segment offsets, row k
// the first output node of each segment after launch k (a segment with c
// nodes gets max(1, ceil(c / w)) outputs, w = merkle_width(entries of row
// k - 1)) -- and `launches` the launch count.  Launch k is a group launch
// exactly when merkle_grouped(entries of row k - 1).
hv_status merkle_plan(const uint64_t* seg_offsets, uint32_t n_seg, std::vector<uint64_t>* table, int* launches);

// Segment offsets: start at 0, never decrease, at most the per-call entry limit.
hv_status check_segments(const uint64_t* seg_offsets, uint32_t n_seg);

// The launches a reduction of these (checked) segments makes on a device of
// `cus` compute units (hv_merkle_launches in hv_inspect.h).
hv_status merkle_launch_kinds(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg, uint32_t cus, int* launches,
                              int* kind, uint64_t* units, uint64_t* one_lane);

// Groups a group launch of n_groups groups gives one lane each (the rest, its
// last groups, get four lanes each), for a device of `cus` compute units
// (4 SIMDs each).  A wave of one-lane groups takes D block times (8 entries:
// the leaf hashes in leaf mode, then 7 nodes), a wave of four-lane groups d
// (2 entries, then 3 nodes along the chain) for a quarter of the groups.
// With R = 256 * cus groups per wave on every SIMD, all one-lane costs
// ceil(G / R) * D on the busiest SIMD; the split keeps floor(G / R) whole
// rounds and spreads the rest as four-lane waves, k * D + ceil(4r / R) * d.
// The split is taken when it costs less: it shortens the launch's last round,
// where one wave per SIMD would otherwise run alone.
inline uint64_t merkle_group_main(uint64_t n_groups, bool leaf_mode, bool sha384, uint32_t cus) {
    if (cus == 0) return n_groups;
    const uint64_t leaf = leaf_mode ? 1 : 0, node = sha384 ? 1 : 2;  // 64- or 128-byte blocks per hash
    const uint64_t D = 8 * leaf + 7 * node, d = 2 * leaf + 3 * node;
    const uint64_t R = 256 * (uint64_t)cus;
    const uint64_t k = n_groups / R, r = n_groups % R;
    if (k == 0 || r == 0) return n_groups;
    const uint64_t all = (k + 1) * D, split = k * D + (4 * r + R - 1) / R * d;
    return split < all ? k * R : n_groups;
}

// Nodes any launch of a reduction of n_nodes nodes in n_seg segments writes, at most.
uint64_t merkle_tiles_bound(uint64_t n_nodes, uint32_t n_seg);

// Queues the launches of a planned reduction: `in` (entries; the first launch
// forms their leaf hashes) through ping / pong into `out`.  table: the plan's
// rows on the device; outputs[k]: nodes written by launch k + 1.
hv_status queue_merkle(hv_alg alg, const uint8_t* in, uint8_t* out, const uint64_t* table, uint32_t n_seg,
                       uint64_t n_nodes, int launches, const uint64_t* outputs, uint8_t* ping, uint8_t* pong,
                       hipStream_t stream);

// HIP events around a leaf kernel on `stream` when hv_set_kernel_timing is on
// for this thread (no-ops otherwise).
hv_status leaf_timing_start(hipStream_t stream);
hv_status leaf_timing_stop(hipStream_t stream);

}  // namespace hvh
