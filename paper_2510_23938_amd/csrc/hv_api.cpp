// hv_api.cpp -- the C ABI declared in include/hv.h: argument validation,
// workspace carving and the launch sequence on the caller's stream.  All
// arithmetic on message bytes and digests runs in the kernels; the host only
// plans (offsets and counts from the descriptor array) and launches.
#include "hv.h"
#include "hv_inspect.h"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <thread>
#include <vector>

#include "hv_host.h"
#include "hv_kernels.h"

namespace hvh {

thread_local char g_error[512] = "";

hv_status fail(hv_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return st;
}

hv_status hip_fail(hipError_t e, const char* what) {
    return fail(HV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

HashLayout hash_layout(void* ws, uint32_t n_msgs, uint64_t n_leaves) {
    Carver c(ws);
    HashLayout L;
    L.msgs = c.take<hv::MsgDesc>(n_msgs);
    L.cnt = c.take<hv::Pair>(n_msgs);
    L.off = c.take<hv::Pair>((size_t)n_msgs + 1);
    L.partials = c.take<hv::Pair>(hv::scan_partials_count(n_msgs));
    L.hist = c.take<uint64_t>(hv::kSortBuckets);
    L.desc = c.take<hv::LeafDesc>(n_leaves);
    L.bytes = c.used;
    return L;
}

namespace {

// Why a message is refused (kNone: it is not).
enum BadMsg : int { kNone = 0, kNullData, kWraps, kChunkTooLarge, kCountOverflow };

// Validates messages [lo, hi) and counts their leaves (and full chunks); with
// seg_offsets, writes seg_offsets[m + 1] = base + leaves of messages lo..m.
// Stops at the first refused message: *bad_at and the returned reason.
BadMsg scan_messages(const hv_msg* msgs, uint32_t lo, uint32_t hi, uint64_t C, uint64_t base,
                     uint64_t* seg_offsets, uint64_t* leaves_out, uint64_t* full_out, uint32_t* bad_at) {
    uint64_t total = 0, full = 0;
    for (uint32_t m = lo; m < hi; ++m) {
        const uint64_t len = msgs[m].nbytes;
        BadMsg why = kNone;
        if (len > 0 && msgs[m].data == nullptr) why = kNullData;
        else if ((uintptr_t)msgs[m].data + len < (uintptr_t)msgs[m].data) why = kWraps;
        else if ((C == 0 || len < C ? len : C) > kMaxChunkBytes) why = kChunkTooLarge;
        uint64_t leaves = 0;
        if (why == kNone) {
            if (C == 0) {
                leaves = 1;
            } else {
                leaves = len / C + (len % C != 0);
                full += len / C;
            }
            if (total + leaves < total || base + total + leaves < base) why = kCountOverflow;
        }
        if (why != kNone) {
            *bad_at = m;
            return why;
        }
        total += leaves;
        if (seg_offsets) seg_offsets[m + 1] = base + total;
    }
    *leaves_out = total;
    *full_out = full;
    return kNone;
}

hv_status refuse(const hv_msg* msgs, uint32_t m, uint64_t C, BadMsg why) {
    switch (why) {
        case kNullData:
            return fail(HV_ERR_INVALID_ARG, "message %u has NULL data and %llu bytes", m,
                        (unsigned long long)msgs[m].nbytes);
        case kWraps:
            return fail(HV_ERR_INVALID_ARG, "message %u wraps the address space", m);
        case kChunkTooLarge: {
            const uint64_t len = msgs[m].nbytes;
            return fail(HV_ERR_INVALID_ARG, "message %u: a chunk of %llu bytes exceeds the %llu-byte limit", m,
                        (unsigned long long)(C == 0 || len < C ? len : C), (unsigned long long)kMaxChunkBytes);
        }
        default:
            return fail(HV_ERR_INVALID_ARG, "leaf count overflows");
    }
}

// Message tables at least this long are scanned by several host threads.
constexpr uint32_t kParallelScanMin = 1u << 16;

// Runs body(0 .. T-1), body(0) on the calling thread.  Returns false when the
// host could not start every thread (the parts that ran are then incomplete).
template <class F>
bool run_parts(unsigned T, F&& body) {
    std::vector<std::thread> pool;
    bool started = true;
    try {
        pool.reserve(T - 1);
        for (unsigned t = 1; t < T; ++t) pool.emplace_back(body, t);
    } catch (...) {
        started = false;
    }
    body(0u);
    for (auto& th : pool) th.join();
    return started;
}

enum class Parallel { kDone, kRefused, kUnavailable };

// layout's pass split over T threads: counts per part, then (with
// seg_offsets) the offsets of each part from its base.  kRefused: the lowest
// refused message is reported through fail(); kUnavailable: threads could
// not be started and nothing the caller keeps was written but seg_offsets
// entries the single pass rewrites.
Parallel parallel_layout(const hv_msg* msgs, uint32_t n_msgs, uint64_t C, uint64_t* seg_offsets, unsigned T,
                         uint64_t* total_out, uint64_t* full_out) {
    std::vector<uint64_t> leaves(T, 0), fulls(T, 0), base(T, 0);
    std::vector<uint32_t> bad(T, 0);
    std::vector<BadMsg> why(T, kNone);
    auto part = [&](unsigned t) { return (uint32_t)((uint64_t)n_msgs * t / T); };
    if (!run_parts(T, [&](unsigned t) {
            why[t] = scan_messages(msgs, part(t), part(t + 1), C, 0, nullptr, &leaves[t], &fulls[t], &bad[t]);
        }))
        return Parallel::kUnavailable;
    uint64_t total = 0, full = 0;
    for (unsigned t = 0; t < T; ++t) {
        if (why[t] != kNone) {
            (void)refuse(msgs, bad[t], C, why[t]);
            return Parallel::kRefused;
        }
        if (total + leaves[t] < total) {
            (void)fail(HV_ERR_INVALID_ARG, "leaf count overflows");
            return Parallel::kRefused;
        }
        base[t] = total;
        total += leaves[t];
        full += fulls[t];
    }
    if (seg_offsets && !run_parts(T, [&](unsigned t) {
            uint64_t l, f;
            uint32_t b;
            (void)scan_messages(msgs, part(t), part(t + 1), C, base[t], seg_offsets, &l, &f, &b);
        }))
        return Parallel::kUnavailable;
    *total_out = total;
    *full_out = full;
    return Parallel::kDone;
}

}  // namespace

// Leaf counts of a message list; fills seg_offsets when given.  Large tables
// are split over host threads (a single pass when threads cannot be started);
// whatever the split, the error reported is the one of the lowest refused
// message, as a single pass would report it.
hv_status layout(const hv_msg* msgs, uint32_t n_msgs, uint64_t C, uint64_t* seg_offsets, uint64_t* n_leaves,
                 uint64_t* n_full) {
    if (n_msgs > 0 && msgs == nullptr) return fail(HV_ERR_INVALID_ARG, "msgs is NULL with n_msgs = %u", n_msgs);
    if (C % 64 != 0) return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 64",
                                 (unsigned long long)C);
    if (seg_offsets) seg_offsets[0] = 0;
    unsigned T = 1;
    if (n_msgs >= kParallelScanMin) {
        const unsigned hw = std::thread::hardware_concurrency();
        T = hw == 0 ? 1 : (hw < 16 ? hw : 16);
    }
    uint64_t total = 0, full = 0;
    Parallel got = Parallel::kUnavailable;
    if (T > 1) got = parallel_layout(msgs, n_msgs, C, seg_offsets, T, &total, &full);
    if (got == Parallel::kRefused) return HV_ERR_INVALID_ARG;
    if (got == Parallel::kUnavailable) {
        uint32_t bad = 0;
        const BadMsg why = scan_messages(msgs, 0, n_msgs, C, 0, seg_offsets, &total, &full, &bad);
        if (why != kNone) return refuse(msgs, bad, C, why);
    }
    *n_leaves = total;
    if (n_full) *n_full = full;
    return HV_OK;
}

}  // namespace hvh

using namespace hvh;

namespace {

struct Timing {
    bool enabled = false;
    bool have = false;
    hipEvent_t start = nullptr, stop = nullptr;
};
thread_local Timing g_timing;
thread_local int g_leaf_kernel = 0;

constexpr int kMaxLaunches = kMaxMerkleLaunches;

struct MerkleLayout {
    uint64_t* table;
    uint8_t* ping;
    uint8_t* pong;
    size_t bytes;
};

uint32_t digest_bytes(hv_alg alg) { return alg == HV_SHA384 ? 48 : 32; }

MerkleLayout merkle_layout(void* ws, uint64_t n_nodes, uint32_t n_seg, uint32_t D) {
    Carver c(ws);
    MerkleLayout L;
    L.table = c.take<uint64_t>((size_t)(kMaxLaunches + 1) * ((size_t)n_seg + 1));
    const uint64_t nb = merkle_tiles_bound(n_nodes, n_seg);
    L.ping = c.take<uint8_t>(nb * D);
    L.pong = c.take<uint8_t>(nb * D);
    L.bytes = c.used;
    return L;
}

}  // namespace

namespace hvh {

uint64_t merkle_tiles_bound(uint64_t n_nodes, uint32_t n_seg) {
    // a launch over c entries of a segment writes max(1, ceil(c / w)) <= c / w + 1 nodes
    const uint64_t w = merkle_grouped(n_nodes) ? (uint64_t)hv::kGroupNodes : (uint64_t)hv::kTileNodes;
    return n_nodes / w + (uint64_t)n_seg + 1;
}

hv_status check_segments(const uint64_t* seg_offsets, uint32_t n_seg) {
    if (seg_offsets[0] != 0) return fail(HV_ERR_INVALID_ARG, "seg_offsets[0] = %llu, not 0",
                                         (unsigned long long)seg_offsets[0]);
    for (uint32_t s = 0; s < n_seg; ++s)
        if (seg_offsets[s + 1] < seg_offsets[s])
            return fail(HV_ERR_INVALID_ARG, "seg_offsets decreases at segment %u", s);
    if (seg_offsets[n_seg] > kMaxLeaves)
        return fail(HV_ERR_INVALID_ARG, "%llu entries exceed the per-call limit",
                    (unsigned long long)seg_offsets[n_seg]);
    return HV_OK;
}

hv_status merkle_plan(const uint64_t* seg_offsets, uint32_t n_seg, std::vector<uint64_t>* table, int* launches) {
    const size_t row = (size_t)n_seg + 1;
    table->assign(seg_offsets, seg_offsets + row);
    int k = 0;
    for (;;) {
        const uint64_t entries = (*table)[(size_t)k * row + n_seg];
        const uint64_t w = merkle_width(entries);
        std::vector<uint64_t> next(row);
        next[0] = 0;
        bool more = false;
        for (uint32_t s = 0; s < n_seg; ++s) {
            const uint64_t* prev = table->data() + (size_t)k * row;
            const uint64_t c = prev[s + 1] - prev[s];
            const uint64_t tiles = c <= w ? 1 : (c + w - 1) / w;
            if (tiles > 1) more = true;
            next[s + 1] = next[s] + tiles;
        }
        table->insert(table->end(), next.begin(), next.end());
        ++k;
        if (!more) break;
        if (k == kMaxMerkleLaunches) return fail(HV_ERR_INVALID_ARG, "tree too deep");
    }
    *launches = k;
    return HV_OK;
}

namespace {

constexpr int kCuDevices = 64;
std::atomic<uint32_t> g_cus[kCuDevices];  // compute units per device, 0 until asked

// Compute units of device `dev`, asked once per device.
hipError_t device_cus(int dev, uint32_t* cus) {
    if (dev < 0 || dev >= kCuDevices) return hipErrorInvalidDevice;
    uint32_t n = g_cus[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        int v = 0;
        const hipError_t e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        n = v > 0 ? (uint32_t)v : 0u;
        g_cus[dev].store(n, std::memory_order_relaxed);
    }
    *cus = n;
    return hipSuccess;
}

hipError_t stream_cus(hipStream_t stream, uint32_t* cus) {
    int dev = -1;
    const hipError_t e = hipStreamGetDevice(stream, &dev);
    return e != hipSuccess ? e : device_cus(dev, cus);
}

}  // namespace

hv_status merkle_launch_kinds(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg, uint32_t cus, int* launches,
                              int* kind, uint64_t* units, uint64_t* one_lane) {
    std::vector<uint64_t> table;
    hv_status st = merkle_plan(seg_offsets, n_seg, &table, launches);
    if (st != HV_OK) return st;
    const size_t row = (size_t)n_seg + 1;
    for (int k = 1; k <= *launches; ++k) {
        const uint64_t entries = table[(size_t)(k - 1) * row + n_seg], out = table[(size_t)k * row + n_seg];
        const bool grouped = merkle_grouped(entries);
        kind[k - 1] = grouped ? 1 : 2;
        units[k - 1] = out;
        one_lane[k - 1] = grouped ? merkle_group_main(out, k == 1, alg == HV_SHA384, cus) : 0;
    }
    return HV_OK;
}

hv_status queue_merkle(hv_alg alg, const uint8_t* in, uint8_t* out, const uint64_t* table, uint32_t n_seg,
                       uint64_t n_nodes, int launches, const uint64_t* outputs, uint8_t* ping, uint8_t* pong,
                       hipStream_t stream) {
    const size_t row = (size_t)n_seg + 1;
    const int a = alg == HV_SHA384 ? hv::kAlgSha384 : hv::kAlgSha256;
    uint32_t cus = 0;
    for (int k = 1; k <= launches; ++k) {
        uint8_t* dst = k == launches ? out : (k % 2 ? ping : pong);
        const uint64_t* in_off = table + (size_t)(k - 1) * row;
        const uint64_t* out_off = table + (size_t)k * row;
        const uint64_t entries = k == 1 ? n_nodes : outputs[k - 2];  // the plan's rule, from the same counts
        hipError_t e;
        if (merkle_grouped(entries)) {
            if (cus == 0 && (e = stream_cus(stream, &cus)) != hipSuccess) return hip_fail(e, "device query");
            const uint64_t n_main = merkle_group_main(outputs[k - 1], k == 1, alg == HV_SHA384, cus);
            e = hv::launch_merkle_groups(a, in, dst, in_off, out_off, n_seg, outputs[k - 1], n_main, k == 1, stream);
        } else {
            e = hv::launch_merkle_tiles(a, in, dst, in_off, out_off, n_seg, outputs[k - 1], k == 1, stream);
        }
        if (e != hipSuccess) return hip_fail(e, "merkle kernel");
        in = dst;
    }
    return HV_OK;
}

// Scheduling kernels over device-resident descriptors: the leaf table of
// n_msgs messages goes to L.desc (which must be sized for n_leaves).
hv_status queue_schedule(const hv::MsgDesc* msgs_dev, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t n_full,
                         uint64_t n_leaves, const HashLayout& L, hipStream_t stream) {
    hipError_t e;
    if ((e = hv::launch_sched_count(msgs_dev, n_msgs, chunk_bytes, L.cnt, stream)) != hipSuccess)
        return hip_fail(e, "count kernel");
    if ((e = hv::launch_scan_pairs(L.cnt, L.off, n_msgs, L.partials, stream)) != hipSuccess)
        return hip_fail(e, "scan kernels");
    if (n_full > 0 &&
        (e = hv::launch_sched_full(msgs_dev, L.off, n_msgs, chunk_bytes, n_full, L.desc, stream)) != hipSuccess)
        return hip_fail(e, "full-chunk kernel");
    if (n_leaves > n_full &&
        (e = hv::launch_sched_tails(msgs_dev, L.off, n_msgs, chunk_bytes, n_full, L.hist, L.desc, stream)) !=
            hipSuccess)
        return hip_fail(e, "tail sort kernels");
    return HV_OK;
}

}  // namespace hvh

namespace {

// A descriptor upload started before the host validates the table, so that
// the DMA runs under the validation.  The host array is consumed once wait()
// returns; every path out of a call that started one goes through wait().
constexpr uint32_t kEarlyUploadMin = 4096;  // smaller tables upload in a few microseconds
constexpr int kEventDevices = 64;
thread_local hipEvent_t g_upload_event[kEventDevices] = {};  // per thread and device, kept for the thread's life

// This thread's upload event for the device that owns `stream` (an event
// records only on streams of the device it was made on).
hipError_t upload_event(hipStream_t stream, hipEvent_t* ev) {
    int dev = -1;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kEventDevices) return hipErrorInvalidDevice;
    if (g_upload_event[dev] == nullptr) {
        int cur = -1;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
        hipEvent_t made = nullptr;
        e = hipEventCreateWithFlags(&made, hipEventDisableTiming);
        if (cur != dev) {
            const hipError_t back = hipSetDevice(cur);
            if (e == hipSuccess) e = back;
        }
        if (e != hipSuccess) return e;
        g_upload_event[dev] = made;
    }
    *ev = g_upload_event[dev];
    return hipSuccess;
}

struct Upload {
    hipEvent_t ev = nullptr;
    bool pending = false;
    hv_status wait(hv_status st) {
        if (!pending) return st;
        pending = false;
        const hipError_t e = hipEventSynchronize(ev);
        return st == HV_OK && e != hipSuccess ? hip_fail(e, "descriptor upload") : st;
    }
};

// Validation plus the scheduling kernels shared by hv_hash_chunks and
// hv_leaf_schedule.  On HV_OK the leaf table is queued into L.desc.  With
// early_upload, a large descriptor table is copied asynchronously while the
// host validates it; the caller then queues its own kernels and calls
// up->wait() before returning (on an error, schedule has already waited).
hv_status schedule(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, bool need_out, const void* out,
                   void* workspace, size_t workspace_bytes, bool early_upload, Upload* up, hipStream_t stream,
                   HashLayout* L_out, uint64_t* n_leaves_out) {
    static_assert(sizeof(hv_msg) == sizeof(hv::MsgDesc), "hv_msg layout");
    // The descriptors are the workspace's first region; start their copy when
    // the workspace can hold them (it is scratch, whatever the checks find).
    if (early_upload && n_msgs >= kEarlyUploadMin && msgs != nullptr && chunk_bytes % 64 == 0 &&
        workspace != nullptr && (uintptr_t)workspace % kAlign == 0 &&
        workspace_bytes >= round_up(sizeof(hv_msg) * (size_t)n_msgs)) {
        hipError_t e = upload_event(stream, &up->ev);
        if (e == hipSuccess) e = hipMemcpyAsync(workspace, msgs, sizeof(hv_msg) * n_msgs, hipMemcpyHostToDevice, stream);
        if (e == hipSuccess) {
            up->pending = true;
            e = hipEventRecord(up->ev, stream);
            if (e != hipSuccess) {
                // no event to wait on: wait for the stream itself before the host array is released
                up->pending = false;
                (void)hipStreamSynchronize(stream);
            }
        }
        if (e != hipSuccess) return hip_fail(e, "descriptor upload");
    }
    uint64_t n_leaves = 0, n_full = 0;
    hv_status st = layout(msgs, n_msgs, chunk_bytes, nullptr, &n_leaves, &n_full);
    if (st != HV_OK) return up->wait(st);
    if (n_leaves > kMaxLeaves)
        return up->wait(fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit", (unsigned long long)n_leaves));
    if (need_out && n_leaves > 0 && out == nullptr) return up->wait(fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL"));
    if (need_out && (uintptr_t)out % 16 != 0)
        return up->wait(fail(HV_ERR_INVALID_ARG, "leaf_digests is not 16-byte aligned"));
    if (!need_out && n_leaves > 0 && out == nullptr) return up->wait(fail(HV_ERR_INVALID_ARG, "table is NULL"));
    const HashLayout need = hash_layout(nullptr, n_msgs, n_leaves);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return up->wait(fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu%s", need.bytes, workspace_bytes,
                             workspace ? "" : " (NULL)"));
    if ((uintptr_t)workspace % kAlign != 0) return up->wait(fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned"));
    *n_leaves_out = n_leaves;
    *L_out = hash_layout(workspace, n_msgs, n_leaves);
    if (n_msgs == 0) return HV_OK;

    const HashLayout& L = *L_out;
    if (!up->pending) {
        const hipError_t e = hipMemcpyWithStream(L.msgs, msgs, sizeof(hv_msg) * n_msgs, hipMemcpyHostToDevice, stream);
        if (e != hipSuccess) return hip_fail(e, "descriptor upload");
    }
    st = hvh::queue_schedule(L.msgs, n_msgs, chunk_bytes, n_full, n_leaves, L, stream);
    return st == HV_OK ? st : up->wait(st);
}

}  // namespace

namespace hvh {

hv_status hash_chunks_into(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                           uint8_t* leaf_digests, void* workspace, size_t workspace_bytes, bool events,
                           hipStream_t stream) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (alg == HV_SHA384 && chunk_bytes % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)chunk_bytes);
    HashLayout L;
    uint64_t n_leaves = 0;
    // with events, the descriptor upload overlaps the validation
    Upload up;
    hv_status st = schedule(msgs, n_msgs, chunk_bytes, true, leaf_digests, workspace, workspace_bytes, events, &up,
                            stream, &L, &n_leaves);
    if (st != HV_OK) return st;
    if (n_leaves == 0) return up.wait(HV_OK);

    if (events && (st = leaf_timing_start(stream)) != HV_OK) return up.wait(st);
    const hipError_t e = alg == HV_SHA384 ? hv::launch_sha384_auto(L.desc, n_leaves, n_leaves, leaf_digests, stream)
                                          : hv::launch_sha256_auto(L.desc, n_leaves, n_leaves, leaf_digests, stream);
    if (e != hipSuccess) return up.wait(hip_fail(e, "leaf kernel"));
    return up.wait(events ? leaf_timing_stop(stream) : HV_OK);
}

}  // namespace hvh

extern "C" {

const char* hv_last_error(void) { return g_error; }

hv_status hv_leaf_layout(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t* seg_offsets,
                         uint64_t* n_leaves) {
    if (n_leaves == nullptr) return fail(HV_ERR_INVALID_ARG, "n_leaves is NULL");
    return layout(msgs, n_msgs, chunk_bytes, seg_offsets, n_leaves, nullptr);
}

size_t hv_hash_workspace_bytes(uint32_t n_msgs, uint64_t n_leaves) {
    if (n_leaves > kMaxLeaves) {
        (void)fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit", (unsigned long long)n_leaves);
        return 0;
    }
    return hash_layout(nullptr, n_msgs, n_leaves).bytes;
}

hv_status hv_hash_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                             uint8_t* leaf_digests, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return hash_chunks_into(alg, msgs, n_msgs, chunk_bytes, leaf_digests, workspace, workspace_bytes, true, stream);
}

hv_status hv_hash_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint8_t* leaf_digests,
                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return hv_hash_chunks_alg(HV_SHA256, msgs, n_msgs, chunk_bytes, leaf_digests, workspace, workspace_bytes, stream);
}

hv_status hv_leaf_schedule(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t* table,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
    HashLayout L;
    uint64_t n_leaves = 0;
    Upload up;
    hv_status st = schedule(msgs, n_msgs, chunk_bytes, false, table, workspace, workspace_bytes, true, &up, stream,
                            &L, &n_leaves);
    if ((st = up.wait(st)) != HV_OK || n_leaves == 0) return st;
    static_assert(sizeof(hv::LeafDesc) == 3 * sizeof(uint64_t), "leaf table layout");
    hipError_t e = hipMemcpyAsync(table, L.desc, n_leaves * sizeof(hv::LeafDesc), hipMemcpyDeviceToHost, stream);
    if (e != hipSuccess) return hip_fail(e, "table copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "stream synchronize");
    return HV_OK;
}

size_t hv_merkle_workspace_bytes_alg(hv_alg alg, uint64_t n_nodes, uint32_t n_seg) {
    if (alg != HV_SHA256 && alg != HV_SHA384) {
        (void)fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
        return 0;
    }
    if (n_nodes > kMaxLeaves) {
        (void)fail(HV_ERR_INVALID_ARG, "%llu entries exceed the per-call limit", (unsigned long long)n_nodes);
        return 0;
    }
    return merkle_layout(nullptr, n_nodes, n_seg, digest_bytes(alg)).bytes;
}

size_t hv_merkle_workspace_bytes(uint64_t n_nodes, uint32_t n_seg) {
    return hv_merkle_workspace_bytes_alg(HV_SHA256, n_nodes, n_seg);
}

hv_status hv_merkle_reduce_alg(hv_alg alg, const uint8_t* nodes, const uint64_t* seg_offsets, uint32_t n_seg,
                               uint8_t* roots, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    const uint32_t D = digest_bytes(alg);
    if (n_seg == 0) return fail(HV_ERR_INVALID_ARG, "n_seg is 0");
    if (seg_offsets == nullptr) return fail(HV_ERR_INVALID_ARG, "seg_offsets is NULL");
    if (roots == nullptr) return fail(HV_ERR_INVALID_ARG, "roots is NULL");
    hv_status st = check_segments(seg_offsets, n_seg);
    if (st != HV_OK) return st;
    const uint64_t n_nodes = seg_offsets[n_seg];
    if (n_nodes > 0 && nodes == nullptr) return fail(HV_ERR_INVALID_ARG, "nodes is NULL");
    if ((uintptr_t)nodes % 16 != 0 || (uintptr_t)roots % 16 != 0)
        return fail(HV_ERR_INVALID_ARG, "nodes and roots must be 16-byte aligned");
    const MerkleLayout need = merkle_layout(nullptr, n_nodes, n_seg, D);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu%s", need.bytes, workspace_bytes,
                    workspace ? "" : " (NULL)");
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");

    // Plan on the host: rows of n_seg + 1 offsets, one per launch level.
    const size_t row = (size_t)n_seg + 1;
    std::vector<uint64_t> table;
    int launches = 0;
    if ((st = merkle_plan(seg_offsets, n_seg, &table, &launches)) != HV_OK) return st;

    const MerkleLayout L = merkle_layout(workspace, n_nodes, n_seg, D);
    const hipError_t e = hipMemcpyWithStream(L.table, table.data(), table.size() * sizeof(uint64_t),
                                             hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "plan upload");
    uint64_t outputs[kMaxMerkleLaunches];
    for (int k = 1; k <= launches; ++k) outputs[k - 1] = table[(size_t)k * row + n_seg];
    return queue_merkle(alg, nodes, roots, L.table, n_seg, n_nodes, launches, outputs, L.ping, L.pong, stream);
}

hv_status hv_merkle_reduce(const uint8_t* nodes, const uint64_t* seg_offsets, uint32_t n_seg, uint8_t* roots,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return hv_merkle_reduce_alg(HV_SHA256, nodes, seg_offsets, n_seg, roots, workspace, workspace_bytes, stream);
}

size_t hv_verify_workspace_bytes(void) { return kAlign; }

hv_status hv_verify_root_alg(hv_alg alg, const uint8_t* root, const uint8_t* expected, int* match, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (root == nullptr || expected == nullptr || match == nullptr)
        return fail(HV_ERR_INVALID_ARG, "root, expected and match must be non-NULL");
    if (workspace == nullptr || workspace_bytes < hv_verify_workspace_bytes())
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes", hv_verify_workspace_bytes());
    if ((uintptr_t)workspace % 4 != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 4-byte aligned");
    uint32_t* flag = static_cast<uint32_t*>(workspace);
    hipError_t e = hv::launch_verify_root(root, expected, digest_bytes(alg), flag, stream);
    if (e != hipSuccess) return hip_fail(e, "verify kernel");
    uint32_t host_flag = 0;
    if ((e = hipMemcpyAsync(&host_flag, flag, sizeof host_flag, hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "flag copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "stream synchronize");
    *match = host_flag == 1 ? 1 : 0;
    return HV_OK;
}

hv_status hv_verify_root(const uint8_t* root, const uint8_t expected[32], int* match, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    return hv_verify_root_alg(HV_SHA256, root, expected, match, workspace, workspace_bytes, stream);
}

hv_status hv_compare_roots_alg(hv_alg alg, const uint8_t* roots, const uint8_t* expected, uint32_t n,
                               uint32_t* mismatch, hipStream_t stream) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (n > 0 && (roots == nullptr || expected == nullptr || mismatch == nullptr))
        return fail(HV_ERR_INVALID_ARG, "roots, expected and mismatch must be non-NULL");
    hipError_t e = hv::launch_compare_roots(roots, expected, n, digest_bytes(alg), mismatch, stream);
    if (e != hipSuccess) return hip_fail(e, "compare kernel");
    return HV_OK;
}

hv_status hv_compare_roots(const uint8_t* roots, const uint8_t* expected, uint32_t n, uint32_t* mismatch,
                           hipStream_t stream) {
    return hv_compare_roots_alg(HV_SHA256, roots, expected, n, mismatch, stream);
}

}  // extern "C"

namespace hv {
int leaf_kernel_choice() { return g_leaf_kernel; }
}  // namespace hv

namespace hvh {

hv_status leaf_timing_start(hipStream_t stream) {
    Timing& T = g_timing;
    if (!T.enabled) return HV_OK;
    hipError_t e;
    if (!T.start && (e = hipEventCreate(&T.start)) != hipSuccess) return hip_fail(e, "event create");
    if (!T.stop && (e = hipEventCreate(&T.stop)) != hipSuccess) return hip_fail(e, "event create");
    if ((e = hipEventRecord(T.start, stream)) != hipSuccess) return hip_fail(e, "event record");
    return HV_OK;
}

hv_status leaf_timing_stop(hipStream_t stream) {
    Timing& T = g_timing;
    if (!T.enabled) return HV_OK;
    const hipError_t e = hipEventRecord(T.stop, stream);
    if (e != hipSuccess) return hip_fail(e, "event record");
    T.have = true;
    return HV_OK;
}

}  // namespace hvh

extern "C" {

hv_status hv_set_leaf_kernel(int choice) {
    if (choice < 0 || choice > 3) return fail(HV_ERR_INVALID_ARG, "leaf kernel choice %d is not 0, 1, 2 or 3", choice);
    g_leaf_kernel = choice;
    return HV_OK;
}

hv_status hv_leaf_kernel_for(uint64_t n_leaves, int* kernel) {
    if (kernel == nullptr) return fail(HV_ERR_INVALID_ARG, "kernel is NULL");
    *kernel = hv::leaf_kernel_for(n_leaves, false);
    return HV_OK;
}

hv_status hv_merkle_launches(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg, uint32_t cus, int* launches,
                             int* kind, uint64_t* units, uint64_t* one_lane) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (n_seg == 0) return fail(HV_ERR_INVALID_ARG, "n_seg is 0");
    if (seg_offsets == nullptr || launches == nullptr || kind == nullptr || units == nullptr || one_lane == nullptr)
        return fail(HV_ERR_INVALID_ARG, "seg_offsets, launches, kind, units and one_lane must be non-NULL");
    hv_status st = check_segments(seg_offsets, n_seg);
    if (st != HV_OK) return st;
    if (cus == 0) {
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e == hipSuccess) e = device_cus(dev, &cus);
        if (e != hipSuccess) return hip_fail(e, "device query");
    }
    return merkle_launch_kinds(alg, seg_offsets, n_seg, cus, launches, kind, units, one_lane);
}

hv_status hv_set_kernel_timing(int enable) {
    g_timing.enabled = enable != 0;
    return HV_OK;
}

hv_status hv_leaf_kernel_ms(float* ms) {
    if (ms == nullptr) return fail(HV_ERR_INVALID_ARG, "ms is NULL");
    if (!g_timing.have) return fail(HV_ERR_INVALID_ARG, "no timed hv_hash_chunks call on this thread");
    hipError_t e = hipEventSynchronize(g_timing.stop);
    if (e != hipSuccess) return hip_fail(e, "event synchronize");
    if ((e = hipEventElapsedTime(ms, g_timing.start, g_timing.stop)) != hipSuccess) return hip_fail(e, "elapsed");
    return HV_OK;
}

}  // extern "C"
