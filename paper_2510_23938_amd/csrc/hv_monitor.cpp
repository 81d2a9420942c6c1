// hv_monitor.cpp -- C ABI of continuous runtime monitoring: a plan made once
// (message table and leaf offsets on the device), then scans that rehash a
// range of leaves and compare them with reference digests, with nothing but
// kernel launches per scan.
#include "hv.h"
#include "hv_host.h"
#include "hv_monitor.h"

using namespace hvh;

namespace {

struct PlanLayout {
    hv::MsgDesc* msgs;
    hv::Pair* cnt;
    hv::Pair* off;
    hv::Pair* partials;
    size_t bytes;
};

PlanLayout plan_layout(void* mem, uint32_t n_msgs) {
    Carver c(mem);
    PlanLayout P;
    P.msgs = c.take<hv::MsgDesc>(n_msgs);
    P.cnt = c.take<hv::Pair>(n_msgs);
    P.off = c.take<hv::Pair>((size_t)n_msgs + 1);
    P.partials = c.take<hv::Pair>(hv::scan_partials_count(n_msgs));
    P.bytes = c.used;
    return P;
}

struct ScanLayout {
    hv::LeafDesc* desc;
    uint8_t* digests;
    size_t bytes;
};

ScanLayout scan_layout(void* ws, uint32_t D, uint64_t k) {
    Carver c(ws);
    ScanLayout S;
    S.desc = c.take<hv::LeafDesc>(k);
    S.digests = c.take<uint8_t>((size_t)D * k);
    S.bytes = c.used;
    return S;
}

bool known(hv_alg alg) { return alg == HV_SHA256 || alg == HV_SHA384; }
uint32_t digest_size(hv_alg alg) { return alg == HV_SHA384 ? 48 : 32; }

}  // namespace

extern "C" {

size_t hv_monitor_plan_bytes(uint32_t n_msgs) { return plan_layout(nullptr, n_msgs).bytes; }

hv_status hv_monitor_init(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, void* plan_memory,
                          size_t plan_bytes, hv_monitor_plan* plan, hipStream_t stream) {
    if (!known(alg)) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (plan == nullptr) return fail(HV_ERR_INVALID_ARG, "plan is NULL");
    if (alg == HV_SHA384 && chunk_bytes % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)chunk_bytes);
    uint64_t n_leaves = 0;
    hv_status st = layout(msgs, n_msgs, chunk_bytes, nullptr, &n_leaves, nullptr);
    if (st != HV_OK) return st;
    if (n_leaves > kMaxLeaves) return fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit",
                                           (unsigned long long)n_leaves);
    const size_t need = hv_monitor_plan_bytes(n_msgs);
    if (plan_memory == nullptr || plan_bytes < need)
        return fail(HV_ERR_WORKSPACE, "plan memory needs %zu bytes, got %zu%s", need, plan_bytes,
                    plan_memory ? "" : " (NULL)");
    if ((uintptr_t)plan_memory % kAlign != 0) return fail(HV_ERR_WORKSPACE, "plan memory is not 256-byte aligned");
    const PlanLayout P = plan_layout(plan_memory, n_msgs);
    hipError_t e;
    if (n_msgs > 0) {
        static_assert(sizeof(hv_msg) == sizeof(hv::MsgDesc), "hv_msg layout");
        if ((e = hipMemcpyWithStream(P.msgs, msgs, sizeof(hv_msg) * n_msgs, hipMemcpyHostToDevice, stream)) !=
            hipSuccess)
            return hip_fail(e, "message table upload");
        if ((e = hv::launch_sched_count(P.msgs, n_msgs, chunk_bytes, P.cnt, stream)) != hipSuccess)
            return hip_fail(e, "count kernel");
    }
    if ((e = hv::launch_scan_pairs(P.cnt, P.off, n_msgs, P.partials, stream)) != hipSuccess)
        return hip_fail(e, "scan kernels");
    plan->device = plan_memory;
    plan->alg = alg;
    plan->n_msgs = n_msgs;
    plan->chunk_bytes = chunk_bytes;
    plan->n_leaves = n_leaves;
    return HV_OK;
}

size_t hv_monitor_scan_workspace_bytes(hv_alg alg, uint64_t max_slice) {
    if (!known(alg)) {
        (void)fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
        return 0;
    }
    if (max_slice > kMaxLeaves) {
        (void)fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit", (unsigned long long)max_slice);
        return 0;
    }
    return scan_layout(nullptr, digest_size(alg), max_slice).bytes;
}

hv_status hv_monitor_scan(const hv_monitor_plan* plan, uint64_t first_leaf, uint64_t n_slice,
                          const uint8_t* ref_digests, uint8_t* slice_digests, uint64_t* result, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
    if (plan == nullptr || plan->device == nullptr) return fail(HV_ERR_INVALID_ARG, "plan is NULL or not initialised");
    if (!known(plan->alg)) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)plan->alg);
    if (result == nullptr || (uintptr_t)result % 8 != 0)
        return fail(HV_ERR_INVALID_ARG, "result is NULL or not 8-byte aligned");
    if (first_leaf > plan->n_leaves || n_slice > plan->n_leaves - first_leaf)
        return fail(HV_ERR_INVALID_ARG, "leaves [%llu, %llu + %llu) are not within the %llu leaves of the plan",
                    (unsigned long long)first_leaf, (unsigned long long)first_leaf, (unsigned long long)n_slice,
                    (unsigned long long)plan->n_leaves);
    if (n_slice > 0 && ref_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "ref_digests is NULL");
    if ((uintptr_t)ref_digests % 16 != 0 || (uintptr_t)slice_digests % 16 != 0)
        return fail(HV_ERR_INVALID_ARG, "ref_digests and slice_digests must be 16-byte aligned");
    const uint32_t D = digest_size(plan->alg);
    const ScanLayout need = scan_layout(nullptr, D, n_slice);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu%s", need.bytes, workspace_bytes,
                    workspace ? "" : " (NULL)");
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");

    const PlanLayout P = plan_layout(plan->device, plan->n_msgs);
    const ScanLayout S = scan_layout(workspace, D, n_slice);
    uint8_t* out = slice_digests != nullptr ? slice_digests : S.digests;
    // the range kernel also resets `result`, so an empty slice reports no mismatch
    hipError_t e = hv::launch_sched_range(P.msgs, P.off, plan->n_msgs, plan->chunk_bytes, first_leaf, n_slice, S.desc,
                                          result, stream);
    if (e != hipSuccess) return hip_fail(e, "range kernel");
    if (n_slice == 0) return HV_OK;
    e = plan->alg == HV_SHA384 ? hv::launch_sha384_auto(S.desc, n_slice, n_slice, out, stream, true)
                               : hv::launch_sha256_auto(S.desc, n_slice, n_slice, out, stream, true);
    if (e != hipSuccess) return hip_fail(e, "leaf kernel");
    if ((e = hv::launch_monitor_compare(out, ref_digests, first_leaf, n_slice, D, result, stream)) != hipSuccess)
        return hip_fail(e, "compare kernel");
    return HV_OK;
}

hv_status hv_stream_create_cu_masked(const uint32_t* mask, uint32_t n_words, hipStream_t* stream) {
    if (mask == nullptr || stream == nullptr || n_words == 0)
        return fail(HV_ERR_INVALID_ARG, "mask and stream must be non-NULL and n_words > 0");
    int device = 0, n_cu = 0;
    hipError_t e = hipGetDevice(&device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return hip_fail(e, "device query");
    uint32_t selected = 0;
    for (int cu = 0; cu < n_cu && (uint32_t)cu < 32 * n_words; ++cu) selected += (mask[cu / 32] >> (cu % 32)) & 1u;
    if (selected == 0) return fail(HV_ERR_INVALID_ARG, "the mask selects none of the device's %d compute units", n_cu);
    if ((e = hipExtStreamCreateWithCUMask(stream, n_words, mask)) != hipSuccess) return hip_fail(e, "stream create");
    return HV_OK;
}

hv_status hv_stream_cu_mask(hipStream_t stream, uint32_t* mask, uint32_t n_words) {
    if (stream == nullptr || mask == nullptr || n_words == 0)
        return fail(HV_ERR_INVALID_ARG, "stream and mask must be non-NULL and n_words > 0");
    const hipError_t e = hipExtStreamGetCUMask(stream, n_words, mask);
    return e == hipSuccess ? HV_OK : hip_fail(e, "stream mask query");
}

hv_status hv_stream_destroy(hipStream_t stream) {
    if (stream == nullptr) return fail(HV_ERR_INVALID_ARG, "stream is NULL");
    hipError_t e = hipStreamSynchronize(stream);
    if (e == hipSuccess) e = hipStreamDestroy(stream);
    return e == hipSuccess ? HV_OK : hip_fail(e, "stream destroy");
}

}  // extern "C"
