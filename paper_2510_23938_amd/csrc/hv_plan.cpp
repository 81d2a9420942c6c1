// hv_plan.cpp -- prepared verification: the host work for one message set
// (message table, leaf table, Merkle launch tables) done once, then runs that
// only queue kernels on the caller's stream.
#include <algorithm>
#include <chrono>
#include <cstring>
#include <vector>

#include "hv.h"
#include "hv_host.h"
#include "hv_plan.h"

using namespace hvh;

namespace {

struct PlanMem {
    HashLayout hash;     // message table, scheduler scratch, leaf table
    uint64_t* table[2];  // Merkle launch tables: first tree, manifest
    uint8_t* ping;
    uint8_t* pong;
    size_t bytes;
};

// rows[i] = entries of Merkle table i; scratch = nodes held by each of ping and pong.
PlanMem plan_mem(void* mem, uint32_t n_msgs, uint64_t n_leaves, const size_t rows[2], uint64_t scratch, uint32_t D) {
    PlanMem P;
    P.hash = hash_layout(mem, n_msgs, n_leaves);
    Carver c(mem);
    c.used = P.hash.bytes;
    P.table[0] = c.take<uint64_t>(rows[0]);
    P.table[1] = c.take<uint64_t>(rows[1]);
    P.ping = c.take<uint8_t>(scratch * D);
    P.pong = c.take<uint8_t>(scratch * D);
    P.bytes = c.used;
    return P;
}

uint32_t digest_size(hv_alg alg) { return alg == HV_SHA384 ? 48 : 32; }

uint64_t scratch_nodes(uint64_t n_leaves, uint32_t n_seg, uint32_t n_msgs, int manifest) {
    const uint64_t first = n_seg > 0 ? merkle_tiles_bound(n_leaves, n_seg) : 0;
    const uint64_t top = manifest ? merkle_tiles_bound(n_msgs, 1) : 0;
    return std::max(first, top);
}

// Host-side preparation shared by hv_plan_bytes and hv_plan_init.
struct Prep {
    uint64_t n_leaves = 0, n_full = 0;
    uint32_t n_seg = 0;
    std::vector<uint64_t> table[2];
    int launches[2] = {0, 0};
    size_t rows[2] = {0, 0};
    uint64_t scratch = 0;
};

hv_status prepare(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t C, int manifest, Prep* p) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (alg == HV_SHA384 && C % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)C);
    std::vector<uint64_t> offs((size_t)n_msgs + 1, 0);
    hv_status st = layout(msgs, n_msgs, C, offs.data(), &p->n_leaves, &p->n_full);
    if (st != HV_OK) return st;
    if (p->n_leaves > kMaxLeaves)
        return fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit", (unsigned long long)p->n_leaves);
    std::vector<uint64_t> seg;
    if (manifest) {
        p->n_seg = n_msgs;
        seg = offs;
    } else {
        p->n_seg = 1;
        seg = {0, p->n_leaves};
    }
    if (p->n_seg > 0 && (st = merkle_plan(seg.data(), p->n_seg, &p->table[0], &p->launches[0])) != HV_OK) return st;
    if (manifest) {
        const uint64_t top[2] = {0, n_msgs};
        if ((st = merkle_plan(top, 1, &p->table[1], &p->launches[1])) != HV_OK) return st;
    }
    p->rows[0] = p->table[0].size();
    p->rows[1] = p->table[1].size();
    p->scratch = scratch_nodes(p->n_leaves, p->n_seg, n_msgs, manifest);
    return HV_OK;
}

// Workspace of hv_verify_model: the plan, then its outputs and the comparison buffers.
struct ModelLayout {
    void* plan;
    uint8_t* leaves;
    uint8_t* roots;
    uint8_t* root;
    uint8_t* expected;
    uint32_t* match;
    size_t bytes;
};

ModelLayout model_layout(void* ws, size_t plan_bytes, uint64_t n_leaves, uint32_t n_seg, uint32_t D) {
    Carver c(ws);
    ModelLayout M;
    M.plan = c.take<uint8_t>(plan_bytes);
    M.leaves = c.take<uint8_t>(n_leaves * D);
    M.roots = c.take<uint8_t>((size_t)std::max<uint32_t>(n_seg, 1) * D);
    M.root = c.take<uint8_t>(D);
    M.expected = c.take<uint8_t>(D);
    M.match = c.take<uint32_t>(1);
    M.bytes = c.used;
    return M;
}

}  // namespace

extern "C" {

size_t hv_plan_bytes(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest) {
    Prep p;
    if (prepare(alg, msgs, n_msgs, chunk_bytes, manifest != 0, &p) != HV_OK) return 0;
    return plan_mem(nullptr, n_msgs, p.n_leaves, p.rows, p.scratch, digest_size(alg)).bytes;
}

hv_status hv_plan_init(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest,
                       void* plan_memory, size_t plan_bytes, hv_verify_plan* plan, hipStream_t stream) {
    if (plan == nullptr) return fail(HV_ERR_INVALID_ARG, "plan is NULL");
    manifest = manifest != 0;
    Prep p;
    hv_status st = prepare(alg, msgs, n_msgs, chunk_bytes, manifest, &p);
    if (st != HV_OK) return st;
    const uint32_t D = digest_size(alg);
    const PlanMem need = plan_mem(nullptr, n_msgs, p.n_leaves, p.rows, p.scratch, D);
    if (plan_memory == nullptr || plan_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "plan memory needs %zu bytes, got %zu%s", need.bytes, plan_bytes,
                    plan_memory ? "" : " (NULL)");
    if ((uintptr_t)plan_memory % kAlign != 0) return fail(HV_ERR_WORKSPACE, "plan memory is not 256-byte aligned");
    const PlanMem P = plan_mem(plan_memory, n_msgs, p.n_leaves, p.rows, p.scratch, D);
    hipError_t e;
    static_assert(sizeof(hv_msg) == sizeof(hv::MsgDesc), "hv_msg layout");
    if (n_msgs > 0 &&
        (e = hipMemcpyWithStream(P.hash.msgs, msgs, sizeof(hv_msg) * n_msgs, hipMemcpyHostToDevice, stream)) !=
            hipSuccess)
        return hip_fail(e, "message table upload");
    for (int i = 0; i < 2; ++i)
        if (p.rows[i] > 0 && (e = hipMemcpyWithStream(P.table[i], p.table[i].data(), p.rows[i] * sizeof(uint64_t),
                                                      hipMemcpyHostToDevice, stream)) != hipSuccess)
            return hip_fail(e, "merkle table upload");
    if (n_msgs > 0 &&
        (st = queue_schedule(P.hash.msgs, n_msgs, chunk_bytes, p.n_full, p.n_leaves, P.hash, stream)) != HV_OK)
        return st;
    *plan = hv_verify_plan{};
    plan->device = plan_memory;
    plan->bytes = need.bytes;
    plan->alg = alg;
    plan->manifest = manifest;
    plan->n_msgs = n_msgs;
    plan->n_seg = p.n_seg;
    plan->chunk_bytes = chunk_bytes;
    plan->n_leaves = p.n_leaves;
    for (int i = 0; i < 2; ++i) {
        plan->launches[i] = (uint32_t)p.launches[i];
        const uint32_t segs = i == 0 ? p.n_seg : 1;
        for (int k = 0; k < p.launches[i]; ++k) plan->tiles[i][k] = p.table[i][(size_t)(k + 1) * (segs + 1) + segs];
    }
    return HV_OK;
}

hv_status hv_plan_run(const hv_verify_plan* plan, uint8_t* leaf_digests, uint8_t* roots, uint8_t* root,
                      const uint8_t* expected, uint32_t* match, hipStream_t stream) {
    if (plan == nullptr || plan->device == nullptr) return fail(HV_ERR_INVALID_ARG, "plan is NULL or not initialised");
    if (plan->alg != HV_SHA256 && plan->alg != HV_SHA384)
        return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)plan->alg);
    if (plan->launches[0] > HV_PLAN_MAX_LAUNCHES || plan->launches[1] > HV_PLAN_MAX_LAUNCHES)
        return fail(HV_ERR_INVALID_ARG, "plan is corrupt (launch counts)");
    const uint32_t D = digest_size(plan->alg);
    if (plan->n_leaves > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if (plan->n_seg > 0 && roots == nullptr) return fail(HV_ERR_INVALID_ARG, "roots is NULL");
    if (plan->manifest && root == nullptr) return fail(HV_ERR_INVALID_ARG, "root is NULL");
    if ((uintptr_t)leaf_digests % 16 || (uintptr_t)roots % 16 || (uintptr_t)root % 16)
        return fail(HV_ERR_INVALID_ARG, "leaf_digests, roots and root must be 16-byte aligned");
    if ((expected == nullptr) != (match == nullptr))
        return fail(HV_ERR_INVALID_ARG, "expected and match must both be given or both be NULL");
    if ((uintptr_t)match % 4 != 0) return fail(HV_ERR_INVALID_ARG, "match is not 4-byte aligned");
    const size_t rows[2] = {plan->n_seg > 0 ? ((size_t)plan->launches[0] + 1) * ((size_t)plan->n_seg + 1) : 0,
                            plan->manifest ? ((size_t)plan->launches[1] + 1) * 2 : 0};
    const uint64_t scratch = scratch_nodes(plan->n_leaves, plan->n_seg, plan->n_msgs, plan->manifest);
    const PlanMem P = plan_mem(plan->device, plan->n_msgs, plan->n_leaves, rows, scratch, D);
    if (P.bytes > plan->bytes) return fail(HV_ERR_INVALID_ARG, "plan is corrupt (layout exceeds its memory)");

    hv_status st;
    hipError_t e;
    if (plan->n_leaves > 0) {
        if ((st = leaf_timing_start(stream)) != HV_OK) return st;
        e = plan->alg == HV_SHA384
                ? hv::launch_sha384_auto(P.hash.desc, plan->n_leaves, plan->n_leaves, leaf_digests, stream)
                : hv::launch_sha256_auto(P.hash.desc, plan->n_leaves, plan->n_leaves, leaf_digests, stream);
        if (e != hipSuccess) return hip_fail(e, "leaf kernel");
        if ((st = leaf_timing_stop(stream)) != HV_OK) return st;
    }
    // the first tree has n_leaves entries (per-message segments, or one), the manifest one per message
    if (plan->n_seg > 0 &&
        (st = queue_merkle(plan->alg, leaf_digests, roots, P.table[0], plan->n_seg, plan->n_leaves,
                           (int)plan->launches[0], plan->tiles[0], P.ping, P.pong, stream)) != HV_OK)
        return st;
    const uint8_t* top = roots;
    if (plan->manifest) {
        if ((st = queue_merkle(plan->alg, roots, root, P.table[1], 1, plan->n_msgs, (int)plan->launches[1],
                               plan->tiles[1], P.ping, P.pong, stream)) != HV_OK)
            return st;
        top = root;
    }
    if (expected != nullptr && (e = hv::launch_verify_root_dev(top, expected, D, match, stream)) != hipSuccess)
        return hip_fail(e, "verify kernel");
    return HV_OK;
}

size_t hv_verify_model_workspace_bytes(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                       int manifest) {
    Prep p;
    if (prepare(alg, msgs, n_msgs, chunk_bytes, manifest != 0, &p) != HV_OK) return 0;
    const uint32_t D = digest_size(alg);
    const size_t plan_bytes = plan_mem(nullptr, n_msgs, p.n_leaves, p.rows, p.scratch, D).bytes;
    return model_layout(nullptr, plan_bytes, p.n_leaves, p.n_seg, D).bytes;
}

hv_status hv_verify_model(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, int manifest,
                          const uint8_t* expected, void* workspace, size_t workspace_bytes, hv_result* result,
                          hipStream_t stream) {
    const auto t0 = std::chrono::steady_clock::now();
    if (result == nullptr) return fail(HV_ERR_INVALID_ARG, "result is NULL");
    manifest = manifest != 0;
    Prep p;
    hv_status st = prepare(alg, msgs, n_msgs, chunk_bytes, manifest, &p);
    if (st != HV_OK) return st;
    const uint32_t D = digest_size(alg);
    const size_t plan_bytes = plan_mem(nullptr, n_msgs, p.n_leaves, p.rows, p.scratch, D).bytes;
    const ModelLayout need = model_layout(nullptr, plan_bytes, p.n_leaves, p.n_seg, D);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu%s", need.bytes, workspace_bytes,
                    workspace ? "" : " (NULL)");
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    const ModelLayout M = model_layout(workspace, plan_bytes, p.n_leaves, p.n_seg, D);
    hv_verify_plan plan;
    if ((st = hv_plan_init(alg, msgs, n_msgs, chunk_bytes, manifest, M.plan, plan_bytes, &plan, stream)) != HV_OK)
        return st;
    hipError_t e;
    if (expected != nullptr &&
        (e = hipMemcpyAsync(M.expected, expected, D, hipMemcpyHostToDevice, stream)) != hipSuccess)
        return hip_fail(e, "expected root upload");
    if ((st = hv_plan_run(&plan, M.leaves, M.roots, M.root, expected ? M.expected : nullptr,
                          expected ? M.match : nullptr, stream)) != HV_OK)
        return st;
    uint8_t root[48];
    uint32_t match = 0;
    const uint8_t* top = manifest ? M.root : M.roots;
    if ((e = hipMemcpyAsync(root, top, D, hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return hip_fail(e, "root copy");
    if (expected != nullptr && (e = hipMemcpyAsync(&match, M.match, sizeof match, hipMemcpyDeviceToHost, stream)) !=
                                   hipSuccess)
        return hip_fail(e, "verdict copy");
    if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e, "stream synchronize");
    *result = hv_result{};
    result->integrity_verified = expected != nullptr && match == 1 ? 1 : 0;
    result->root_bytes = D;
    std::memcpy(result->root, root, D);
    result->verification_time_ns = (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                                       std::chrono::steady_clock::now() - t0)
                                       .count();
    return HV_OK;
}

}  // extern "C"
