// hv_incr.cpp -- incremental re-verification (include/hv_incremental.h): a
// persistent per-segment Merkle tree on the device, updated along the paths of
// the leaves whose chunks changed, and rehashing of a listed set of chunks.
#include <vector>

#include "hv.h"
#include "hv_host.h"
#include "hv_incremental.h"

using namespace hvh;

namespace {

// Level offsets of the persistent tree: row j has n_seg + 1 entries, row 0 is
// seg_offsets; a segment with c nodes at level j has ceil(c / 2) at level j+1.
// Rows are added until every segment has at most one node.
bool tree_rows(const uint64_t* seg_offsets, uint32_t n_seg, std::vector<uint64_t>* rows, uint32_t* levels) {
    const size_t w = (size_t)n_seg + 1;
    rows->assign(seg_offsets, seg_offsets + w);
    uint32_t j = 0;
    for (;;) {
        const uint64_t* prev = rows->data() + (size_t)j * w;
        bool more = false;
        for (uint32_t s = 0; s < n_seg; ++s)
            if (prev[s + 1] - prev[s] > 1) more = true;
        if (!more) break;
        std::vector<uint64_t> next(w, 0);
        for (uint32_t s = 0; s < n_seg; ++s) next[s + 1] = next[s] + (prev[s + 1] - prev[s] + 1) / 2;
        rows->insert(rows->end(), next.begin(), next.end());
        ++j;
        if (j > 64) return false;
    }
    *levels = j;  // rows 0..j
    return true;
}

struct TreeLayout {
    uint64_t* table;               // device copy of the rows
    std::vector<uint8_t*> level;   // level j node array
    size_t bytes;
};

hv_status check_offsets(const uint64_t* seg_offsets, uint32_t n_seg) {
    if (n_seg == 0) return fail(HV_ERR_INVALID_ARG, "n_seg is 0");
    if (seg_offsets == nullptr) return fail(HV_ERR_INVALID_ARG, "seg_offsets is NULL");
    if (seg_offsets[0] != 0) return fail(HV_ERR_INVALID_ARG, "seg_offsets[0] is not 0");
    for (uint32_t s = 0; s < n_seg; ++s)
        if (seg_offsets[s + 1] < seg_offsets[s]) return fail(HV_ERR_INVALID_ARG, "seg_offsets decreases at %u", s);
    if (seg_offsets[n_seg] > kMaxLeaves) return fail(HV_ERR_INVALID_ARG, "too many entries");
    return HV_OK;
}

TreeLayout tree_layout(void* tree, const std::vector<uint64_t>& rows, uint32_t n_seg, uint32_t levels, uint32_t D) {
    Carver c(tree);
    TreeLayout T;
    T.table = c.take<uint64_t>(rows.size());
    const size_t w = (size_t)n_seg + 1;
    for (uint32_t j = 0; j <= levels; ++j) T.level.push_back(c.take<uint8_t>(rows[j * w + n_seg] * D));
    T.bytes = c.used;
    return T;
}

// Strictly increasing leaf numbers below n.
hv_status check_list(const uint64_t* list, uint32_t k, uint64_t n, const char* what) {
    if (k > 0 && list == nullptr) return fail(HV_ERR_INVALID_ARG, "%s is NULL", what);
    for (uint32_t i = 0; i < k; ++i) {
        if (list[i] >= n) return fail(HV_ERR_INVALID_ARG, "%s[%u] = %llu is not below %llu", what, i,
                                      (unsigned long long)list[i], (unsigned long long)n);
        if (i > 0 && list[i] <= list[i - 1]) return fail(HV_ERR_INVALID_ARG, "%s is not strictly increasing", what);
    }
    return HV_OK;
}

struct UpdateLayout {
    uint64_t* dirty;
    uint32_t* seg_of;
    uint64_t* local;
    size_t bytes;
};

UpdateLayout update_layout(void* ws, uint32_t k) {
    Carver c(ws);
    UpdateLayout U;
    U.dirty = c.take<uint64_t>(k);
    U.seg_of = c.take<uint32_t>(k);
    U.local = c.take<uint64_t>(k);
    U.bytes = c.used;
    return U;
}

struct RehashLayout {
    uint64_t* list;
    HashLayout hash;
    size_t bytes;
};

RehashLayout rehash_layout(void* ws, uint32_t n_msgs, uint32_t k) {
    Carver c(ws);
    RehashLayout R;
    R.list = c.take<uint64_t>(k);
    const size_t before = c.used;
    R.hash = hash_layout(ws ? static_cast<uint8_t*>(ws) + before : nullptr, n_msgs, k);
    R.bytes = before + R.hash.bytes;
    return R;
}

bool known(hv_alg alg) { return alg == HV_SHA256 || alg == HV_SHA384; }
uint32_t digest_size(hv_alg alg) { return alg == HV_SHA384 ? 48 : 32; }
int kernel_alg(hv_alg alg) { return alg == HV_SHA384 ? hv::kAlgSha384 : hv::kAlgSha256; }

}  // namespace

extern "C" {

size_t hv_tree_bytes_alg(hv_alg alg, const uint64_t* seg_offsets, uint32_t n_seg) {
    if (!known(alg)) {
        (void)fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
        return 0;
    }
    if (check_offsets(seg_offsets, n_seg) != HV_OK) return 0;
    std::vector<uint64_t> rows;
    uint32_t levels = 0;
    if (!tree_rows(seg_offsets, n_seg, &rows, &levels)) return 0;
    return tree_layout(nullptr, rows, n_seg, levels, digest_size(alg)).bytes;
}

size_t hv_tree_bytes(const uint64_t* seg_offsets, uint32_t n_seg) {
    return hv_tree_bytes_alg(HV_SHA256, seg_offsets, n_seg);
}

hv_status hv_tree_build_alg(hv_alg alg, const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg,
                            void* tree, size_t tree_bytes, uint8_t* roots, hipStream_t stream) {
    if (!known(alg)) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    const uint32_t D = digest_size(alg);
    const int ka = kernel_alg(alg);
    hv_status st = check_offsets(seg_offsets, n_seg);
    if (st != HV_OK) return st;
    const uint64_t n = seg_offsets[n_seg];
    if (n > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if (roots == nullptr) return fail(HV_ERR_INVALID_ARG, "roots is NULL");
    if ((uintptr_t)leaf_digests % 16 || (uintptr_t)roots % 16)
        return fail(HV_ERR_INVALID_ARG, "leaf_digests and roots must be 16-byte aligned");
    std::vector<uint64_t> rows;
    uint32_t levels = 0;
    if (!tree_rows(seg_offsets, n_seg, &rows, &levels)) return fail(HV_ERR_INVALID_ARG, "tree too deep");
    const TreeLayout need = tree_layout(nullptr, rows, n_seg, levels, D);
    if (tree == nullptr || tree_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "tree needs %zu bytes, got %zu", need.bytes, tree_bytes);
    if ((uintptr_t)tree % kAlign != 0) return fail(HV_ERR_WORKSPACE, "tree is not 256-byte aligned");
    const TreeLayout T = tree_layout(tree, rows, n_seg, levels, D);
    const size_t w = (size_t)n_seg + 1;
    hipError_t e =
        hipMemcpyWithStream(T.table, rows.data(), rows.size() * sizeof(uint64_t), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "table upload");
    if ((e = hv::launch_tree_leaf_level(ka, leaf_digests, n, T.level[0], stream)) != hipSuccess)
        return hip_fail(e, "leaf level");
    for (uint32_t j = 0; j < levels; ++j)
        if ((e = hv::launch_tree_build_level(ka, T.level[j], T.level[j + 1], T.table + j * w, T.table + (j + 1) * w,
                                             n_seg, rows[(j + 1) * w + n_seg], stream)) != hipSuccess)
            return hip_fail(e, "tree level");
    if ((e = hv::launch_tree_roots(ka, T.level[levels], T.table + levels * w, n_seg, roots, stream)) != hipSuccess)
        return hip_fail(e, "roots");
    return HV_OK;
}

hv_status hv_tree_build(const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg, void* tree,
                        size_t tree_bytes, uint8_t* roots, hipStream_t stream) {
    return hv_tree_build_alg(HV_SHA256, leaf_digests, seg_offsets, n_seg, tree, tree_bytes, roots, stream);
}

size_t hv_tree_update_workspace_bytes(uint32_t n_dirty) { return update_layout(nullptr, n_dirty).bytes; }

hv_status hv_tree_update_alg(hv_alg alg, const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg,
                             void* tree, size_t tree_bytes, const uint64_t* dirty, uint32_t n_dirty, uint8_t* roots,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!known(alg)) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    const uint32_t D = digest_size(alg);
    const int ka = kernel_alg(alg);
    hv_status st = check_offsets(seg_offsets, n_seg);
    if (st != HV_OK) return st;
    const uint64_t n = seg_offsets[n_seg];
    if ((st = check_list(dirty, n_dirty, n, "dirty")) != HV_OK) return st;
    if (n > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if (roots == nullptr) return fail(HV_ERR_INVALID_ARG, "roots is NULL");
    if ((uintptr_t)leaf_digests % 16 || (uintptr_t)roots % 16)
        return fail(HV_ERR_INVALID_ARG, "leaf_digests and roots must be 16-byte aligned");
    std::vector<uint64_t> rows;
    uint32_t levels = 0;
    if (!tree_rows(seg_offsets, n_seg, &rows, &levels)) return fail(HV_ERR_INVALID_ARG, "tree too deep");
    const TreeLayout need = tree_layout(nullptr, rows, n_seg, levels, D);
    if (tree == nullptr || tree_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "tree needs %zu bytes, got %zu", need.bytes, tree_bytes);
    if ((uintptr_t)tree % kAlign != 0) return fail(HV_ERR_WORKSPACE, "tree is not 256-byte aligned");
    const UpdateLayout uneed = update_layout(nullptr, n_dirty);
    if (workspace == nullptr || workspace_bytes < uneed.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", uneed.bytes, workspace_bytes);
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    const TreeLayout T = tree_layout(tree, rows, n_seg, levels, D);
    const size_t w = (size_t)n_seg + 1;
    // the offset table is re-sent so the kernels walk exactly the layout planned here
    hipError_t e =
        hipMemcpyWithStream(T.table, rows.data(), rows.size() * sizeof(uint64_t), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "table upload");
    if (n_dirty > 0) {
        const UpdateLayout U = update_layout(workspace, n_dirty);
        if ((e = hipMemcpyWithStream(U.dirty, dirty, n_dirty * sizeof(uint64_t), hipMemcpyHostToDevice, stream)) !=
            hipSuccess)
            return hip_fail(e, "dirty list upload");
        if ((e = hv::launch_tree_locate(U.dirty, n_dirty, T.table, n_seg, U.seg_of, U.local, stream)) != hipSuccess)
            return hip_fail(e, "locate");
        if ((e = hv::launch_tree_update_leaves(ka, leaf_digests, U.dirty, n_dirty, T.level[0], stream)) != hipSuccess)
            return hip_fail(e, "leaf update");
        for (uint32_t j = 0; j < levels; ++j)
            if ((e = hv::launch_tree_update_level(ka, T.level[j], T.level[j + 1], T.table + j * w,
                                                  T.table + (j + 1) * w, U.seg_of, U.local, n_dirty, j + 1, stream)) !=
                hipSuccess)
                return hip_fail(e, "path update");
    }
    if ((e = hv::launch_tree_roots(ka, T.level[levels], T.table + levels * w, n_seg, roots, stream)) != hipSuccess)
        return hip_fail(e, "roots");
    return HV_OK;
}

hv_status hv_tree_update(const uint8_t* leaf_digests, const uint64_t* seg_offsets, uint32_t n_seg, void* tree,
                         size_t tree_bytes, const uint64_t* dirty, uint32_t n_dirty, uint8_t* roots, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
    return hv_tree_update_alg(HV_SHA256, leaf_digests, seg_offsets, n_seg, tree, tree_bytes, dirty, n_dirty, roots,
                              workspace, workspace_bytes, stream);
}

size_t hv_rehash_workspace_bytes(uint32_t n_msgs, uint32_t n_listed) {
    return rehash_layout(nullptr, n_msgs, n_listed).bytes;
}

hv_status hv_rehash_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                               const uint64_t* leaves, uint32_t n_listed, uint8_t* leaf_digests, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
    if (!known(alg)) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (alg == HV_SHA384 && chunk_bytes % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)chunk_bytes);
    uint64_t n_leaves = 0, n_full = 0;
    hv_status st = layout(msgs, n_msgs, chunk_bytes, nullptr, &n_leaves, &n_full);
    if (st != HV_OK) return st;
    if ((st = check_list(leaves, n_listed, n_leaves, "leaves")) != HV_OK) return st;
    if (n_listed > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if ((uintptr_t)leaf_digests % 16 != 0) return fail(HV_ERR_INVALID_ARG, "leaf_digests is not 16-byte aligned");
    const RehashLayout need = rehash_layout(nullptr, n_msgs, n_listed);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need.bytes, workspace_bytes);
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (n_listed == 0) return HV_OK;
    const RehashLayout R = rehash_layout(workspace, n_msgs, n_listed);
    const HashLayout& L = R.hash;
    hipError_t e = hipMemcpyWithStream(L.msgs, msgs, sizeof(hv_msg) * n_msgs, hipMemcpyHostToDevice, stream);
    if (e == hipSuccess)
        e = hipMemcpyWithStream(R.list, leaves, n_listed * sizeof(uint64_t), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(e, "upload");
    if ((e = hv::launch_sched_count(L.msgs, n_msgs, chunk_bytes, L.cnt, stream)) != hipSuccess)
        return hip_fail(e, "count kernel");
    if ((e = hv::launch_scan_pairs(L.cnt, L.off, n_msgs, L.partials, stream)) != hipSuccess)
        return hip_fail(e, "scan kernels");
    if ((e = hv::launch_sched_select(L.msgs, L.off, n_msgs, chunk_bytes, R.list, n_listed, L.desc, stream)) !=
        hipSuccess)
        return hip_fail(e, "select kernel");
    e = alg == HV_SHA384 ? hv::launch_sha384_auto(L.desc, n_listed, n_leaves, leaf_digests, stream)
                         : hv::launch_sha256_auto(L.desc, n_listed, n_leaves, leaf_digests, stream);
    if (e != hipSuccess) return hip_fail(e, "leaf kernel");
    return HV_OK;
}

hv_status hv_rehash_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, const uint64_t* leaves,
                           uint32_t n_listed, uint8_t* leaf_digests, void* workspace, size_t workspace_bytes,
                           hipStream_t stream) {
    return hv_rehash_chunks_alg(HV_SHA256, msgs, n_msgs, chunk_bytes, leaves, n_listed, leaf_digests, workspace,
                                workspace_bytes, stream);
}

}  // extern "C"
