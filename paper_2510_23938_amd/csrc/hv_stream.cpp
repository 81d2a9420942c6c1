// hv_stream.cpp -- chunk digests of host-resident messages, streamed through
// GPU memory: Algorithm 1's loop (load a model chunk into GPU memory, hash it,
// keep its digest, free the memory) for weights that do not fit in, or do not
// live in, HBM.
//
// Whole chunks are grouped into batches of at most batch_bytes, in leaf order,
// so each batch covers a contiguous range of leaf numbers.  A batch is a list
// of pieces: a run of whole chunks of one message (ending with the message's
// tail chunk when the run reaches the message end), copied to a 256-byte
// aligned offset of one of two device staging buffers.  Copies go on
// copy_stream, hashing on hash_stream: the scheduler and the leaf kernel of
// the resident path run on each batch's pieces, so chunk i of a piece is chunk
// (start / C + i) of its message and every digest equals the resident path's.
// Events order the reuse of a staging buffer after its batch is hashed, so
// the copy of batch b+1 overlaps the hashing of batch b.  All descriptors are
// planned on the host and uploaded once before the loop.
#include <stdio.h>

#include <vector>

#include "hv.h"
#include "hv_host.h"
#include "hv_stream.h"

using namespace hvh;

namespace {

struct Piece {
    uint32_t msg;
    uint64_t src_off;    // byte offset in the message (a multiple of C when C > 0)
    uint64_t len;
    uint64_t stage_off;  // byte offset in the staging buffer (256-byte aligned)
};

struct Batch {
    size_t p0, p1;        // pieces [p0, p1)
    uint64_t first_leaf;  // leaf number of the batch's first chunk
    uint64_t n_leaves, n_full;
};

struct Plan {
    std::vector<Piece> pieces;
    std::vector<Batch> batches;
    uint64_t n_leaves = 0;
    uint32_t max_pieces = 0;
    uint64_t max_leaves = 0;
};

uint64_t leaves_of(uint64_t len, uint64_t C) { return C == 0 ? 1 : len / C + (len % C != 0); }

hv_status make_plan(const hv_msg* msgs, uint32_t n_msgs, uint64_t C, uint64_t batch_bytes, Plan* P) {
    uint64_t n_leaves = 0;
    hv_status st = layout(msgs, n_msgs, C, nullptr, &n_leaves, nullptr);
    if (st != HV_OK) return st;
    if (batch_bytes < kAlign || batch_bytes % kAlign != 0)
        return fail(HV_ERR_INVALID_ARG, "batch_bytes = %llu is not a positive multiple of 256",
                    (unsigned long long)batch_bytes);
    for (uint32_t m = 0; m < n_msgs; ++m) {
        const uint64_t L = msgs[m].nbytes;
        const uint64_t longest = C == 0 || L < C ? L : C;
        if (longest > batch_bytes)
            return fail(HV_ERR_INVALID_ARG, "message %u: a %llu-byte chunk does not fit a %llu-byte batch", m,
                        (unsigned long long)longest, (unsigned long long)batch_bytes);
    }
    P->n_leaves = n_leaves;
    Batch cur = {0, 0, 0, 0, 0};
    uint64_t used = 0;  // staging bytes of the current batch, pieces at 256-byte aligned offsets
    auto close = [&]() {
        cur.p1 = P->pieces.size();
        if (cur.p1 > cur.p0) {
            P->batches.push_back(cur);
            P->max_pieces = std::max<uint32_t>(P->max_pieces, (uint32_t)(cur.p1 - cur.p0));
            P->max_leaves = std::max(P->max_leaves, cur.n_leaves);
        }
        const uint64_t next_leaf = cur.first_leaf + cur.n_leaves;
        cur = {P->pieces.size(), 0, next_leaf, 0, 0};
        used = 0;
    };
    for (uint32_t m = 0; m < n_msgs; ++m) {
        const uint64_t L = msgs[m].nbytes;
        if (C != 0 && L == 0) continue;  // no chunks, no leaves
        uint64_t pos = 0;
        do {
            const uint64_t at = round_up(used);
            const uint64_t space = at < batch_bytes ? batch_bytes - at : 0;
            const uint64_t rest = L - pos;
            uint64_t take;
            if (rest <= space) take = rest;                    // the rest of the message, tail included
            else if (C != 0) take = space / C * C;             // whole chunks only
            else take = 0;                                     // a whole message must fit
            if (take == 0 && !(rest == 0 && C == 0)) {         // nothing fits: next batch
                if (used == 0) return fail(HV_ERR_INVALID_ARG, "message %u does not fit a batch", m);
                close();
                continue;
            }
            P->pieces.push_back({m, pos, take, at});
            cur.n_leaves += leaves_of(take, C);
            cur.n_full += C == 0 ? 0 : take / C;
            used = at + take;
            pos += take;
        } while (pos < L);
    }
    close();
    return HV_OK;
}

struct StreamLayout {
    uint8_t* stage[2];
    hv::MsgDesc* descs;
    HashLayout hash;
    size_t bytes;
};

StreamLayout stream_layout(void* ws, const Plan& P, uint64_t batch_bytes) {
    Carver c(ws);
    StreamLayout L;
    L.stage[0] = c.take<uint8_t>(batch_bytes);
    L.stage[1] = c.take<uint8_t>(batch_bytes);
    L.descs = c.take<hv::MsgDesc>(P.pieces.size());
    const size_t before = c.used;
    L.hash = hash_layout(ws ? static_cast<uint8_t*>(ws) + before : nullptr, P.max_pieces, P.max_leaves);
    L.bytes = before + L.hash.bytes;
    return L;
}

}  // namespace

extern "C" {

size_t hv_stream_workspace_bytes(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint64_t batch_bytes) {
    Plan P;
    if (make_plan(msgs, n_msgs, chunk_bytes, batch_bytes, &P) != HV_OK) return 0;
    return stream_layout(nullptr, P, batch_bytes).bytes;
}

hv_status hv_hash_host_chunks_alg(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                  uint8_t* leaf_digests, uint64_t batch_bytes, void* workspace, size_t workspace_bytes,
                                  hipStream_t copy_stream, hipStream_t hash_stream) {
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (alg == HV_SHA384 && chunk_bytes % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)chunk_bytes);
    const uint64_t D = alg == HV_SHA384 ? 48 : 32;
    Plan P;
    hv_status st = make_plan(msgs, n_msgs, chunk_bytes, batch_bytes, &P);
    if (st != HV_OK) return st;
    if (P.n_leaves > kMaxLeaves) return fail(HV_ERR_INVALID_ARG, "too many leaves");
    if (P.n_leaves > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if ((uintptr_t)leaf_digests % 16 != 0) return fail(HV_ERR_INVALID_ARG, "leaf_digests is not 16-byte aligned");
    const StreamLayout need = stream_layout(nullptr, P, batch_bytes);
    if (workspace == nullptr || workspace_bytes < need.bytes)
        return fail(HV_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu%s", need.bytes, workspace_bytes,
                    workspace ? "" : " (NULL)");
    if ((uintptr_t)workspace % kAlign != 0) return fail(HV_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    if (P.batches.empty()) return HV_OK;

    const StreamLayout L = stream_layout(workspace, P, batch_bytes);
    // descriptors of every piece, pointing into the staging buffer its batch uses
    std::vector<hv::MsgDesc> descs(P.pieces.size());
    for (size_t b = 0; b < P.batches.size(); ++b)
        for (size_t i = P.batches[b].p0; i < P.batches[b].p1; ++i)
            descs[i] = {(uint64_t)(uintptr_t)(L.stage[b % 2] + P.pieces[i].stage_off), P.pieces[i].len};
    hipError_t e = hipMemcpyWithStream(L.descs, descs.data(), descs.size() * sizeof(hv::MsgDesc),
                                       hipMemcpyHostToDevice, hash_stream);
    if (e != hipSuccess) return hip_fail(e, "descriptor upload");

    hipEvent_t copied[2] = {nullptr, nullptr}, hashed[2] = {nullptr, nullptr};
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
        e = hipEventCreateWithFlags(&copied[i], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&hashed[i], hipEventDisableTiming);
    }
    st = e == hipSuccess ? HV_OK : hip_fail(e, "event create");
    // copies start only after the work the caller queued on hash_stream before
    // this call (which may still be writing the host bytes, e.g. a device-to-host copy)
    if (st == HV_OK && ((e = hipEventRecord(hashed[1], hash_stream)) != hipSuccess ||
                        (e = hipStreamWaitEvent(copy_stream, hashed[1], 0)) != hipSuccess))
        st = hip_fail(e, "stream ordering");
    for (size_t b = 0; b < P.batches.size() && st == HV_OK; ++b) {
        const Batch& B = P.batches[b];
        const int buf = (int)(b % 2);
        if (b >= 2 && (e = hipStreamWaitEvent(copy_stream, hashed[buf], 0)) != hipSuccess) {
            st = hip_fail(e, "stream wait");
            break;
        }
        for (size_t i = B.p0; i < B.p1 && e == hipSuccess; ++i) {
            const Piece& pc = P.pieces[i];
            if (pc.len == 0) continue;
            const uint8_t* src = static_cast<const uint8_t*>(msgs[pc.msg].data) + pc.src_off;
            e = hipMemcpyAsync(L.stage[buf] + pc.stage_off, src, pc.len, hipMemcpyHostToDevice, copy_stream);
        }
        if (e == hipSuccess) e = hipEventRecord(copied[buf], copy_stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(hash_stream, copied[buf], 0);
        if (e != hipSuccess) {
            st = hip_fail(e, "batch copy");
            break;
        }
        st = queue_schedule(L.descs + B.p0, (uint32_t)(B.p1 - B.p0), chunk_bytes, B.n_full, B.n_leaves, L.hash,
                            hash_stream);
        if (st != HV_OK) break;
        uint8_t* out = leaf_digests + D * B.first_leaf;
        e = alg == HV_SHA384 ? hv::launch_sha384_auto(L.hash.desc, B.n_leaves, B.n_leaves, out, hash_stream)
                             : hv::launch_sha256_auto(L.hash.desc, B.n_leaves, B.n_leaves, out, hash_stream);
        if (e != hipSuccess || (e = hipEventRecord(hashed[buf], hash_stream)) != hipSuccess)
            st = hip_fail(e, "leaf kernel");
    }
    // every copy was waited on by hash_stream, so this also drains copy_stream's work
    e = hipStreamSynchronize(hash_stream);
    if (st == HV_OK && e != hipSuccess) st = hip_fail(e, "stream synchronize");
    if ((e = hipStreamSynchronize(copy_stream)) != hipSuccess && st == HV_OK) st = hip_fail(e, "stream synchronize");
    for (int i = 0; i < 2; ++i) {
        if (copied[i]) (void)hipEventDestroy(copied[i]);
        if (hashed[i]) (void)hipEventDestroy(hashed[i]);
    }
    return st;
}

hv_status hv_hash_host_chunks(const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes, uint8_t* leaf_digests,
                              uint64_t batch_bytes, void* workspace, size_t workspace_bytes, hipStream_t copy_stream,
                              hipStream_t hash_stream) {
    return hv_hash_host_chunks_alg(HV_SHA256, msgs, n_msgs, chunk_bytes, leaf_digests, batch_bytes, workspace,
                                   workspace_bytes, copy_stream, hash_stream);
}

}  // extern "C"
