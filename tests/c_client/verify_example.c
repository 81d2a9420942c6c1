/*
 * verify_example.c -- a C client of libhv with no Python and no torch: device
 * buffers from hipMalloc, the one-shot calls of hv.h (chunk digests ->
 * per-message roots -> manifest root -> on-GPU comparison) and the one-call
 * hv_verify_model of hv_plan.h, for SHA-256 and SHA-384.
 *
 *   verify_example <chunk_bytes> <len0> [len1 ...]
 *
 * Message m holds bytes (i * 131 + 7 * m + 1) mod 256 for i < len_m.  Prints
 * one line per hash: "<hash> <manifest root hex> <verdict of hv_verify_model>".
 * Exit status 0 when every call succeeded and both forms agree.
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "hv.h"
#include "hv_plan.h"

static int fail_hv(const char* what, hv_status st) {
    fprintf(stderr, "%s: status %d: %s\n", what, (int)st, hv_last_error());
    return 1;
}

static int fail_hip(const char* what, hipError_t e) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 1;
}

static void print_hex(const uint8_t* p, uint32_t n) {
    for (uint32_t i = 0; i < n; ++i) printf("%02x", p[i]);
}

int main(int argc, char** argv) {
    if (argc < 3) {
        fprintf(stderr, "usage: %s chunk_bytes len0 [len1 ...]\n", argv[0]);
        return 2;
    }
    const uint64_t C = strtoull(argv[1], NULL, 10);
    const uint32_t n = (uint32_t)(argc - 2);
    hv_msg* msgs = calloc(n, sizeof *msgs);
    void** bufs = calloc(n, sizeof *bufs);
    if (!msgs || !bufs) return 1;
    hipError_t e;
    for (uint32_t m = 0; m < n; ++m) {
        const uint64_t len = strtoull(argv[2 + m], NULL, 10);
        uint8_t* host = malloc(len ? len : 1);
        if (!host) return 1;
        for (uint64_t i = 0; i < len; ++i) host[i] = (uint8_t)(i * 131 + 7 * m + 1);
        if ((e = hipMalloc(&bufs[m], len ? len : 1)) != hipSuccess) return fail_hip("hipMalloc", e);
        if (len && (e = hipMemcpy(bufs[m], host, len, hipMemcpyHostToDevice)) != hipSuccess)
            return fail_hip("hipMemcpy", e);
        free(host);
        msgs[m].data = len ? bufs[m] : NULL;
        msgs[m].nbytes = len;
    }
    hipStream_t stream;
    if ((e = hipStreamCreate(&stream)) != hipSuccess) return fail_hip("hipStreamCreate", e);

    int rc = 0;
    const hv_alg algs[2] = {HV_SHA256, HV_SHA384};
    for (int k = 0; k < 2 && rc == 0; ++k) {
        const hv_alg alg = algs[k];
        const uint32_t D = alg == HV_SHA384 ? 48 : 32;
        uint64_t* seg = calloc((size_t)n + 1, sizeof *seg);
        uint64_t n_leaves = 0;
        hv_status st = hv_leaf_layout(msgs, n, C, seg, &n_leaves);
        if (st != HV_OK) return fail_hv("hv_leaf_layout", st);
        /* device outputs and workspaces, sized by the library */
        uint8_t *leaves = NULL, *roots = NULL, *root = NULL;
        void *ws_hash = NULL, *ws_tree = NULL, *ws_top = NULL, *ws_verify = NULL, *ws_model = NULL;
        const size_t b_hash = hv_hash_workspace_bytes(n, n_leaves);
        const size_t b_tree = hv_merkle_workspace_bytes_alg(alg, n_leaves, n);
        const size_t b_top = hv_merkle_workspace_bytes_alg(alg, n, 1);
        const size_t b_model = hv_verify_model_workspace_bytes(alg, msgs, n, C, 1);
        if ((e = hipMalloc((void**)&leaves, n_leaves ? n_leaves * D : 16)) != hipSuccess ||
            (e = hipMalloc((void**)&roots, (size_t)n * D)) != hipSuccess ||
            (e = hipMalloc((void**)&root, D)) != hipSuccess || (e = hipMalloc(&ws_hash, b_hash)) != hipSuccess ||
            (e = hipMalloc(&ws_tree, b_tree)) != hipSuccess || (e = hipMalloc(&ws_top, b_top)) != hipSuccess ||
            (e = hipMalloc(&ws_verify, hv_verify_workspace_bytes())) != hipSuccess ||
            (e = hipMalloc(&ws_model, b_model)) != hipSuccess)
            return fail_hip("hipMalloc", e);
        const uint64_t top_seg[2] = {0, n};
        if ((st = hv_hash_chunks_alg(alg, msgs, n, C, n_leaves ? leaves : NULL, ws_hash, b_hash, stream)) != HV_OK)
            return fail_hv("hv_hash_chunks_alg", st);
        if ((st = hv_merkle_reduce_alg(alg, leaves, seg, n, roots, ws_tree, b_tree, stream)) != HV_OK)
            return fail_hv("hv_merkle_reduce_alg (messages)", st);
        if ((st = hv_merkle_reduce_alg(alg, roots, top_seg, 1, root, ws_top, b_top, stream)) != HV_OK)
            return fail_hv("hv_merkle_reduce_alg (manifest)", st);
        uint8_t host_root[48];
        if ((e = hipMemcpyAsync(host_root, root, D, hipMemcpyDeviceToHost, stream)) != hipSuccess ||
            (e = hipStreamSynchronize(stream)) != hipSuccess)
            return fail_hip("root copy", e);
        int match = -1;
        if ((st = hv_verify_root_alg(alg, root, host_root, &match, ws_verify, hv_verify_workspace_bytes(),
                                     stream)) != HV_OK)
            return fail_hv("hv_verify_root_alg", st);
        hv_result res;
        if ((st = hv_verify_model(alg, msgs, n, C, 1, host_root, ws_model, b_model, &res, stream)) != HV_OK)
            return fail_hv("hv_verify_model", st);
        printf("%s ", alg == HV_SHA384 ? "sha384" : "sha256");
        print_hex(host_root, D);
        printf(" %d\n", res.integrity_verified);
        if (match != 1 || !res.integrity_verified || res.root_bytes != D || memcmp(res.root, host_root, D) != 0)
            rc = 3;
        (void)hipFree(leaves); (void)hipFree(roots); (void)hipFree(root); (void)hipFree(ws_hash);
        (void)hipFree(ws_tree); (void)hipFree(ws_top); (void)hipFree(ws_verify); (void)hipFree(ws_model);
        free(seg);
    }
    for (uint32_t m = 0; m < n; ++m) (void)hipFree(bufs[m]);
    (void)hipStreamDestroy(stream);
    free(msgs);
    free(bufs);
    return rc;
}
