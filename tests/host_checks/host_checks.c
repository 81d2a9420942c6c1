/* host_checks.c -- the library's host-side logic, run under AddressSanitizer
 * and UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py: leaf
 * layout, workspace and plan sizing, Merkle launch planning, persistent-tree
 * planning, stream batch planning, over many seeded random message sets, and
 * the argument checks each entry point makes before it queues any work.
 *
 * No call here reaches the GPU.  Each is host-only or is rejected by the
 * library's own checks before any HIP call, so the "device" addresses below
 * are never dereferenced by anyone.  Exit status 0 and the last line
 * "host checks passed" mean every check held and no sanitizer fired. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "hv.h"
#include "hv_incremental.h"
#include "hv_inspect.h"
#include "hv_monitor.h"
#include "hv_plan.h"
#include "hv_stream.h"

static int failures = 0;

#define CHECK(cond)                                                                                 \
    do {                                                                                            \
        if (!(cond)) {                                                                              \
            fprintf(stderr, "check failed, line %d: %s [%s]\n", __LINE__, #cond, hv_last_error()); \
            ++failures;                                                                             \
        }                                                                                           \
    } while (0)

/* A rejection must say why. */
#define REJECTED(expr, status) CHECK((expr) == (status) && hv_last_error()[0] != '\0')

static uint64_t rng = 0x243F6A8885A308D3ull;
static uint64_t next(void) { /* splitmix64 */
    uint64_t z = (rng += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Addresses that stand for device memory: only compared and stored. */
#define DEV(off) ((void*)(uintptr_t)(0x7f0000000000ull + (uint64_t)(off)))

static uint64_t leaves_of(uint64_t len, uint64_t C) { return C == 0 ? 1 : len / C + (len % C != 0); }

/* n messages with lengths clustered around block and chunk multiples. */
static void random_set(hv_msg* m, uint32_t n, uint64_t C, uint64_t max_len) {
    uint64_t at = 0;
    for (uint32_t i = 0; i < n; ++i) {
        const uint64_t unit = C ? C : 4096, r = next() % 4;
        uint64_t len = r == 0 ? next() % 200 : r == 1 ? (next() % 8) * unit + next() % 3 : r == 2 ? next() % max_len : 0;
        if (len > max_len) len = max_len;
        m[i].data = len ? DEV(at) : NULL;
        m[i].nbytes = len;
        at += (len + 255) / 256 * 256 + 256;
    }
}

static void layouts_and_sizes(void) {
    static hv_msg m[400];
    static uint64_t seg[401];
    for (int t = 0; t < 3000; ++t) {
        const uint32_t n = (uint32_t)(next() % 400);
        const uint64_t C = (next() % 5) == 0 ? 0 : 128ull << (next() % 11); /* 0 or 128 .. 128 KiB */
        random_set(m, n, C, 1u << 20);
        uint64_t n_leaves = 0, want = 0;
        CHECK(hv_leaf_layout(m, n, C, seg, &n_leaves) == HV_OK);
        CHECK(seg[0] == 0);
        for (uint32_t i = 0; i < n; ++i) {
            const uint64_t k = m[i].nbytes == 0 && C ? 0 : leaves_of(m[i].nbytes, C);
            CHECK(seg[i + 1] - seg[i] == k);
            want += k;
        }
        CHECK(n_leaves == want && seg[n] == want);
        CHECK(hv_hash_workspace_bytes(n, n_leaves) > 0);
        CHECK(hv_merkle_workspace_bytes(n_leaves, n ? n : 1) > 0);
        for (int alg = 0; alg < 2; ++alg) {
            const int manifest = (int)(next() % 2);
            const size_t p = hv_plan_bytes((hv_alg)alg, m, n, C, manifest);
            CHECK(p > 0);
            CHECK(hv_verify_model_workspace_bytes((hv_alg)alg, m, n, C, manifest) > p);
            if (n > 0) CHECK(hv_tree_bytes_alg((hv_alg)alg, seg, n) > 0);
            CHECK((hv_monitor_scan_workspace_bytes((hv_alg)alg, n_leaves) > 0) == (n_leaves > 0));
        }
        CHECK(hv_monitor_plan_bytes(n) > 0);
        CHECK(hv_rehash_workspace_bytes(n, (uint32_t)(n_leaves < 100000 ? n_leaves : 100000)) > 0);
        const uint32_t k = (uint32_t)(next() % 1000);
        CHECK((hv_tree_update_workspace_bytes(k) > 0) == (k > 0));
    }
}

/* Tables of 2^16 messages or more are validated on several host threads:
 * the same offsets as the per-message rule, and the lowest refused message. */
static void large_layouts(void) {
    enum { N = 150000 };
    static hv_msg m[N];
    static uint64_t seg[N + 1];
    for (int t = 0; t < 6; ++t) {
        const uint64_t C = t % 3 == 0 ? 0 : 4096ull << (t % 3);
        random_set(m, N, C, 1u << 18);
        uint64_t n_leaves = 0, want = 0;
        CHECK(hv_leaf_layout(m, N, C, seg, &n_leaves) == HV_OK);
        CHECK(seg[0] == 0);
        for (uint32_t i = 0; i < N; ++i) {
            want += m[i].nbytes == 0 && C ? 0 : leaves_of(m[i].nbytes, C);
            CHECK(seg[i + 1] == want);
        }
        CHECK(n_leaves == want);
        CHECK(hv_leaf_layout(m, N, C, NULL, &n_leaves) == HV_OK && n_leaves == want);
        /* two refused messages: the lower one is reported */
        const uint32_t a = (uint32_t)(next() % N), b = (uint32_t)(next() % N);
        const hv_msg ka = m[a], kb = m[b];
        m[a].data = NULL;
        m[a].nbytes = 1;
        m[b].data = NULL;
        m[b].nbytes = 1;
        REJECTED(hv_leaf_layout(m, N, C, seg, &n_leaves), HV_ERR_INVALID_ARG);
        char want_msg[64];
        snprintf(want_msg, sizeof want_msg, "message %u has NULL data", a < b ? a : b);
        CHECK(strstr(hv_last_error(), want_msg) != NULL);
        m[a] = ka;
        m[b] = kb;
    }
}

static void stream_plans(void) {
    static hv_msg m[64];
    for (int t = 0; t < 500; ++t) {
        const uint32_t n = (uint32_t)(next() % 64);
        const uint64_t C = (next() % 4) == 0 ? 0 : 64ull << (next() % 10);
        random_set(m, n, C, 300000);
        uint64_t longest = 0; /* longest chunk */
        for (uint32_t i = 0; i < n; ++i) {
            const uint64_t c = C && m[i].nbytes > C ? C : m[i].nbytes;
            longest = c > longest ? c : longest;
        }
        const uint64_t unit = C ? C : (longest ? longest : 256);
        const uint64_t batch = ((unit * (1 + next() % 5) + next() % 4096) + 255) / 256 * 256;
        CHECK(hv_stream_workspace_bytes(m, n, C, batch) > 0);
        const uint64_t small = longest / 256 * 256; /* a batch one step short of the longest chunk */
        if (longest > 256 && small < longest)
            REJECTED(hv_stream_workspace_bytes(m, n, C, small) == 0 ? HV_ERR_INVALID_ARG : HV_OK, HV_ERR_INVALID_ARG);
        else if (longest > 256)
            REJECTED(hv_stream_workspace_bytes(m, n, C, small - 256) == 0 ? HV_ERR_INVALID_ARG : HV_OK,
                     HV_ERR_INVALID_ARG);
    }
}

static void tree_sizes(void) {
    static uint64_t seg[300];
    for (int t = 0; t < 2000; ++t) {
        const uint32_t n = 1 + (uint32_t)(next() % 299);
        seg[0] = 0;
        for (uint32_t s = 0; s < n; ++s) seg[s + 1] = seg[s] + ((next() % 3) == 0 ? 0 : next() % 70000);
        CHECK(hv_tree_bytes(seg, n) > 0);
        CHECK(hv_tree_bytes_alg(HV_SHA384, seg, n) > hv_tree_bytes(seg, n) || seg[n] == 0);
        if (n > 1 && seg[n] > 0) {
            const uint64_t keep = seg[1];
            seg[1] = seg[n] + 1; /* offsets that decrease */
            CHECK(hv_tree_bytes(seg, n) == 0);
            seg[1] = keep;
        }
    }
    CHECK(hv_tree_bytes(seg, 0) == 0);
    CHECK(hv_tree_bytes_alg((hv_alg)7, seg, 1) == 0);
}

static void rejections(void) {
    hv_msg m[3] = {{DEV(0), 5000}, {DEV(8192), 70000}, {NULL, 0}};
    hv_msg bad_null[1] = {{NULL, 10}};
    hv_msg wraps[1] = {{(void*)(uintptr_t)0xFFFFFFFFFFFFFFF0ull, 0x20}};
    uint64_t seg[4], n_leaves = 0;
    uint8_t expected[48] = {0};
    int match = 0;
    const size_t ws_need = hv_hash_workspace_bytes(3, 20);

    REJECTED(hv_leaf_layout(NULL, 3, 4096, seg, &n_leaves), HV_ERR_INVALID_ARG);
    REJECTED(hv_leaf_layout(m, 3, 100, seg, &n_leaves), HV_ERR_INVALID_ARG);
    REJECTED(hv_leaf_layout(m, 3, 4096, seg, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_leaf_layout(bad_null, 1, 4096, seg, &n_leaves), HV_ERR_INVALID_ARG);
    REJECTED(hv_leaf_layout(wraps, 1, 4096, seg, &n_leaves), HV_ERR_INVALID_ARG);

    REJECTED(hv_hash_chunks(NULL, 3, 4096, DEV(0), DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_chunks(m, 3, 100, DEV(0), DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_chunks(m, 3, 4096, NULL, DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_chunks(m, 3, 4096, DEV(1), DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_chunks(m, 3, 4096, DEV(0), NULL, ws_need, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_hash_chunks(m, 3, 4096, DEV(0), DEV(0), 16, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_hash_chunks(m, 3, 4096, DEV(0), DEV(8), ws_need, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_hash_chunks_alg(HV_SHA384, m, 3, 64, DEV(0), DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_chunks_alg((hv_alg)9, m, 3, 4096, DEV(0), DEV(0), ws_need, NULL), HV_ERR_INVALID_ARG);

    const uint64_t ok_seg[3] = {0, 5, 9}, bad0[3] = {1, 5, 9}, down[3] = {0, 5, 4};
    const size_t mws = hv_merkle_workspace_bytes(9, 2);
    REJECTED(hv_merkle_reduce(DEV(0), ok_seg, 0, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(DEV(0), NULL, 2, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(DEV(0), bad0, 2, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(DEV(0), down, 2, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(NULL, ok_seg, 2, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(DEV(0), ok_seg, 2, DEV(4), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_merkle_reduce(DEV(0), ok_seg, 2, DEV(0), DEV(0), 8, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_merkle_reduce_alg((hv_alg)3, DEV(0), ok_seg, 2, DEV(0), DEV(0), mws, NULL), HV_ERR_INVALID_ARG);

    REJECTED(hv_verify_root(NULL, expected, &match, DEV(0), hv_verify_workspace_bytes(), NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_verify_root(DEV(0), NULL, &match, DEV(0), hv_verify_workspace_bytes(), NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_verify_root(DEV(0), expected, NULL, DEV(0), hv_verify_workspace_bytes(), NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_verify_root(DEV(0), expected, &match, NULL, hv_verify_workspace_bytes(), NULL), HV_ERR_WORKSPACE);

    hv_verify_plan plan;
    memset(&plan, 0, sizeof plan);
    const size_t pb = hv_plan_bytes(HV_SHA256, m, 3, 4096, 1);
    CHECK(pb > 0);
    REJECTED(hv_plan_init(HV_SHA256, m, 3, 4096, 1, DEV(0), pb, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_init(HV_SHA256, m, 3, 4096, 1, DEV(0), pb - 1, &plan, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_plan_init(HV_SHA256, m, 3, 4096, 1, DEV(16), pb, &plan, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_plan_run(NULL, DEV(0), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG); /* not initialised */
    plan.device = DEV(0);
    plan.bytes = 256;
    plan.alg = (hv_alg)5;
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    plan.alg = HV_SHA256;
    plan.launches[0] = 1000;
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    plan.launches[0] = 2;
    plan.n_leaves = 20;
    plan.n_seg = 3;
    plan.n_msgs = 3;
    plan.manifest = 1;
    REJECTED(hv_plan_run(&plan, NULL, DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), NULL, DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), NULL, NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(8), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), DEV(0), NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), DEV(0), DEV(2), NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_plan_run(&plan, DEV(0), DEV(0), DEV(0), NULL, NULL, NULL), HV_ERR_INVALID_ARG); /* layout > bytes */

    hv_result res;
    REJECTED(hv_verify_model(HV_SHA256, m, 3, 4096, 1, NULL, DEV(0), 1u << 30, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_verify_model(HV_SHA256, m, 3, 4096, 1, NULL, DEV(0), 16, &res, NULL), HV_ERR_WORKSPACE);

    const uint64_t unsorted[2] = {5, 3}, beyond[1] = {1000};
    const size_t tb = hv_tree_bytes(ok_seg, 2);
    REJECTED(hv_tree_update(DEV(0), ok_seg, 2, DEV(0), tb, unsorted, 2, DEV(0), DEV(0),
                            hv_tree_update_workspace_bytes(2), NULL),
             HV_ERR_INVALID_ARG);
    REJECTED(hv_tree_update(DEV(0), ok_seg, 2, DEV(0), tb, beyond, 1, DEV(0), DEV(0),
                            hv_tree_update_workspace_bytes(1), NULL),
             HV_ERR_INVALID_ARG);
    REJECTED(hv_tree_build(DEV(0), ok_seg, 2, DEV(0), tb - 1, DEV(0), NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_rehash_chunks(m, 3, 4096, unsorted, 2, DEV(0), DEV(0), hv_rehash_workspace_bytes(3, 2), NULL),
             HV_ERR_INVALID_ARG);
    REJECTED(hv_rehash_chunks(m, 3, 4096, beyond, 1, DEV(0), DEV(0), hv_rehash_workspace_bytes(3, 1), NULL),
             HV_ERR_INVALID_ARG);

    hv_monitor_plan mp;
    memset(&mp, 0, sizeof mp);
    uint64_t result[2];
    REJECTED(hv_monitor_init(HV_SHA256, m, 3, 4096, DEV(0), hv_monitor_plan_bytes(3), NULL, NULL),
             HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_init((hv_alg)4, m, 3, 4096, DEV(0), hv_monitor_plan_bytes(3), &mp, NULL),
             HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_init(HV_SHA256, m, 3, 4096, DEV(0), 8, &mp, NULL), HV_ERR_WORKSPACE);
    REJECTED(hv_monitor_scan(NULL, 0, 1, DEV(0), NULL, result, DEV(0), 1u << 20, NULL), HV_ERR_INVALID_ARG);
    mp.device = DEV(0);
    mp.alg = HV_SHA256;
    mp.n_msgs = 3;
    mp.chunk_bytes = 4096;
    mp.n_leaves = 20;
    REJECTED(hv_monitor_scan(&mp, 15, 6, DEV(0), NULL, result, DEV(0), 1u << 20, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_scan(&mp, 21, 0, DEV(0), NULL, result, DEV(0), 1u << 20, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_scan(&mp, 0, 1, DEV(0), NULL, NULL, DEV(0), 1u << 20, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_scan(&mp, 0, 1, NULL, NULL, result, DEV(0), 1u << 20, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_monitor_scan(&mp, 0, 1, DEV(0), NULL, result, DEV(0), 8, NULL), HV_ERR_WORKSPACE);

    REJECTED(hv_hash_host_chunks(m, 3, 4096, DEV(0), 1000, DEV(0), 1u << 30, NULL, NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_hash_host_chunks(m, 3, 4096, DEV(0), 2048, DEV(0), 1u << 30, NULL, NULL), HV_ERR_INVALID_ARG);

    REJECTED(hv_set_leaf_kernel(-1), HV_ERR_INVALID_ARG);
    REJECTED(hv_set_leaf_kernel(4), HV_ERR_INVALID_ARG);
    CHECK(hv_set_leaf_kernel(0) == HV_OK);
    float ms = 0;
    REJECTED(hv_leaf_kernel_ms(NULL), HV_ERR_INVALID_ARG);
    REJECTED(hv_leaf_kernel_ms(&ms), HV_ERR_INVALID_ARG); /* nothing was timed on this thread */
    uint32_t mask[8] = {0};
    hipStream_t s = NULL;
    REJECTED(hv_stream_create_cu_masked(NULL, 8, &s), HV_ERR_INVALID_ARG);
    REJECTED(hv_stream_create_cu_masked(mask, 0, &s), HV_ERR_INVALID_ARG);
    REJECTED(hv_stream_destroy(NULL), HV_ERR_INVALID_ARG);
}

/* Merkle launch plans over random segment sets and compute-unit counts: the
 * launches end with one node per segment, and every group launch's one-lane
 * part is all of it or whole rounds of 256 groups per compute unit (and then
 * less than one round remains). */
static void merkle_plans(void) {
    enum { MAXSEG = 300 };
    static uint64_t seg[MAXSEG + 1];
    for (int it = 0; it < 3000; ++it) {
        const uint32_t n_seg = 1 + (uint32_t)(next() % MAXSEG);
        const uint64_t scale = (uint64_t)1 << (next() % 23);
        seg[0] = 0;
        for (uint32_t i = 0; i < n_seg; ++i) seg[i + 1] = seg[i] + (next() % 5 == 0 ? 0 : next() % (2 * scale + 1));
        const uint32_t cus = 1 + (uint32_t)(next() % 512);
        int launches = 0, kind[8];
        uint64_t units[8], one[8];
        const hv_alg alg = (next() & 1) ? HV_SHA384 : HV_SHA256;
        if (hv_merkle_launches(alg, seg, n_seg, cus, &launches, kind, units, one) != HV_OK) {
            CHECK(seg[n_seg] > ((uint64_t)1 << 31)); /* only the entry limit may refuse a valid set */
            continue;
        }
        CHECK(launches >= 1 && launches <= 8);
        CHECK(units[launches - 1] == n_seg);
        const uint64_t R = 256 * (uint64_t)cus;
        for (int k = 0; k < launches; ++k) {
            CHECK(kind[k] == 1 || kind[k] == 2);
            CHECK(units[k] >= n_seg);
            if (kind[k] == 1) CHECK(one[k] == units[k] || (one[k] % R == 0 && one[k] > 0 && units[k] - one[k] < R));
            else CHECK(one[k] == 0);
        }
    }
    /* no device is asked for when cus > 0; cus = 0 without one fails cleanly */
    const uint64_t two[3] = {0, 5, 9};
    int launches = 0, kind[8];
    uint64_t units[8], one[8];
    const hv_status st = hv_merkle_launches(HV_SHA256, two, 2, 0, &launches, kind, units, one);
    CHECK(st == HV_OK || st == HV_ERR_HIP);
}

int main(void) {
    layouts_and_sizes();
    merkle_plans();
    large_layouts();
    stream_plans();
    tree_sizes();
    rejections();
    if (failures) {
        fprintf(stderr, "%d host checks failed\n", failures);
        return 1;
    }
    printf("host checks passed\n");
    return 0;
}
