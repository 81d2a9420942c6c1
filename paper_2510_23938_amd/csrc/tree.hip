// tree.hip -- a persistent Merkle tree on the device, for incremental
// re-verification after a model update (the paper's fine-tuning / partial
// update case: only changed chunks are rehashed, only the tree nodes above
// them are recomputed).
//
// The tree of every segment is kept level by level with RFC 6962's bottom-up
// shape (section 2.1): level 0 holds the leaf nodes SHA-256(0x00 || d); level
// j+1 pairs neighbours (2i, 2i+1) of level j into SHA-256(0x01 || L || R) and
// moves an unpaired last node up unchanged.  A segment with c nodes at level j
// has ceil(c / 2) at level j+1, so after enough levels every non-empty segment
// has exactly one node: its root.  Level arrays hold all segments back to
// back; the offset table off[j][s] gives segment s's first node at level j.
#include "hv_kernels.h"
#include "sha256_device.h"

namespace hv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void leaf_node(const uint32_t d[8], uint32_t out[8]) {
    uint32_t W[16];
    W[0] = d[0] >> 8;
#pragma unroll
    for (int i = 1; i < 8; ++i) W[i] = (d[i - 1] << 24) | (d[i] >> 8);
    W[8] = (d[7] << 24) | 0x00800000u;
#pragma unroll
    for (int i = 9; i < 15; ++i) W[i] = 0;
    W[15] = 33 * 8;
    init_state(out);
    compress(out, W);
}

__device__ __forceinline__ void inner_node(const uint32_t L[8], const uint32_t R[8], uint32_t out[8]) {
    uint32_t W[16];
    W[0] = 0x01000000u | (L[0] >> 8);
#pragma unroll
    for (int i = 1; i < 8; ++i) W[i] = (L[i - 1] << 24) | (L[i] >> 8);
    W[8] = (L[7] << 24) | (R[0] >> 8);
#pragma unroll
    for (int i = 1; i < 8; ++i) W[8 + i] = (R[i - 1] << 24) | (R[i] >> 8);
    init_state(out);
    compress(out, W);
    W[0] = (R[7] << 24) | 0x00800000u;
#pragma unroll
    for (int i = 1; i < 15; ++i) W[i] = 0;
    W[15] = 65 * 8;
    compress(out, W);
}

__device__ __forceinline__ uint32_t owner(const uint64_t* __restrict__ off, uint32_t n_seg, uint64_t g) {
    uint32_t lo = 0, hi = n_seg;  // largest s with off[s] <= g (off[n_seg] > g)
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (off[mid] <= g) lo = mid; else hi = mid;
    }
    return lo;
}

// Parent i of segment s at level j+1 from its children at level j.
__device__ __forceinline__ void make_parent(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                            const uint64_t* __restrict__ in_off, const uint64_t* __restrict__ out_off,
                                            uint32_t s, uint64_t i) {
    const uint64_t c = in_off[s + 1] - in_off[s];
    uint32_t L[8], P[8];
    load_digest(in + 32 * (in_off[s] + 2 * i), L);
    if (2 * i + 1 < c) {
        uint32_t R[8];
        load_digest(in + 32 * (in_off[s] + 2 * i + 1), R);
        inner_node(L, R, P);
    } else {
#pragma unroll
        for (int w = 0; w < 8; ++w) P[w] = L[w];
    }
    store_digest(out + 32 * (out_off[s] + i), P);
}

__global__ void __launch_bounds__(kThreads) leaf_level_kernel(const uint8_t* __restrict__ digests, uint64_t n,
                                                              uint8_t* __restrict__ level0) {
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < n; g += (uint64_t)gridDim.x * kThreads) {
        uint32_t D[8], P[8];
        load_digest(digests + 32 * g, D);
        leaf_node(D, P);
        store_digest(level0 + 32 * g, P);
    }
}

__global__ void __launch_bounds__(kThreads) build_level_kernel(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                                               const uint64_t* __restrict__ in_off,
                                                               const uint64_t* __restrict__ out_off, uint32_t n_seg,
                                                               uint64_t n_out) {
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < n_out; g += (uint64_t)gridDim.x * kThreads) {
        const uint32_t s = owner(out_off, n_seg, g);
        make_parent(in, out, in_off, out_off, s, g - out_off[s]);
    }
}

// Dirty leaves (sorted, unique, global leaf numbers) -> segment and local index.
__global__ void __launch_bounds__(kThreads) locate_kernel(const uint64_t* __restrict__ dirty, uint32_t k,
                                                          const uint64_t* __restrict__ seg_off, uint32_t n_seg,
                                                          uint32_t* __restrict__ seg_of, uint64_t* __restrict__ local) {
    for (uint32_t e = blockIdx.x * kThreads + threadIdx.x; e < k; e += gridDim.x * kThreads) {
        const uint32_t s = owner(seg_off, n_seg, dirty[e]);
        seg_of[e] = s;
        local[e] = dirty[e] - seg_off[s];
    }
}

__global__ void __launch_bounds__(kThreads) update_leaves_kernel(const uint8_t* __restrict__ digests,
                                                                 const uint64_t* __restrict__ dirty, uint32_t k,
                                                                 uint8_t* __restrict__ level0) {
    for (uint32_t e = blockIdx.x * kThreads + threadIdx.x; e < k; e += gridDim.x * kThreads) {
        uint32_t D[8], P[8];
        load_digest(digests + 32 * dirty[e], D);
        leaf_node(D, P);
        store_digest(level0 + 32 * dirty[e], P);
    }
}

// Level j -> j+1 along the dirty paths: entry e's node at level j+1 is
// local[e] >> (j+1); the first entry of each run of equal (segment, node)
// recomputes it, the others return (their leaves share the parent).
__global__ void __launch_bounds__(kThreads) update_level_kernel(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                                                const uint64_t* __restrict__ in_off,
                                                                const uint64_t* __restrict__ out_off,
                                                                const uint32_t* __restrict__ seg_of,
                                                                const uint64_t* __restrict__ local, uint32_t k,
                                                                uint32_t shift) {
    for (uint32_t e = blockIdx.x * kThreads + threadIdx.x; e < k; e += gridDim.x * kThreads) {
        const uint32_t s = seg_of[e];
        const uint64_t p = local[e] >> shift;
        if (e > 0 && seg_of[e - 1] == s && (local[e - 1] >> shift) == p) continue;
        make_parent(in, out, in_off, out_off, s, p);
    }
}

// roots[s] = the top-level node of segment s, or SHA-256("") when it is empty.
__global__ void __launch_bounds__(kThreads) roots_kernel(const uint8_t* __restrict__ top, const uint64_t* __restrict__ top_off,
                                                         uint32_t n_seg, uint8_t* __restrict__ roots) {
    for (uint32_t s = blockIdx.x * kThreads + threadIdx.x; s < n_seg; s += gridDim.x * kThreads) {
        uint32_t R[8];
        if (top_off[s + 1] > top_off[s]) {
            load_digest(top + 32 * top_off[s], R);
        } else {
            uint32_t W[16];
            W[0] = 0x80000000u;
#pragma unroll
            for (int i = 1; i < 16; ++i) W[i] = 0;
            init_state(R);
            compress(R, W);
        }
        store_digest(roots + 32 * (uint64_t)s, R);
    }
}

unsigned grid_for(uint64_t n) {
    const uint64_t blocks = (n + kThreads - 1) / kThreads;
    return (unsigned)(blocks == 0 ? 1 : (blocks < 65536 ? blocks : 65536));
}

}  // namespace

hipError_t launch_tree_leaf_level(const uint8_t* digests, uint64_t n, uint8_t* level0, hipStream_t s) {
    if (n == 0) return hipSuccess;
    leaf_level_kernel<<<grid_for(n), kThreads, 0, s>>>(digests, n, level0);
    return hipGetLastError();
}

hipError_t launch_tree_build_level(const uint8_t* in, uint8_t* out, const uint64_t* in_off, const uint64_t* out_off,
                                   uint32_t n_seg, uint64_t n_out, hipStream_t s) {
    if (n_out == 0) return hipSuccess;
    build_level_kernel<<<grid_for(n_out), kThreads, 0, s>>>(in, out, in_off, out_off, n_seg, n_out);
    return hipGetLastError();
}

hipError_t launch_tree_locate(const uint64_t* dirty, uint32_t k, const uint64_t* seg_off, uint32_t n_seg,
                              uint32_t* seg_of, uint64_t* local, hipStream_t s) {
    if (k == 0) return hipSuccess;
    locate_kernel<<<grid_for(k), kThreads, 0, s>>>(dirty, k, seg_off, n_seg, seg_of, local);
    return hipGetLastError();
}

hipError_t launch_tree_update_leaves(const uint8_t* digests, const uint64_t* dirty, uint32_t k, uint8_t* level0,
                                     hipStream_t s) {
    if (k == 0) return hipSuccess;
    update_leaves_kernel<<<grid_for(k), kThreads, 0, s>>>(digests, dirty, k, level0);
    return hipGetLastError();
}

hipError_t launch_tree_update_level(const uint8_t* in, uint8_t* out, const uint64_t* in_off, const uint64_t* out_off,
                                    const uint32_t* seg_of, const uint64_t* local, uint32_t k, uint32_t shift,
                                    hipStream_t s) {
    if (k == 0) return hipSuccess;
    update_level_kernel<<<grid_for(k), kThreads, 0, s>>>(in, out, in_off, out_off, seg_of, local, k, shift);
    return hipGetLastError();
}

hipError_t launch_tree_roots(const uint8_t* top, const uint64_t* top_off, uint32_t n_seg, uint8_t* roots,
                             hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    roots_kernel<<<grid_for(n_seg), kThreads, 0, s>>>(top, top_off, n_seg, roots);
    return hipGetLastError();
}

}  // namespace hv
