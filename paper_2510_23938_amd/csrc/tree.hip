// tree.hip -- a persistent Merkle tree on the device, for incremental
// re-verification after a model update (the paper's fine-tuning / partial
// update case: only changed chunks are rehashed, only the tree nodes above
// them are recomputed).
//
// The tree of every segment is kept level by level with RFC 6962's bottom-up
// shape (section 2.1): level 0 holds the leaf nodes H(0x00 || d); level j+1
// pairs neighbours (2i, 2i+1) of level j into H(0x01 || L || R) and moves an
// unpaired last node up unchanged.  A segment with c nodes at level j has
// ceil(c / 2) at level j+1, so after enough levels every non-empty segment
// has exactly one node: its root.  Level arrays hold all segments back to
// back; the offset table off[j][s] gives segment s's first node at level j.
// Every kernel is written once over the node-hash policy (SHA-256 or
// SHA-384 nodes, tree_hash.h).
#include "hv_kernels.h"
#include "tree_hash.h"

namespace hv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t owner(const uint64_t* __restrict__ off, uint32_t n_seg, uint64_t g) {
    uint32_t lo = 0, hi = n_seg;  // largest s with off[s] <= g (off[n_seg] > g)
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (off[mid] <= g) lo = mid; else hi = mid;
    }
    return lo;
}

// Parent i of segment s at level j+1 from its children at level j.
template <class T>
__device__ __forceinline__ void make_parent(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                            const uint64_t* __restrict__ in_off, const uint64_t* __restrict__ out_off,
                                            uint32_t s, uint64_t i) {
    constexpr int NW = T::kWords, NB = T::kBytes;
    const uint64_t c = in_off[s + 1] - in_off[s];
    uint32_t L[NW], P[NW];
    T::load(in + NB * (in_off[s] + 2 * i), L);
    if (2 * i + 1 < c) {
        uint32_t R[NW];
        T::load(in + NB * (in_off[s] + 2 * i + 1), R);
        T::node_hash(L, R, P);
    } else {
#pragma unroll
        for (int w = 0; w < NW; ++w) P[w] = L[w];
    }
    T::store(out + NB * (out_off[s] + i), P);
}

template <class T>
__global__ void __launch_bounds__(kThreads) leaf_level_kernel(const uint8_t* __restrict__ digests, uint64_t n,
                                                              uint8_t* __restrict__ level0) {
    constexpr int NW = T::kWords, NB = T::kBytes;
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < n; g += (uint64_t)gridDim.x * kThreads) {
        uint32_t D[NW], P[NW];
        T::load(digests + NB * g, D);
        T::leaf_hash(D, P);
        T::store(level0 + NB * g, P);
    }
}

template <class T>
__global__ void __launch_bounds__(kThreads) build_level_kernel(const uint8_t* __restrict__ in, uint8_t* __restrict__ out,
                                                               const uint64_t* __restrict__ in_off,
                                                               const uint64_t* __restrict__ out_off, uint32_t n_seg,
                                                               uint64_t n_out) {
    for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < n_out; g += (uint64_t)gridDim.x * kThreads) {
        const uint32_t s = owner(out_off, n_seg, g);
        make_parent<T>(in, out, in_off, out_off, s, g - out_off[s]);
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

template <class T>
__global__ void __launch_bounds__(kThreads) update_leaves_kernel(const uint8_t* __restrict__ digests,
                                                                 const uint64_t* __restrict__ dirty, uint32_t k,
                                                                 uint8_t* __restrict__ level0) {
    constexpr int NW = T::kWords, NB = T::kBytes;
    for (uint32_t e = blockIdx.x * kThreads + threadIdx.x; e < k; e += gridDim.x * kThreads) {
        uint32_t D[NW], P[NW];
        T::load(digests + NB * dirty[e], D);
        T::leaf_hash(D, P);
        T::store(level0 + NB * dirty[e], P);
    }
}

// Level j -> j+1 along the dirty paths: entry e's node at level j+1 is
// local[e] >> (j+1); the first entry of each run of equal (segment, node)
// recomputes it, the others return (their leaves share the parent).
template <class T>
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
        make_parent<T>(in, out, in_off, out_off, s, p);
    }
}

// roots[s] = the top-level node of segment s, or H("") when it is empty.
template <class T>
__global__ void __launch_bounds__(kThreads) roots_kernel(const uint8_t* __restrict__ top, const uint64_t* __restrict__ top_off,
                                                         uint32_t n_seg, uint8_t* __restrict__ roots) {
    constexpr int NW = T::kWords, NB = T::kBytes;
    for (uint32_t s = blockIdx.x * kThreads + threadIdx.x; s < n_seg; s += gridDim.x * kThreads) {
        uint32_t R[NW];
        if (top_off[s + 1] > top_off[s])
            T::load(top + NB * top_off[s], R);
        else
            T::empty_hash(R);
        T::store(roots + NB * (uint64_t)s, R);
    }
}

unsigned grid_for(uint64_t n) {
    const uint64_t blocks = (n + kThreads - 1) / kThreads;
    return (unsigned)(blocks == 0 ? 1 : (blocks < 65536 ? blocks : 65536));
}

}  // namespace

hipError_t launch_tree_leaf_level(int alg, const uint8_t* digests, uint64_t n, uint8_t* level0, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if (alg == kAlgSha384)
        leaf_level_kernel<Sha384Tree><<<grid_for(n), kThreads, 0, s>>>(digests, n, level0);
    else
        leaf_level_kernel<Sha256Tree><<<grid_for(n), kThreads, 0, s>>>(digests, n, level0);
    return hipGetLastError();
}

hipError_t launch_tree_build_level(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                   const uint64_t* out_off, uint32_t n_seg, uint64_t n_out, hipStream_t s) {
    if (n_out == 0) return hipSuccess;
    if (alg == kAlgSha384)
        build_level_kernel<Sha384Tree><<<grid_for(n_out), kThreads, 0, s>>>(in, out, in_off, out_off, n_seg, n_out);
    else
        build_level_kernel<Sha256Tree><<<grid_for(n_out), kThreads, 0, s>>>(in, out, in_off, out_off, n_seg, n_out);
    return hipGetLastError();
}

hipError_t launch_tree_locate(const uint64_t* dirty, uint32_t k, const uint64_t* seg_off, uint32_t n_seg,
                              uint32_t* seg_of, uint64_t* local, hipStream_t s) {
    if (k == 0) return hipSuccess;
    locate_kernel<<<grid_for(k), kThreads, 0, s>>>(dirty, k, seg_off, n_seg, seg_of, local);
    return hipGetLastError();
}

hipError_t launch_tree_update_leaves(int alg, const uint8_t* digests, const uint64_t* dirty, uint32_t k,
                                     uint8_t* level0, hipStream_t s) {
    if (k == 0) return hipSuccess;
    if (alg == kAlgSha384)
        update_leaves_kernel<Sha384Tree><<<grid_for(k), kThreads, 0, s>>>(digests, dirty, k, level0);
    else
        update_leaves_kernel<Sha256Tree><<<grid_for(k), kThreads, 0, s>>>(digests, dirty, k, level0);
    return hipGetLastError();
}

hipError_t launch_tree_update_level(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                    const uint64_t* out_off, const uint32_t* seg_of, const uint64_t* local, uint32_t k,
                                    uint32_t shift, hipStream_t s) {
    if (k == 0) return hipSuccess;
    if (alg == kAlgSha384)
        update_level_kernel<Sha384Tree><<<grid_for(k), kThreads, 0, s>>>(in, out, in_off, out_off, seg_of, local, k,
                                                                          shift);
    else
        update_level_kernel<Sha256Tree><<<grid_for(k), kThreads, 0, s>>>(in, out, in_off, out_off, seg_of, local, k,
                                                                          shift);
    return hipGetLastError();
}

hipError_t launch_tree_roots(int alg, const uint8_t* top, const uint64_t* top_off, uint32_t n_seg, uint8_t* roots,
                             hipStream_t s) {
    if (n_seg == 0) return hipSuccess;
    if (alg == kAlgSha384)
        roots_kernel<Sha384Tree><<<grid_for(n_seg), kThreads, 0, s>>>(top, top_off, n_seg, roots);
    else
        roots_kernel<Sha256Tree><<<grid_for(n_seg), kThreads, 0, s>>>(top, top_off, n_seg, roots);
    return hipGetLastError();
}

}  // namespace hv
