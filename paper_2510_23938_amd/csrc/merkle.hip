// merkle.hip -- segmented RFC 6962 Merkle Tree Hash, bottom-up, on the GPU
// (Algorithm 1's "construct Merkle tree from leaf_hashes using GPU").
//
// RFC 6962 section 2.1 defines MTH recursively, splitting n entries at the
// largest power of two below n.  Built bottom-up that is: level 0 holds the
// leaf hashes SHA-256(0x00 || d_i); each level pairs neighbours (2i, 2i+1)
// into SHA-256(0x01 || left || right) and moves an unpaired last node up
// unchanged.  (Node i of level j then covers entries [i*2^j, min((i+1)*2^j, n)),
// so the root's two children split exactly where the recursion splits.)
//
// A workgroup reduces a tile of up to 512 = 2^9 consecutive nodes of one
// segment by nine levels, to one node.  Tiles start at multiples of 512, so no
// pair ever straddles two tiles, and the tile's last unpaired node at any level
// is the segment's last node there -- the same promotion the whole tree
// makes.  One launch therefore takes every segment nine levels up; the host
// chains such launches until one node per segment is left, and the first
// launch of a reduction also forms the leaf hashes as it loads the entries.
// Level 1 is formed in registers from the two entries a thread loads.  Levels
// of more than 64 nodes go through LDS, with idle waves waiting at the
// barriers; the last six levels of a full tile (64 nodes down to one) stay in
// wave 0 and exchange children by cross-lane shuffles.  A wave with any node
// to form hashes on all its lanes and keeps the needed results by selects:
// the top levels are a chain of one wave's block latencies, and a wave with
// few active lanes runs each block markedly slower (the per-tensor tops of
// the 70B-shaped set: 57 us against 70).
//
// Levels of at least 2^18 entries run as group launches instead (below): one
// lane per aligned group of 8 entries, three levels in registers, so that the
// widest levels keep every lane busy; the tile launches then start from the
// group nodes.  The tile kernel alone leaves lanes idle on its top levels and
// costs more for the same nodes: on the 70B-shaped set (2.15 M leaves in 723
// segments, two group launches) the per-tensor reduction takes about 30% less.
//
// The kernels are written once over a node-hash policy: SHA-256 (32-byte nodes;
// an interior node is two blocks) or SHA-384 (48-byte nodes; leaf and
// interior nodes are one 128-byte block each).
#include "hv_kernels.h"
#include "tree_hash.h"

namespace hv {
namespace {

constexpr int kThreads = kTileNodes / 2;  // 256: each thread owns one pair of level 0
constexpr uint32_t kWave = 64;             // lanes of a wave

__device__ __forceinline__ uint32_t find_segment(const uint64_t* __restrict__ tile_off, uint32_t n_seg, uint64_t tile) {
    uint32_t lo = 0, hi = n_seg;  // tile_off[lo] <= tile < tile_off[hi]
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (tile_off[mid] <= tile) lo = mid; else hi = mid;
    }
    return lo;
}

// Four tiles per CU where LDS allows (SHA-384 nodes); with SHA-256 the
// node-tail table (33 KB) beside the 8 KB of level exchange leaves room for three.
template <class T>
__global__ void __launch_bounds__(kThreads, T::kTableWords > 4 ? 3 : 4)
    merkle_tile_kernel(const uint8_t* __restrict__ in, uint8_t* __restrict__ out, const uint64_t* __restrict__ in_off,
                       const uint64_t* __restrict__ tile_off, uint32_t n_seg, uint64_t n_tiles, int leaf_mode) {
    constexpr int NW = T::kWords;
    constexpr int NB = T::kBytes;
    constexpr uint32_t Nodes = kTileNodes;
    __shared__ uint32_t lds[NW][kThreads];  // word-major: node i's word w at lds[w][i]
    __shared__ __align__(16) uint32_t tab[T::kTableWords];
    const uint32_t i = threadIdx.x;
    T::stage_table(tab);
    __syncthreads();
    for (uint64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
        const uint32_t s = find_segment(tile_off, n_seg, tile);
        const uint64_t t = tile - tile_off[s];
        const uint64_t c = in_off[s + 1] - in_off[s];
        const uint64_t first = t * Nodes;
        const uint32_t cnt = c > first ? (uint32_t)(c - first < (uint64_t)Nodes ? c - first : Nodes) : 0u;
        const uint8_t* base = in + NB * (in_off[s] + first);

        uint32_t P[NW] = {};  // lanes without a node feed zeros to the shuffles
        uint32_t n = 1;  // nodes of the current level (after the first)
        if (cnt == 0) {  // empty segment (only ever a first-launch tile)
            if (i == 0) T::empty_hash(P);
        } else if ((i & ~(kWave - 1)) * 2 < cnt) {
            // A wave that holds any node of level 1 hashes on every lane (a
            // wave with few active lanes runs each block slower; it issues the
            // same instructions either way): lanes past the tile's end take
            // its last entry, and selects keep what the lane's own entries
            // give -- a pair's node, an unpaired last node moved up, or none.
            const bool hasA = 2 * i < cnt, hasB = 2 * i + 1 < cnt;
            const uint32_t ea = hasA ? 2 * i : cnt - 1, eb = hasB ? 2 * i + 1 : cnt - 1;
            uint32_t A[NW], B[NW], Z[NW];
            T::load(base + NB * ea, A);
            T::load(base + NB * eb, B);
            if (leaf_mode) {
                uint32_t X[NW];
                T::leaf_hash(A, X);
                for (int w = 0; w < NW; ++w) A[w] = X[w];
                T::leaf_hash(B, X);
                for (int w = 0; w < NW; ++w) B[w] = X[w];
            }
            T::node_hash(A, B, Z, tab);
            for (int w = 0; w < NW; ++w) P[w] = hasB ? Z[w] : hasA ? A[w] : 0u;
        }
        if (cnt > 0) n = (cnt + 1) / 2;
        // Thread k now holds node k of the current level in P (k < n).  While
        // the level spans more than one wave, children meet through LDS; as
        // above, a wave with any parent to form hashes on every lane, reading
        // in-bounds children, and a select keeps the lanes k < m.
        while (n > kWave) {
            const uint32_t m = (n + 1) / 2;
            if (i < n) for (int w = 0; w < NW; ++w) lds[w][i] = P[w];
            __syncthreads();
            if ((i & ~(kWave - 1)) < m) {
                const uint32_t a = 2 * i < n ? 2 * i : n - 1, b = 2 * i + 1 < n ? 2 * i + 1 : n - 1;
                uint32_t L[NW], R[NW], Z[NW];
                for (int w = 0; w < NW; ++w) {
                    L[w] = lds[w][a];
                    R[w] = lds[w][b];
                }
                T::node_hash(L, R, Z, tab);
                const bool pair = i < m && 2 * i + 1 < n, single = i < m && 2 * i + 1 >= n;
                for (int w = 0; w < NW; ++w) P[w] = pair ? Z[w] : single ? L[w] : P[w];
            }
            __syncthreads();  // every read of lds is done before the next level writes it
            n = m;
        }
        // The rest of the tile lies in wave 0's lanes: children come from
        // lanes 2k and 2k+1 by cross-lane shuffles, with no barrier.  Every
        // lane of the wave takes part in the shuffles and hashes (a wave with
        // few active lanes runs each block slower, and the wave issues the
        // same instructions either way); a select keeps the lanes k < m.
        if (i < kWave) {
            while (n > 1) {
                const uint32_t m = (n + 1) / 2;
                uint32_t L[NW], R[NW], Z[NW];
                for (int w = 0; w < NW; ++w) {
                    L[w] = __shfl(P[w], (int)((2 * i) & (kWave - 1)));
                    R[w] = __shfl(P[w], (int)((2 * i + 1) & (kWave - 1)));
                }
                T::node_hash(L, R, Z, tab);
                const bool pair = i < m && 2 * i + 1 < n, single = i < m && 2 * i + 1 >= n;
                for (int w = 0; w < NW; ++w) P[w] = pair ? Z[w] : single ? L[w] : P[w];
                n = m;
            }
            if (i == 0) T::store(out + NB * tile, P);
        }
        __syncthreads();  // lds is reused by the next tile
    }
}

// A launch over a level of 2^18 entries or more (the host plans which):
// group g of its segment -- entries [8t, min(8t + 8, c)) for the segment's
// t-th group, c its entry count -- is reduced to one node in registers,
// forming the leaf hashes first in leaf mode.  Groups start at multiples of
// 8, so, as with tiles, the promotion of a short last group is the whole
// tree's.  An empty segment has one group, the hash of no entries.
//
// Groups g < n_main take one lane each (blocks below main_blocks).  The
// entries go through a stack of perfect subtrees: entry j is merged with the
// subtrees of the trailing one bits of j (a binary counter), and a short
// group folds what is left, smallest subtree first, which is RFC 6962's split
// at the largest power of two.  Every lane of a wave works on the widest
// levels, with no barrier and no LDS exchange; the loops stay rolled (one
// leaf-hash and one node-hash site), and stack slots are picked with selects
// so that the stack stays in registers.
//
// The launch's last groups, g >= n_main, take four lanes each (the blocks
// after main_blocks): lane q forms the node of entries 2q and 2q + 1, then
// two levels pair lanes (q, q + 1) and (0, 2) through cross-lane shuffles.
// A wave then needs a third of the time per group that a one-lane wave
// needs, which shortens the launch's last round (the host sizes n_main to
// whole rounds of the chip's SIMDs).
template <class T>
__global__ void __launch_bounds__(kThreads, 4) merkle_group_kernel(const uint8_t* __restrict__ in,
                                                                    uint8_t* __restrict__ out,
                                                                    const uint64_t* __restrict__ in_off,
                                                                    const uint64_t* __restrict__ grp_off,
                                                                    uint32_t n_seg, uint64_t n_groups,
                                                                    uint64_t n_main, uint32_t main_blocks,
                                                                    int leaf_mode) {
    constexpr int NW = T::kWords;
    constexpr int NB = T::kBytes;
    constexpr int L = kGroupLevels;
    __shared__ __align__(16) uint32_t tab[T::kTableWords];
    T::stage_table(tab);
    __syncthreads();
    if (blockIdx.x < main_blocks) {
        for (uint64_t g = (uint64_t)blockIdx.x * kThreads + threadIdx.x; g < n_main;
             g += (uint64_t)main_blocks * kThreads) {
            const uint32_t s = find_segment(grp_off, n_seg, g);
            const uint64_t t = g - grp_off[s];
            const uint64_t c = in_off[s + 1] - in_off[s];
            const uint64_t first = t * kGroupNodes;
            const uint32_t cnt =
                c > first ? (uint32_t)(c - first < (uint64_t)kGroupNodes ? c - first : kGroupNodes) : 0u;
            const uint8_t* base = in + NB * (in_off[s] + first);
            uint32_t S[L][NW];  // S[l]: the perfect subtree of 2^l entries waiting for its right sibling
            uint32_t X[NW];
#pragma unroll
            for (int l = 0; l < L; ++l)
                for (int w = 0; w < NW; ++w) S[l][w] = 0;
            if (cnt == 0) T::empty_hash(X);
#pragma nounroll
            for (uint32_t j = 0; j < cnt; ++j) {
                uint32_t A[NW];
                T::load(base + NB * j, A);
                if (leaf_mode) T::leaf_hash(A, X); else for (int w = 0; w < NW; ++w) X[w] = A[w];
                uint32_t l = 0;
#pragma nounroll
                while (l < (uint32_t)L && ((j >> l) & 1u)) {
                    uint32_t Y[NW], Z[NW];
                    for (int w = 0; w < NW; ++w) {
                        uint32_t v = S[0][w];
#pragma unroll
                        for (int q = 1; q < L; ++q) v = l == (uint32_t)q ? S[q][w] : v;
                        Y[w] = v;
                    }
                    T::node_hash(Y, X, Z, tab);
                    for (int w = 0; w < NW; ++w) X[w] = Z[w];
                    ++l;
                }
#pragma unroll
                for (int q = 0; q < L; ++q)
                    for (int w = 0; w < NW; ++w) S[q][w] = l == (uint32_t)q ? X[w] : S[q][w];
            }
            if (cnt > 0 && cnt < (uint32_t)kGroupNodes) {
                bool have = false;
#pragma nounroll
                for (uint32_t l = 0; l < (uint32_t)L; ++l) {
                    if (!((cnt >> l) & 1u)) continue;
                    uint32_t Y[NW];
                    for (int w = 0; w < NW; ++w) {
                        uint32_t v = S[0][w];
#pragma unroll
                        for (int q = 1; q < L; ++q) v = l == (uint32_t)q ? S[q][w] : v;
                        Y[w] = v;
                    }
                    if (!have) {
                        for (int w = 0; w < NW; ++w) X[w] = Y[w];
                        have = true;
                    } else {
                        uint32_t Z[NW];
                        T::node_hash(Y, X, Z, tab);
                        for (int w = 0; w < NW; ++w) X[w] = Z[w];
                    }
                }
            }
            T::store(out + NB * g, X);
        }
        return;
    }
    // Four lanes per group.  The four lanes of a quad share g, so they enter
    // and leave the loop together and every shuffle reads a lane of the same
    // group.
    constexpr uint32_t Q = kGroupQuad;
    const uint32_t q = threadIdx.x % Q;
    const uint64_t quads = (uint64_t)(gridDim.x - main_blocks) * (kThreads / Q);
    for (uint64_t g = n_main + (uint64_t)(blockIdx.x - main_blocks) * (kThreads / Q) + threadIdx.x / Q; g < n_groups;
         g += quads) {
        const uint32_t s = find_segment(grp_off, n_seg, g);
        const uint64_t t = g - grp_off[s];
        const uint64_t c = in_off[s + 1] - in_off[s];
        const uint64_t first = t * kGroupNodes;
        const uint32_t cnt =
            c > first ? (uint32_t)(c - first < (uint64_t)kGroupNodes ? c - first : kGroupNodes) : 0u;
        const uint8_t* base = in + NB * (in_off[s] + first);
        // N: this lane's entry 2q (then its node); X: entry 2q + 1.  Lanes
        // past the group's end keep zeros.
        uint32_t N[NW], X[NW];
        for (int w = 0; w < NW; ++w) N[w] = X[w] = 0;
        if (cnt == 0 && q == 0) T::empty_hash(N);
#pragma nounroll
        for (uint32_t j = 0; j < 2; ++j) {
            const uint32_t e = 2 * q + j;
            uint32_t Y[NW] = {};
            if (e < cnt) {
                uint32_t A[NW];
                T::load(base + NB * e, A);
                if (leaf_mode) T::leaf_hash(A, Y); else for (int w = 0; w < NW; ++w) Y[w] = A[w];
            }
            for (int w = 0; w < NW; ++w) {
                N[w] = j == 0 && e < cnt ? Y[w] : N[w];
                X[w] = j == 1 && e < cnt ? Y[w] : X[w];
            }
        }
        // Level l + 1 from level l: the left node's lane q is a multiple of
        // 2^l; its right sibling is this lane's entry 2q + 1 (l = 0) or the
        // node of lane q + 2^(l-1), which exists when its first entry,
        // 2q + 1 or 2(q + 2^(l-1)), is in the group.  Every lane hashes (these
        // waves run at the end of the launch, where one wave's latency is the
        // time, and a wave with few active lanes runs each block slower); a
        // select keeps the pairs that exist.
#pragma nounroll
        for (uint32_t l = 0; l < (uint32_t)L; ++l) {
            const uint32_t d = l == 0 ? 1u : 1u << (l - 1);
            uint32_t R[NW], Z[NW];
            for (int w = 0; w < NW; ++w) {
                const uint32_t v = (uint32_t)__shfl_xor((int)N[w], (int)d, (int)Q);
                R[w] = l == 0 ? X[w] : v;
            }
            const bool left = (q & ((1u << l) - 1u)) == 0;
            const uint32_t right_first = l == 0 ? 2 * q + 1 : 2 * (q + d);
            T::node_hash(N, R, Z, tab);
            for (int w = 0; w < NW; ++w) N[w] = left && right_first < cnt ? Z[w] : N[w];
        }
        if (q == 0) T::store(out + NB * g, N);
    }
}

}  // namespace

hipError_t launch_merkle_groups(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                                const uint64_t* grp_off, uint32_t n_seg, uint64_t n_groups, uint64_t n_main,
                                int leaf_mode, hipStream_t s) {
    if (n_groups == 0) return hipSuccess;
    if (n_main > n_groups) return hipErrorInvalidValue;
    const uint64_t cap = 1u << 19;  // blocks per part; both parts loop over their groups
    const uint64_t mb = (n_main + kThreads - 1) / kThreads;
    const uint64_t fb = ((n_groups - n_main) * kGroupQuad + kThreads - 1) / kThreads;
    const uint32_t main_blocks = (uint32_t)(mb < cap ? mb : cap);
    const unsigned grid = main_blocks + (unsigned)(fb < cap ? fb : cap);
    if (alg == kAlgSha384)
        merkle_group_kernel<Sha384Tree><<<grid, kThreads, 0, s>>>(in, out, in_off, grp_off, n_seg, n_groups, n_main,
                                                                   main_blocks, leaf_mode);
    else
        merkle_group_kernel<Sha256Tree><<<grid, kThreads, 0, s>>>(in, out, in_off, grp_off, n_seg, n_groups, n_main,
                                                                   main_blocks, leaf_mode);
    return hipGetLastError();
}

hipError_t launch_merkle_tiles(int alg, const uint8_t* in, uint8_t* out, const uint64_t* in_off,
                               const uint64_t* tile_off, uint32_t n_seg, uint64_t n_tiles, int leaf_mode,
                               hipStream_t s) {
    if (n_tiles == 0) return hipSuccess;
    const uint64_t cap = 1u << 20;
    const unsigned grid = (unsigned)(n_tiles < cap ? n_tiles : cap);
    if (alg == kAlgSha384)
        merkle_tile_kernel<Sha384Tree><<<grid, kThreads, 0, s>>>(in, out, in_off, tile_off, n_seg, n_tiles, leaf_mode);
    else
        merkle_tile_kernel<Sha256Tree><<<grid, kThreads, 0, s>>>(in, out, in_off, tile_off, n_seg, n_tiles, leaf_mode);
    return hipGetLastError();
}

}  // namespace hv
