// sched.hip -- chunk scheduler: from message descriptors to the leaf table the
// SHA-256 kernel walks, on the device.
//
// Chunking is Algorithm 1's chunk_count = ceil(|M| / C): message m of L bytes
// has floor(L / C) full chunks and, when L mod C != 0, one shorter tail chunk
// (C == 0: one leaf, the whole message).  Leaf numbers (where the digest goes)
// are message-major, chunk-ascending.
//
// The hash kernel runs one chunk per lane, so a wave costs as much as its
// longest chunk.  The table is therefore ordered by SHA-256 block count,
// longest first: every full chunk has C/64 + 1 blocks, the most any chunk of
// the call can have, so they come first in message order; tails follow,
// counting-sorted on their block count (exact below 2048 blocks, then classes
// 1/32 of an octave wide).  The order only changes speed, never a digest.
#include "hv_kernels.h"

namespace hv {
namespace {

constexpr int kThreads = 256;
constexpr int kScanPerThread = 4;
constexpr int kScanTile = kThreads * kScanPerThread;

__device__ __forceinline__ Pair pair_add(Pair a, Pair b) { return make_ulonglong2(a.x + b.x, a.y + b.y); }

// Exclusive scan of one value per thread over the block; *total gets the sum.
__device__ Pair block_exclusive_scan(Pair v, Pair* total) {
    __shared__ Pair sh[kThreads];
    const int tid = threadIdx.x;
    sh[tid] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        const Pair t = tid >= off ? sh[tid - off] : make_ulonglong2(0, 0);
        __syncthreads();
        sh[tid] = pair_add(sh[tid], t);
        __syncthreads();
    }
    const Pair incl = sh[tid];
    *total = sh[kThreads - 1];
    __syncthreads();
    return make_ulonglong2(incl.x - v.x, incl.y - v.y);
}

__global__ void __launch_bounds__(kThreads) fill_u64_kernel(uint64_t* p, size_t n, uint64_t v) {
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (size_t)gridDim.x * kThreads) p[i] = v;
}

__global__ void __launch_bounds__(kThreads) count_kernel(const MsgDesc* __restrict__ msgs, uint32_t n, uint64_t C,
                                                         Pair* __restrict__ cnt) {
    for (size_t m = (size_t)blockIdx.x * kThreads + threadIdx.x; m < n; m += (size_t)gridDim.x * kThreads) {
        const uint64_t len = msgs[m].nbytes;
        if (C == 0) {
            cnt[m] = make_ulonglong2(0, 1);
        } else {
            cnt[m] = make_ulonglong2(len / C, (len % C) != 0 ? 1 : 0);
        }
    }
}

// Phase 1: sums of kScanTile-element tiles.
__global__ void __launch_bounds__(kThreads) scan_tiles_kernel(const Pair* __restrict__ in, size_t n,
                                                              Pair* __restrict__ partials) {
    const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPerThread;
    Pair s = make_ulonglong2(0, 0);
    for (int k = 0; k < kScanPerThread; ++k)
        if (base + k < n) s = pair_add(s, in[base + k]);
    Pair total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Phase 2: exclusive scan of the tile sums, in place (one block, any length).
__global__ void __launch_bounds__(kThreads) scan_partials_kernel(Pair* __restrict__ partials, size_t m) {
    const size_t per = (m + kThreads - 1) / kThreads;
    const size_t lo = (size_t)threadIdx.x * per;
    const size_t hi = lo + per < m ? lo + per : m;
    Pair s = make_ulonglong2(0, 0);
    for (size_t i = lo; i < hi; ++i) s = pair_add(s, partials[i]);
    Pair total;
    Pair run = block_exclusive_scan(s, &total);
    for (size_t i = lo; i < hi; ++i) {
        const Pair v = partials[i];
        partials[i] = run;
        run = pair_add(run, v);
    }
}

// Phase 3: out[i] = sum of in[0..i) for i in [0, n]; out[n] is the total.
__global__ void __launch_bounds__(kThreads) scan_apply_kernel(const Pair* __restrict__ in, size_t n,
                                                              const Pair* __restrict__ partials, Pair* __restrict__ out) {
    const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPerThread;
    Pair v[kScanPerThread];
    Pair s = make_ulonglong2(0, 0);
    for (int k = 0; k < kScanPerThread; ++k) {
        v[k] = base + k < n ? in[base + k] : make_ulonglong2(0, 0);
        s = pair_add(s, v[k]);
    }
    Pair total;
    Pair run = pair_add(block_exclusive_scan(s, &total), partials[blockIdx.x]);
    for (int k = 0; k < kScanPerThread; ++k) {
        if (base + k < n) out[base + k] = run;
        run = pair_add(run, v[k]);
        if (base + k + 1 == n) out[n] = run;
    }
}

// The message holding full chunk f: off[m].x <= f < off[m+1].x.
__device__ __forceinline__ uint32_t find_full_owner(const Pair* __restrict__ off, uint32_t n, uint64_t f) {
    uint32_t lo = 0, hi = n;  // off[lo].x <= f < off[hi].x
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (off[mid].x <= f) lo = mid; else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(kThreads) full_kernel(const MsgDesc* __restrict__ msgs, const Pair* __restrict__ off,
                                                        uint32_t n, uint64_t C, uint64_t n_full,
                                                        LeafDesc* __restrict__ desc) {
    for (uint64_t f = (uint64_t)blockIdx.x * kThreads + threadIdx.x; f < n_full; f += (uint64_t)gridDim.x * kThreads) {
        const uint32_t m = find_full_owner(off, n, f);
        const uint64_t i = f - off[m].x;
        const uint64_t first_leaf = off[m].x + off[m].y;
        LeafDesc d;
        d.src = msgs[m].data + i * C;
        d.nbytes = C;
        d.out = first_leaf + i;
        desc[f] = d;
    }
}

// SHA-256 blocks of an n-byte message: data, the 0x80 byte and the 8-byte length.
__device__ __forceinline__ uint64_t sha_blocks(uint64_t nbytes) { return (nbytes + 72) / 64; }

// Sort class of a block count, monotone: exact below 2048, then 32 classes per octave.
__device__ __forceinline__ uint32_t block_class(uint64_t nblk) {
    if (nblk < 2048) return (uint32_t)nblk;
    const int e = 63 - __clzll((long long)nblk);  // >= 11
    return 2048u + (uint32_t)(e - 11) * 32u + (uint32_t)((nblk >> (e - 5)) & 31u);
}

__device__ __forceinline__ bool tail_of(const MsgDesc& msg, uint64_t C, uint64_t* start, uint64_t* len) {
    if (C == 0) { *start = 0; *len = msg.nbytes; return true; }
    const uint64_t full = msg.nbytes / C;
    *start = full * C;
    *len = msg.nbytes - *start;
    return *len != 0;
}

// Tail counts per sort class.  Each workgroup counts its messages' classes in
// LDS and adds its non-zero counts to the global histogram: one global atomic
// per class a workgroup meets, not one per message (10^6 messages fall into
// about a thousand classes, and per-message atomics on so few addresses
// serialise).
__global__ void __launch_bounds__(kThreads) tail_hist_kernel(const MsgDesc* __restrict__ msgs, uint32_t n, uint64_t C,
                                                             uint64_t* __restrict__ hist) {
    __shared__ uint32_t local[kSortBuckets];
    for (int k = threadIdx.x; k < kSortBuckets; k += kThreads) local[k] = 0;
    __syncthreads();
    for (size_t m = (size_t)blockIdx.x * kThreads + threadIdx.x; m < n; m += (size_t)gridDim.x * kThreads) {
        uint64_t start, len;
        const MsgDesc msg = msgs[m];
        if (tail_of(msg, C, &start, &len)) atomicAdd(&local[block_class(sha_blocks(len))], 1u);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kSortBuckets; k += kThreads)
        if (local[k] != 0) atomicAdd((unsigned long long*)&hist[k], (unsigned long long)local[k]);
}

// hist[k] <- first table slot of class k, largest class first (one block).
__global__ void __launch_bounds__(kThreads) tail_cursor_kernel(uint64_t* __restrict__ hist, uint64_t n_full) {
    constexpr int per = kSortBuckets / kThreads;
    // thread t owns classes (kSortBuckets-1 - t*per) down to (kSortBuckets - (t+1)*per)
    const int top = kSortBuckets - 1 - threadIdx.x * per;
    uint64_t s = 0;
    for (int k = 0; k < per; ++k) s += hist[top - k];
    Pair total;
    Pair run = block_exclusive_scan(make_ulonglong2(s, 0), &total);
    uint64_t pos = n_full + run.x;
    for (int k = 0; k < per; ++k) {
        const uint64_t c = hist[top - k];
        hist[top - k] = pos;
        pos += c;
    }
}

// Tail leaves into their class ranges.  A workgroup counts its messages per
// class in LDS, reserves one contiguous run of slots per class it meets with
// a single global atomic on that class's cursor, then gives each message the
// next slot of its class's run by an LDS atomic.  Slots of one class are
// therefore handed out in no fixed order, which is fine: leaves of one class
// have (about) the same block count, and the order never changes a digest.
__global__ void __launch_bounds__(kThreads) tail_scatter_kernel(const MsgDesc* __restrict__ msgs,
                                                                const Pair* __restrict__ off, uint32_t n, uint64_t C,
                                                                uint64_t* __restrict__ cursor,
                                                                LeafDesc* __restrict__ desc) {
    __shared__ uint32_t local[kSortBuckets];  // this workgroup's count per class, then the next rank
    __shared__ uint64_t run[kSortBuckets];    // first slot of this workgroup's run in each class
    for (int k = threadIdx.x; k < kSortBuckets; k += kThreads) local[k] = 0;
    __syncthreads();
    for (size_t m = (size_t)blockIdx.x * kThreads + threadIdx.x; m < n; m += (size_t)gridDim.x * kThreads) {
        uint64_t start, len;
        const MsgDesc msg = msgs[m];
        if (tail_of(msg, C, &start, &len)) atomicAdd(&local[block_class(sha_blocks(len))], 1u);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kSortBuckets; k += kThreads) {
        if (local[k] != 0) run[k] = atomicAdd((unsigned long long*)&cursor[k], (unsigned long long)local[k]);
        local[k] = 0;
    }
    __syncthreads();
    for (size_t m = (size_t)blockIdx.x * kThreads + threadIdx.x; m < n; m += (size_t)gridDim.x * kThreads) {
        uint64_t start, len;
        const MsgDesc msg = msgs[m];
        if (!tail_of(msg, C, &start, &len)) continue;
        const uint32_t k = block_class(sha_blocks(len));
        const uint64_t slot = run[k] + atomicAdd(&local[k], 1u);
        const Pair o = off[m];
        LeafDesc d;
        d.src = msg.data + start;
        d.nbytes = len;
        d.out = o.x + o.y + (C == 0 ? 0 : msg.nbytes / C);
        desc[slot] = d;
    }
}

// The message holding leaf number `leaf`: the last m with first(m) <= leaf,
// first(m) = off[m].x + off[m].y (messages without leaves share their
// successor's first leaf and are skipped by taking the last).
__device__ __forceinline__ uint32_t find_leaf_owner(const Pair* __restrict__ off, uint32_t n, uint64_t leaf) {
    uint32_t lo = 0, hi = n;
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (off[mid].x + off[mid].y <= leaf) lo = mid; else hi = mid;
    }
    return lo;
}

__global__ void __launch_bounds__(kThreads) select_kernel(const MsgDesc* __restrict__ msgs, const Pair* __restrict__ off,
                                                          uint32_t n, uint64_t C, const uint64_t* __restrict__ leaves,
                                                          uint64_t k, LeafDesc* __restrict__ desc) {
    for (uint64_t e = (uint64_t)blockIdx.x * kThreads + threadIdx.x; e < k; e += (uint64_t)gridDim.x * kThreads) {
        const uint64_t leaf = leaves[e];
        const uint32_t m = find_leaf_owner(off, n, leaf);
        const MsgDesc msg = msgs[m];
        const uint64_t i = leaf - (off[m].x + off[m].y);
        LeafDesc d;
        if (C == 0) {
            d.src = msg.data;
            d.nbytes = msg.nbytes;
        } else {
            d.src = msg.data + i * C;
            d.nbytes = msg.nbytes - i * C < C ? msg.nbytes - i * C : C;
        }
        d.out = leaf;
        desc[e] = d;
    }
}

// Leaf table of a contiguous range of leaf numbers [first, first + k), slot e
// writing digest e; block 0's first lane also resets a monitor result pair
// (mismatch count 0, lowest mismatching leaf ~0), so that the comparison that
// follows on the same stream starts from a clean result.
__global__ void __launch_bounds__(kThreads) range_select_kernel(const MsgDesc* __restrict__ msgs,
                                                                const Pair* __restrict__ off, uint32_t n, uint64_t C,
                                                                uint64_t first, uint64_t k, LeafDesc* __restrict__ desc,
                                                                uint64_t* __restrict__ reset) {
    if (reset != nullptr && blockIdx.x == 0 && threadIdx.x == 0) {
        reset[0] = 0;
        reset[1] = ~0ull;
    }
    for (uint64_t e = (uint64_t)blockIdx.x * kThreads + threadIdx.x; e < k; e += (uint64_t)gridDim.x * kThreads) {
        const uint64_t leaf = first + e;
        const uint32_t m = find_leaf_owner(off, n, leaf);
        const MsgDesc msg = msgs[m];
        const uint64_t i = leaf - (off[m].x + off[m].y);
        LeafDesc d;
        if (C == 0) {
            d.src = msg.data;
            d.nbytes = msg.nbytes;
        } else {
            d.src = msg.data + i * C;
            d.nbytes = msg.nbytes - i * C < C ? msg.nbytes - i * C : C;
        }
        d.out = e;
        desc[e] = d;
    }
}

unsigned grid_for(uint64_t n) {
    const uint64_t blocks = (n + kThreads - 1) / kThreads;
    const uint64_t cap = 65536;  // grid-stride loops cover the rest
    return (unsigned)(blocks == 0 ? 1 : (blocks < cap ? blocks : cap));
}

}  // namespace

hipError_t launch_fill_u64(uint64_t* p, size_t n, uint64_t v, hipStream_t s) {
    fill_u64_kernel<<<grid_for(n), kThreads, 0, s>>>(p, n, v);
    return hipGetLastError();
}

hipError_t launch_sched_count(const MsgDesc* msgs, uint32_t n, uint64_t C, Pair* cnt, hipStream_t s) {
    count_kernel<<<grid_for(n), kThreads, 0, s>>>(msgs, n, C, cnt);
    return hipGetLastError();
}

size_t scan_partials_count(size_t n) { return n == 0 ? 1 : (n + kScanTile - 1) / kScanTile; }

hipError_t launch_scan_pairs(const Pair* in, Pair* out, size_t n, Pair* partials, hipStream_t s) {
    const size_t tiles = scan_partials_count(n);
    if (n == 0) {
        fill_u64_kernel<<<1, kThreads, 0, s>>>(reinterpret_cast<uint64_t*>(out), 2, 0);
        return hipGetLastError();
    }
    scan_tiles_kernel<<<(unsigned)tiles, kThreads, 0, s>>>(in, n, partials);
    scan_partials_kernel<<<1, kThreads, 0, s>>>(partials, tiles);
    scan_apply_kernel<<<(unsigned)tiles, kThreads, 0, s>>>(in, n, partials, out);
    return hipGetLastError();
}

hipError_t launch_sched_full(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                             LeafDesc* desc, hipStream_t s) {
    full_kernel<<<grid_for(n_full), kThreads, 0, s>>>(msgs, off, n, C, n_full, desc);
    return hipGetLastError();
}

hipError_t launch_sched_select(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, const uint64_t* leaves,
                               uint64_t k, LeafDesc* desc, hipStream_t s) {
    if (k == 0) return hipSuccess;
    select_kernel<<<grid_for(k), kThreads, 0, s>>>(msgs, off, n, C, leaves, k, desc);
    return hipGetLastError();
}

hipError_t launch_sched_range(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t first,
                              uint64_t k, LeafDesc* desc, uint64_t* reset, hipStream_t s) {
    range_select_kernel<<<grid_for(k), kThreads, 0, s>>>(msgs, off, n, C, first, k, desc, reset);
    return hipGetLastError();
}

// Workgroups of the privatised tail kernels: enough to spread the messages,
// few enough that each covers many messages (its class counts are summed
// once per workgroup).
unsigned tail_grid(uint64_t n) {
    const uint64_t blocks = (n + kThreads - 1) / kThreads;
    return (unsigned)(blocks == 0 ? 1 : (blocks < 512 ? blocks : 512));
}

hipError_t launch_sched_tails(const MsgDesc* msgs, const Pair* off, uint32_t n, uint64_t C, uint64_t n_full,
                              uint64_t* hist, LeafDesc* desc, hipStream_t s) {
    fill_u64_kernel<<<grid_for(kSortBuckets), kThreads, 0, s>>>(hist, kSortBuckets, 0);
    tail_hist_kernel<<<tail_grid(n), kThreads, 0, s>>>(msgs, n, C, hist);
    tail_cursor_kernel<<<1, kThreads, 0, s>>>(hist, n_full);
    tail_scatter_kernel<<<tail_grid(n), kThreads, 0, s>>>(msgs, off, n, C, hist, desc);
    return hipGetLastError();
}

}  // namespace hv
