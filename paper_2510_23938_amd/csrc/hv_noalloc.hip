// hv_noalloc.hip -- hv_hash_chunks_noalloc (include/hv.h): the chunk digests of
// hv_hash_chunks_alg for callers that cannot allocate device memory or pass a
// workspace.  The scheduler's scratch (message descriptors, per-message counts
// and their scan, the tail histogram and the leaf table) lives in a static
// device array of HV_NOALLOC_SCRATCH_BYTES, one copy per GPU, held until the
// process ends.  The kernels are those of hv_hash_chunks_alg.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hv.h"
#include "hv_host.h"

using namespace hvh;

// The scratch array.  In host code its name stands for the host-side shadow
// of the variable, not a device address: kernels and copies get the address
// hipGetSymbolAddress returns for the device they run on.
static __device__ __align__(256) uint8_t scratch[HV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the scratch array on the device that owns `stream`,
// looked up once per device with that device current.
hv_status scratch_of(hipStream_t stream, void** out) {
    int dev = -1;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return hip_fail(e, "stream device query");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(HV_ERR_INVALID_ARG, "device %d is outside the %d devices this library tracks", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        int cur = -1;
        if ((e = hipGetDevice(&cur)) != hipSuccess) return hip_fail(e, "device query");
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "set device");
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t back = hipSetDevice(cur);
            if (e == hipSuccess) e = back;
        }
        if (e != hipSuccess) return hip_fail(e, "scratch address");
        if (p == nullptr || (uintptr_t)p % kAlign != 0)
            return fail(HV_ERR_HIP, "scratch address %p is not %zu-byte aligned", p, kAlign);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return HV_OK;
}

}  // namespace

extern "C" hv_status hv_hash_chunks_noalloc(hv_alg alg, const hv_msg* msgs, uint32_t n_msgs, uint64_t chunk_bytes,
                                            uint8_t* leaf_digests, hipStream_t stream) {
    // Every argument check comes before the first HIP call (the scratch lookup).
    if (alg != HV_SHA256 && alg != HV_SHA384) return fail(HV_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
    if (alg == HV_SHA384 && chunk_bytes % 128 != 0)
        return fail(HV_ERR_INVALID_ARG, "chunk_bytes = %llu is not 0 or a multiple of 128 (SHA-384 blocks)",
                    (unsigned long long)chunk_bytes);
    uint64_t n_leaves = 0;
    hv_status st = layout(msgs, n_msgs, chunk_bytes, nullptr, &n_leaves, nullptr);
    if (st != HV_OK) return st;
    if (n_leaves > kMaxLeaves)
        return fail(HV_ERR_INVALID_ARG, "%llu leaves exceed the per-call limit", (unsigned long long)n_leaves);
    if (n_leaves > 0 && leaf_digests == nullptr) return fail(HV_ERR_INVALID_ARG, "leaf_digests is NULL");
    if ((uintptr_t)leaf_digests % 16 != 0) return fail(HV_ERR_INVALID_ARG, "leaf_digests is not 16-byte aligned");
    const size_t need = hash_layout(nullptr, n_msgs, n_leaves).bytes;
    if (need > (size_t)HV_NOALLOC_SCRATCH_BYTES)
        return fail(HV_ERR_INVALID_ARG,
                    "%u messages with %llu leaves need %zu bytes of scratch; the static scratch holds %zu "
                    "(use hv_hash_chunks_alg with a workspace)",
                    n_msgs, (unsigned long long)n_leaves, need, (size_t)HV_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    if ((st = scratch_of(stream, &ws)) != HV_OK) return st;
    // No events here (no timing, a blocking descriptor upload): creating them
    // would allocate runtime objects.
    return hash_chunks_into(alg, msgs, n_msgs, chunk_bytes, leaf_digests, ws, HV_NOALLOC_SCRATCH_BYTES, false,
                            stream);
}
