// base_assign_noalloc: the balanced assignment of base_assign with its
// workspace taken from a library-owned device array instead of the caller,
// for callers that cannot allocate device memory (code under graph capture,
// tight serving loops, harnesses that forbid allocation).
//
// The array is a file-scope __device__ array: every device the library runs
// on holds its own copy, for the life of the process. In host code the
// array's name only stands in for the symbol; its device address on each
// device is resolved once, with that device current, by hipGetSymbolAddress
// and kept per device, and only that address is ever handed to kernels.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "base.h"
#include "internal.hpp"

namespace {

constexpr size_t kScratchBytes = BASE_ASSIGN_NOALLOC_MAX_WORKSPACE;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on device `dev` (resolved once per
// device). Returns nullptr if it cannot be resolved.
void *scratch_on(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] != nullptr) return g_scratch_ptr[dev];
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return nullptr;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
    void *ptr = nullptr;
    const hipError_t err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (err != hipSuccess || ptr == nullptr) {
        (void)hipGetLastError();
        return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
    return ptr;
}

}  // namespace

extern "C" int base_assign_noalloc(const void *S, int s_dtype, int64_t T, int64_t E,
                                   const base_assign_opts *opts, int32_t *assign, int32_t *perm,
                                   void *prices, base_assign_stats *stats, void *stream) {
    const size_t need = base_assign_workspace_size(T, E);
    if (need == 0) {
        // Sizes base_assign rejects: report them as it does (nothing enqueued).
        return base::assign_entry(S, s_dtype, 1, T, E, opts, assign, perm, prices, nullptr, 0,
                                  stats, stream);
    }
    if (need > kScratchBytes) return BASE_ERR_RANGE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = 0;
    if (hipStreamGetDevice(s, &dev) != hipSuccess) {
        (void)hipGetLastError();
        return BASE_ERR_HIP;
    }
    void *ws = scratch_on(dev);
    if (ws == nullptr) return BASE_ERR_HIP;
    return base::assign_entry(S, s_dtype, 1, T, E, opts, assign, perm, prices, ws, kScratchBytes,
                              stats, stream);
}
