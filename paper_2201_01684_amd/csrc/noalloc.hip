// gpoeo_pd_detect_noalloc: gpoeo_pd_detect with its workspace taken from a
// static device array instead of a caller buffer, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops).
//
// The array lives in this code object, so every GPU the library runs on holds
// its own copy, at its own address, until the process ends.  In host code the
// array's name is only a stand-in for the symbol: its device address comes
// from hipGetSymbolAddress, taken once per device (with that device current,
// on the first call made there) and kept; only that address is ever handed to
// kernels.  The detection clears everything it reads back (tier bitmaps,
// queues, window states) with its own fill kernel, so the array's contents on
// entry do not matter.  Calls that overlap on one GPU share the array and
// race: the caller serialises them (one stream, or events between streams).
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "gpoeo_pd.h"
#include "internal.h"

namespace {

constexpr size_t kScratchBytes = GPOEO_PD_NOALLOC_MAX_WORKSPACE;
static_assert(kScratchBytes % 256 == 0, "the workspace must keep its 256-byte alignment");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_init_mutex;
std::atomic<void*> g_scratch[kMaxDevices];

// Device address of `scratch` on the current device (looked up on the first
// call there).
int scratch_on_current_device(hipStream_t stream, void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return GPOEO_PD_EHIP;
    if (dev >= kMaxDevices) return GPOEO_PD_EINVAL;
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return GPOEO_PD_EHIP;
    if (sdev != dev) return GPOEO_PD_EINVAL;   // the stream must belong to the current device
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(g_init_mutex);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
                return GPOEO_PD_EHIP;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return GPOEO_PD_OK;
}

}  // namespace

extern "C" int gpoeo_pd_detect_noalloc(const gpoeo_pd_desc* desc, const float* x, float* scores,
                                       gpoeo_pd_result* results, hipStream_t stream) {
    size_t need = 0;
    const int rc = gpoeo_pd_workspace_bytes(desc, &need);   // validates desc (host only)
    if (rc != GPOEO_PD_OK) return rc;
    if (!x || (!results && !(desc->flags & GPOEO_PD_SCORES_ONLY))) return GPOEO_PD_EINVAL;
    if (need > kScratchBytes) return GPOEO_PD_ETOOBIG;
    void* ws = nullptr;
    const int sc = scratch_on_current_device(stream, &ws);
    if (sc != GPOEO_PD_OK) return sc;
    return gpoeo_pd_detect(desc, x, scores, results, ws, kScratchBytes, stream);
}
