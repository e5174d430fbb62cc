// deer_scan_noalloc: the bare affine scan of deer_scan for callers that cannot allocate device
// memory (code under HIP graph capture, serving loops, harnesses that forbid hipMalloc).  Its
// scratch -- chunk aggregates, carries, group maps, look-back flags -- lives in the file-scope
// device array below instead of a caller-supplied workspace.  Each GPU the library runs on holds
// its own copy of the array from module load until the process ends; every call on a GPU shares
// that GPU's copy, so calls that overlap on one GPU (two streams, two threads) race, and the
// caller must serialise them.  What the scan needs to start at zero (the look-back flags of the
// diagonal scan) is cleared by a kernel of the scan itself; everything else is written before it
// is read.
#include <mutex>

#include "common.h"
#include "launch.h"

namespace deer {

constexpr size_t kScratchBytes = (size_t)64 << 20;   // 64 MiB per GPU
constexpr int kMaxDevices = 64;

// The host-side name of this array is a stand-in, not a device address: host code uses only
// the pointer hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

static std::mutex g_scratch_mu;
static void *g_scratch_ptr[kMaxDevices];

// Device address of the current GPU's copy of `scratch`, looked up on the first call on that
// device (with it current) and kept for the life of the process.
static int scratch_on_current_device(void **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("deer_scan_noalloc: device %d is beyond the %d devices the library tracks", dev, kMaxDevices);
        return DEER_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) {
            set_error("hipGetSymbolAddress(scratch) returned a null address");
            return DEER_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DEER_OK;
}

}  // namespace deer

using namespace deer;

extern "C" {

size_t deer_noalloc_scratch_bytes(void) { return kScratchBytes; }

int deer_scan_noalloc(int layout, int reverse, int transpose, int B, int T, int M, const float *J, const float *b,
                      float *y, void *stream) {
    set_error("");
    const size_t need = deer_scan_workspace_bytes(layout, reverse, transpose, B, T, M);
    if (need == 0) {
        set_error("deer_scan_noalloc: unknown layout or sizes out of range (layout %d, B %d, T %d, M %d)", layout, B,
                  T, M);
        return DEER_ERR_INVALID_ARG;
    }
    if (need > kScratchBytes) {
        set_error("deer_scan_noalloc: B = %d, T = %d, M = %d need %zu bytes of scratch, more than the %zu bytes "
                  "the library holds per GPU (use deer_scan with a workspace)",
                  B, T, M, need, kScratchBytes);
        return DEER_ERR_INVALID_ARG;
    }
    void *ws = nullptr;
    int rc = scratch_on_current_device(&ws);
    if (rc) return rc;
    // the timing diagnostics create HIP events: none are recorded for this call
    TimingSuppress quiet;
    return deer_scan(layout, reverse, transpose, B, T, M, J, b, y, ws, need, stream);
}

}  // extern "C"
