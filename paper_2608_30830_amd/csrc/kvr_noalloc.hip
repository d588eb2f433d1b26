// Allocation-free variant of kvr_cost_grid, for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops).  Its
// workspace is a file-scope device array of KVR_NOALLOC_SCRATCH_BYTES: every
// GPU that loads the library holds one copy of it until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory; the
// device address of each GPU's copy comes from hipGetSymbolAddress, called
// once per device with that device current, and only that address is ever
// handed to kernels.  Calls on one GPU share its copy, so calls that overlap
// in time on one GPU (different streams) race; calls queued on one stream do
// not.  Nothing in the array needs clearing between calls: the kernels of
// kvr_cost_grid clear their status word, counters and sums themselves, as they
// do in a caller's uninitialised workspace.
#include "kvr_internal.h"

#include <atomic>
#include <mutex>

namespace {

constexpr size_t kScratchBytes = KVR_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::atomic<void *> g_scratch_ptr[kMaxDevices];

// Device address of the copy of `scratch` on the device that runs `s` (the
// current device for the null stream), looked up on the first call there.
int scratch_address(hipStream_t s, void **out)
{
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return KVR_E_HIP;
    int dev = cur;
    if (s != nullptr) {
        hipDevice_t sd = 0;
        if (hipStreamGetDevice(s, &sd) != hipSuccess) return KVR_E_HIP;
        dev = (int)sd;
    }
    if (dev < 0 || dev >= kMaxDevices) return KVR_E_HIP;
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == nullptr) {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (p == nullptr) {
            if (dev != cur && hipSetDevice(dev) != hipSuccess) return KVR_E_HIP;
            const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (dev != cur && hipSetDevice(cur) != hipSuccess) return KVR_E_HIP;
            if (e != hipSuccess || p == nullptr) return KVR_E_HIP;
            g_scratch_ptr[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return KVR_OK;
}

}  // namespace

extern "C" int kvr_cost_grid_noalloc(const double *d_wait_s, const int32_t *d_ctx_tokens,
                                     int64_t n, const kvr_prices *p, const kvr_policy_grid *g,
                                     int32_t method, double *d_cost, int32_t *d_perm,
                                     int32_t *d_status, void *hip_stream)
{
    // host checks and the plan first: nothing is launched unless it fits
    size_t need = 0;
    int rc = kvr::cost_grid_entry(d_wait_s, d_ctx_tokens, n, p, g, method, d_cost, d_perm,
                                  nullptr, &need, kScratchBytes, hip_stream);
    if (rc != KVR_OK) return rc;
    if (need > kScratchBytes) return KVR_E_SIZE;
    if (!d_wait_s || !d_ctx_tokens || !d_cost) return KVR_E_NULL;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    void *ws = nullptr;
    if ((rc = scratch_address(s, &ws)) != KVR_OK) return rc;
    size_t have = kScratchBytes;
    rc = kvr::cost_grid_entry(d_wait_s, d_ctx_tokens, n, p, g, method, d_cost, d_perm, ws, &have,
                              kScratchBytes, hip_stream);
    if (rc != KVR_OK) return rc;
    if (d_status != nullptr &&
        kvr::launch_export_status(static_cast<const int *>(ws), d_status, s) != hipSuccess)
        return KVR_E_HIP;
    return KVR_OK;
}
