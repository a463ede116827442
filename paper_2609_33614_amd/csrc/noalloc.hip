// Allocation-free layer forward: eat_moe_forward with its workspace in a
// fixed device array of this library instead of a caller-provided buffer.
//
// `scratch` is a file-scope device array; each GPU that loads this code
// object holds its own copy at its own address.  Host code must not pass
// the array's name to a kernel (on the host it names a stand-in, not device
// memory): the entry point looks the device address up with
// hipGetSymbolAddress once per device, with that device current, keeps it
// in a per-device table and hands that address to the forward's kernels as
// their workspace, exactly as eat_moe_forward hands over the caller's.
#include <atomic>
#include <mutex>

#include "eat_internal.h"

namespace {

constexpr size_t kScratchBytes = EAT_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch keeps the workspace's 256-byte alignment");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];    // device address of `scratch` per device, once known
std::mutex g_lookup;

// Device address of this device's `scratch` (looked up on the first call
// with the device current).
eat_status_t scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return EAT_ERR_HIP;
    void* p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> g(g_lookup);
        p = g_scratch[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return EAT_ERR_HIP;
            g_scratch[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return EAT_OK;
}

}  // namespace

extern "C" eat_status_t eat_moe_forward_noalloc(eat_handle_t h, const void* x, int32_t T, const float* w_router,
                                                const void* w1, const void* w3, const void* w2, const void* ws1,
                                                const void* ws3, const void* ws2, eat_accounts_t acc,
                                                const int8_t* ppl_trend, void* y, uint64_t* mask_out,
                                                int32_t* expert_load_out, hipStream_t stream) {
    const eat_status_t st = eat::check_forward(h, x, T, w_router, w1, w3, w2, ws1, ws3, ws2, acc, y, mask_out,
                                               expert_load_out);
    if (st != EAT_OK) return st;
    if (eat::plan_workspace(*h, T).total > kScratchBytes) return EAT_ERR_SCRATCH_LIMIT;
    if (T == 0) return EAT_OK;
    void* ws = nullptr;
    if (scratch_address(&ws) != EAT_OK) return EAT_ERR_HIP;
    (void)hipGetLastError();
    const hipError_t e = eat::forward_impl(*h, x, T, w_router, w1, w3, w2, ws1, ws3, ws2, acc, ppl_trend, nullptr,
                                           y, mask_out, expert_load_out, nullptr, ws, stream, nullptr, 0);
    return e == hipSuccess ? EAT_OK : EAT_ERR_HIP;
}
