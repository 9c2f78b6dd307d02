// fox_attn_fwd for callers that cannot allocate device memory (code under
// graph capture, tight serving loops): the workspace is a fixed array that the
// library's code object holds on every GPU it runs on, instead of a caller
// buffer.  Everything else is fox_attn_fwd itself.
#include <hip/hip_runtime.h>

#include <mutex>

#include "acp.h"
#include "acp_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;

// One copy per GPU, kept until the process ends.  In host code this name is a
// stand-in, not a device address: only the pointer hipGetSymbolAddress returns
// for the current device may be handed to kernels or copies.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of this GPU's scratch array, looked up once per device
// (with that device current) on its first call.
acp_status scratch_for_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return acp::set_error(ACP_EHIP, "fox_attn_fwd_noalloc: hipGetDevice failed");
    if (dev < 0 || dev >= kMaxDevices)
        return acp::set_error(ACP_EUNSUPPORTED, "fox_attn_fwd_noalloc: device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return acp::set_error(ACP_EHIP, "fox_attn_fwd_noalloc: hipGetSymbolAddress failed");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return ACP_OK;
}

}  // namespace

extern "C" {

size_t acp_noalloc_scratch_bytes(void) { return kScratchBytes; }

acp_status fox_attn_fwd_noalloc(const void* Q, const void* K, const void* V, const float* log_f,
                                acp_dtype dt, int B, int H, int L, int d, double eps, void* O,
                                float* lse, void* stream) {
    // shapes first (nothing touches the GPU before they are known to fit)
    size_t need = 0;
    const acp_status s = acp_workspace_size(B, H, L, d, dt, &need);
    if (s != ACP_OK) return s;
    if (need > kScratchBytes)
        return acp::set_error(ACP_EWORKSPACE,
                              "fox_attn_fwd_noalloc: these shapes need %zu bytes of scratch, more "
                              "than the fixed %zu; call fox_attn_fwd with a workspace",
                              need, kScratchBytes);
    void* ws = nullptr;
    const acp_status t = scratch_for_current_device(&ws);
    if (t != ACP_OK) return t;
    return fox_attn_fwd(Q, K, V, log_f, dt, B, H, L, d, eps, O, lse, ws, kScratchBytes, stream);
}

}  // extern "C"
