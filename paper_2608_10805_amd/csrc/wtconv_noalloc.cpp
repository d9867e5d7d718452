// wtconv_backward_noalloc: wtconv_backward with its workspace taken from a
// static device array instead of a caller's buffer, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid allocation). The kernels and their order are exactly
// wtconv_backward's; only the workspace address differs.
#include <mutex>

#include "wtconv_internal.h"

namespace {

constexpr size_t kScratchBytes = WTCONV_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

}  // namespace

// One copy per GPU the library runs on, held until the process ends. Host
// code never uses this name as an address: the device address comes from
// hipGetSymbolAddress, per device (see scratch_ptr).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up

// Device address of `scratch` on the device `stream` belongs to, looked up
// once per device with that device current.
wtconv_status scratch_ptr(hipStream_t stream, void** out)
{
    int dev = -1;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return WTCONV_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return WTCONV_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return WTCONV_ERR_HIP;
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev && hipSetDevice(cur) != hipSuccess) return WTCONV_ERR_HIP;
        if (e != hipSuccess || !p) return WTCONV_ERR_HIP;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return WTCONV_OK;
}

}  // namespace

extern "C" wtconv_status wtconv_backward_noalloc(const wtconv_desc* desc, const void* x, const void* dy,
                                                 const float* base_w, const float* base_scale,
                                                 const float* base_bias, const float* const* level_w,
                                                 const float* const* level_scale, void* dx, float* d_base_w,
                                                 float* d_base_scale, float* d_base_bias,
                                                 float* const* d_level_w, float* const* d_level_scale,
                                                 hipStream_t stream)
{
    const size_t need = wtconv_backward_workspace_bytes(desc);
    if (need == 0)  // a bad descriptor or no plan: wtconv_backward reports which, before any HIP call
        return wtconv_backward(desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, d_base_w,
                               d_base_scale, d_base_bias, d_level_w, d_level_scale, nullptr, 0, stream);
    if (need > kScratchBytes) return WTCONV_ERR_SCRATCH;
    void* ws = nullptr;
    const wtconv_status st = scratch_ptr(stream, &ws);
    if (st != WTCONV_OK) return st;
    return wtconv_backward(desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, d_base_w,
                           d_base_scale, d_base_bias, d_level_w, d_level_scale, ws, kScratchBytes, stream);
}
