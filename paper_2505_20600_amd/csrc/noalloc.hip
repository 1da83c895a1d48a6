// Step contexts for callers that cannot allocate device memory: the workspace
// of mask_step_init_static is a fixed device array of the library (one copy per
// device the library runs on, held until the process ends) instead of caller
// memory. Every kernel of the step takes the array's device address as an
// ordinary pointer argument, exactly as it takes a caller's workspace.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/maskstep.h"
#include "step_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[MS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];     // device address of `scratch` on each device, resolved once
bool g_held[kMaxDevices];     // a live step context uses the device's array

}  // namespace

namespace ms {

void release_static_scratch(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return;
    std::lock_guard<std::mutex> lk(g_mu);
    g_held[dev] = false;
}

}  // namespace ms

extern "C" ms_status mask_step_init_static(ms_step** out, const ms_model_desc* desc, int32_t batch,
                                           const uint8_t* d_mask, void* stream) {
    if (!out) return ms::set_error(MS_EINVAL, "out is NULL");
    *out = nullptr;
    size_t need = 0;
    ms_status st = ms::workspace_need(desc, batch, &need);
    if (st != MS_OK) return st;
    if (need > MS_STATIC_SCRATCH_BYTES)
        return ms::set_error(MS_EWORKSPACE, "this step needs %zu bytes of workspace; the static scratch holds %zu",
                             need, (size_t)MS_STATIC_SCRATCH_BYTES);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return ms::set_error(MS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return ms::set_error(MS_EINVAL, "device %d outside 0..%d", dev, kMaxDevices - 1);
    void* ws = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (g_held[dev])
            return ms::set_error(MS_ESTATE, "the static scratch of device %d is held by another step context "
                                            "(destroy it first)", dev);
        if (!g_ptr[dev]) {
            // the array's address on this device (the host-side name is not one)
            void* p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p)
                return ms::set_error(MS_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                                     hipGetErrorString(e));
            g_ptr[dev] = p;
        }
        g_held[dev] = true;
        ws = g_ptr[dev];
    }
    st = ms::step_init(out, desc, batch, d_mask, ws, MS_STATIC_SCRATCH_BYTES, stream, dev);
    if (st != MS_OK) ms::release_static_scratch(dev);
    return st;
}
