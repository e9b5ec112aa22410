// Allocation-free variant of the whole-layer forward: the same kernel
// sequence as moe_layer_forward, with its workspace taken from a device array
// of this library instead of a caller buffer.
//
// The array lives in this translation unit's code object, so every GPU the
// library runs on holds its own copy (MOE_NOALLOC_SCRATCH_BYTES) from the
// first call on that GPU until the process ends. Its device address is looked
// up once per device with hipGetSymbolAddress while that device is current;
// host code passes only that address on (the array's own name is a host-side
// stand-in and never reaches a kernel). No kernel of the layer expects zeroed
// workspace: every counter it uses is cleared by a kernel of the same call,
// so the contents left by the previous call do not matter. Calls that overlap
// on one GPU share the array and race.
#include <mutex>

#include "moe_internal.h"

#define MOE_API extern "C" __attribute__((visibility("default")))

namespace moe {
namespace {

static __device__ __align__(256) uint8_t scratch[MOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device (looked up on the first
// call per device).
moe_status_t scratch_address(void** out) {
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_last_error(MOE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return set_last_error(MOE_ERR_UNSUPPORTED, "device %d is beyond the %d devices supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e2 = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e2 != hipSuccess || !p)
            return set_last_error(MOE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                                  hipGetErrorString(e2));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MOE_OK;
}

}  // namespace
}  // namespace moe

using namespace moe;

MOE_API moe_status_t moe_layer_forward_noalloc(const moe_desc_t* desc, const void* x, const void* w_router,
                                               const float* bias, const void* w1, const void* w2,
                                               const void* w1s, const void* w2s, void* y, int32_t* topk_idx_out,
                                               float* topk_gate_out, void* stream) {
    size_t need = 0;
    const moe_status_t st = moe_workspace_size(desc, &need);  // validates desc
    if (st != MOE_OK) return st;
    if (need > (size_t)MOE_NOALLOC_SCRATCH_BYTES)
        return set_last_error(MOE_ERR_WORKSPACE,
                              "the layer needs %zu bytes of scratch; the allocation-free entry point holds %zu",
                              need, (size_t)MOE_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    const moe_status_t sa = scratch_address(&ws);
    if (sa != MOE_OK) return sa;
    return moe_layer_forward(desc, x, w_router, bias, w1, w2, w1s, w2s, y, topk_idx_out, topk_gate_out, ws,
                             (size_t)MOE_NOALLOC_SCRATCH_BYTES, nullptr, stream);
}
