// moe_layer_gpu for callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid hipMalloc): the same launches, with
// the workspace in a file-scope device array instead of a caller's buffer.
//
// The array is a __device__ variable of SPICE_NOALLOC_SCRATCH_BYTES bytes; each GPU the
// library runs on holds its own copy, zero-initialised when the code object is loaded, until
// the process ends.  Its name is only a host-side stand-in: the device address is taken
// once per device with hipGetSymbolAddress (with that device current) and kept, and only
// that address is ever passed to a kernel.  Every completed call leaves the control
// region's counters at zero, which is all the next call needs; the device flags word keeps
// what earlier calls raised and is not reported.  Calls that overlap on one GPU share the
// array and race.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "spice_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[SPICE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of this device's scratch array (taken on the first call on the device).
hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace

namespace spice {
spice_status_t set_error(spice_status_t st, const char* msg);
}

extern "C" spice_status_t moe_layer_gpu_noalloc(
    const spice_moe_cfg_t* cfg, int32_t T, const void* x, const void* w_gate, const float* logit_bias,
    const int32_t* resident_slot, const float* conf, const void* w13_pool, const void* w2_pool, const void* w13_shared,
    const void* w2_shared, const void* w_shared_gate, const void* lore_A, const void* lore_B, double* logits,
    int32_t* topk_idx, float* topk_w, uint8_t* slot_class, int32_t* offsets, int32_t* perm, int32_t* inv_perm,
    float* y_slots, float* y_shared, const spice_host_out_t* host_out, const float* resid, void* out,
    spice_stream_t stream) {
    try {
        const size_t need = spice_workspace_bytes(cfg, T);
        if (need == 0) {  // an invalid cfg or T: the call below reports which
            return moe_layer_gpu(cfg, T, x, w_gate, logit_bias, resident_slot, conf, w13_pool, w2_pool, w13_shared,
                                 w2_shared, w_shared_gate, lore_A, lore_B, logits, topk_idx, topk_w, slot_class,
                                 offsets, perm, inv_perm, y_slots, y_shared, host_out, resid, out, nullptr, 0, stream);
        }
        if (need > (size_t)SPICE_NOALLOC_SCRATCH_BYTES)
            return spice::set_error(SPICE_ERR_UNSUPPORTED,
                                    ("moe_layer_gpu_noalloc: the call needs " + std::to_string(need) +
                                     " bytes of workspace, more than the static scratch of " +
                                     std::to_string((size_t)SPICE_NOALLOC_SCRATCH_BYTES) + " bytes")
                                        .c_str());
        void* ws = nullptr;
        const hipError_t e = scratch_address(&ws);
        if (e != hipSuccess)
            return spice::set_error(SPICE_ERR_HIP, (std::string("moe_layer_gpu_noalloc: scratch address: ") +
                                                    hipGetErrorString(e)).c_str());
        return moe_layer_gpu(cfg, T, x, w_gate, logit_bias, resident_slot, conf, w13_pool, w2_pool, w13_shared,
                             w2_shared, w_shared_gate, lore_A, lore_B, logits, topk_idx, topk_w, slot_class, offsets,
                             perm, inv_perm, y_slots, y_shared, host_out, resid, out, ws,
                             (size_t)SPICE_NOALLOC_SCRATCH_BYTES, stream);
    } catch (...) {
        return spice::set_error(SPICE_ERR_INTERNAL, "moe_layer_gpu_noalloc: internal error");
    }
}
