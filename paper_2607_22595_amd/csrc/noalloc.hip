// SAE encode + TopK without a caller workspace, for callers that cannot
// allocate device memory (code under graph capture, tight serving loops,
// harnesses that forbid allocation).  The workspace of xmix_sae_encode_topk
// (folded-bias area and candidate area) lives in a file-scope device array
// of fixed size; each device holds its own copy of it for the life of the
// process.  Its device address is looked up once per device, with that
// device current, and only that address is handed to the kernels (the
// array's name in host code is a host-side stand-in, not a device address).
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/xmix.h"

static __device__ __align__(256) unsigned char scratch[XMIX_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device (nullptr on error).
void* scratch_on_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> g(g_lock);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_ptr[dev] = p;
    }
    return g_ptr[dev];
}

}  // namespace

extern "C" xmix_status xmix_sae_encode_topk_noalloc(const uint16_t* h, int32_t d,
                                                    const xmix_route* rt, int32_t app_bit,
                                                    const xmix_sae_dict* dict,
                                                    const uint16_t* b_enc, const uint16_t* b_dec,
                                                    const float* c_fold, int32_t k,
                                                    int32_t* idx_out, uint16_t* val_out,
                                                    void* stream) {
    if (!rt || !dict || rt->T_max < 1) return XMIX_E_INVAL;
    const size_t need = xmix_sae_encode_workspace(rt->T_max, d, dict->m, k);
    if (need == 0) return XMIX_E_INVAL;
    if (need > static_cast<size_t>(XMIX_STATIC_SCRATCH_BYTES)) return XMIX_E_UNSUPPORTED;
    void* ws = scratch_on_current_device();
    if (!ws) return XMIX_E_LAUNCH;
    // Nothing in the workspace has to start at zero: the candidates stage
    // writes every (token, slice) entry the merge reads in the same call.
    return xmix_sae_encode_topk(h, d, rt, app_bit, dict, b_enc, b_dec, c_fold, k, idx_out,
                                val_out, ws, static_cast<size_t>(XMIX_STATIC_SCRATCH_BYTES),
                                stream);
}
