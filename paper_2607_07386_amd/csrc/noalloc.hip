// Allocation-free variant of sdm_forward for callers that cannot allocate
// device memory: code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc.  The per-token records and the device-error words that
// sdm_forward keeps in its workspace live here in one file-scope device array
// of fixed size.  Every GPU the library runs on holds its own copy of the array
// until the process ends; host code reaches it only through the address that
// hipGetSymbolAddress returns on that device (the array's name in host code is
// a host-side stand-in, not a device address).
#include <hip/hip_runtime.h>

#include <mutex>

#include "sdm.h"
#include "sdm_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)SDM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up once per
// device with that device current.
int scratch_ptr(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return sdm_set_error(SDM_ERR_HIP, "sdm_forward_noalloc: hipGetDevice failed");
    if (dev < 0 || dev >= kMaxDevices) return sdm_set_error(SDM_ERR_UNSUPPORTED, "sdm_forward_noalloc: device id >= 64");
    std::lock_guard<std::mutex> g(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return sdm_set_error(SDM_ERR_HIP, "sdm_forward_noalloc: hipGetSymbolAddress of the scratch array failed");
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return SDM_OK;
}

}  // namespace

extern "C" {

size_t sdm_forward_noalloc_max_bytes(void) { return kScratchBytes; }

int sdm_forward_noalloc(const void* q, const void* k, int x_dtype, const void* cb_q, const void* cb_k, int d_k,
                        int topk, const void* v, const void* alpha, const void* beta, int in_dtype, float* mem,
                        int B, int H, int T, int d_v, int64_t N, int32_t* r_idx, float* r_val, int32_t* w_idx,
                        float* w_val, float* y, float* saved, size_t saved_bytes, void* stream) {
    // sizes past the array are refused on the host, before any device call
    const bool sane = B >= 0 && H >= 0 && T >= 0 && topk >= 1 && topk <= 128;
    if (sane) {
        const size_t need = sdm_scan_fwd_workspace_bytes(B, H, T, topk, topk);
        if (need > kScratchBytes)
            return sdm_set_error(SDM_ERR_UNSUPPORTED,
                                 "sdm_forward_noalloc: these sizes need more than the fixed scratch array "
                                 "(sdm_scan_fwd_workspace_bytes(B, H, T, topk, topk) > "
                                 "sdm_forward_noalloc_max_bytes())");
    }
    void* ws = nullptr;
    if (sane && (int64_t)B * H * T > 0) {
        const int rc = scratch_ptr(&ws);
        if (rc != SDM_OK) return rc;
    }
    return sdm_forward_impl(q, k, x_dtype, cb_q, cb_k, d_k, topk, topk, v, alpha, beta, in_dtype, mem, B, H, T, d_v,
                            N, r_idx, r_val, w_idx, w_val, y, saved, saved_bytes, 0, ws, kScratchBytes, stream,
                            false, nullptr);
}

}  // extern "C"
