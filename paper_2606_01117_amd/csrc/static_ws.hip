// haste_fwd_bce_static: haste_fwd_bce with its scratch in a library-owned device array, for callers
// that cannot allocate (code under graph capture, tight serving loops, harnesses that forbid it).
//
// The array is a file-scope __device__ object, so every GPU the library is loaded on holds its own
// copy for the life of the process.  In host code its name is only a host-side stand-in; the
// device address is looked up once per device with hipGetSymbolAddress (the device being current)
// and cached, and only that address is ever handed to kernels.
#include <mutex>

#include "common.hpp"

namespace {

constexpr size_t kStaticScratchBytes = size_t(8) << 20;   // 8 MiB per device
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_mu;
void *g_ptr[kMaxDevices];   // device address of `scratch`, per device (nullptr: not looked up yet)

// The device address of this device's scratch array; hipSuccess or the runtime's error.
hipError_t scratch_ptr(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {

size_t haste_fwd_bce_static_max_bytes(void) { return kStaticScratchBytes; }

int haste_fwd_bce_static(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias,
                         const int32_t *pos, int32_t P, void *dY, float *dW, float *dbias, int beta, void *stream) {
    // the scratch this call needs: the X^T copy, and on the fused kernel's shapes the bucketed
    // positives of rows of more than 64 (0 for an invalid descriptor: haste_fwd_bce reports it)
    size_t need = haste_workspace_bytes(d, HASTE_OP_BWD_W);
    if (need) {
        const haste::TailArgs a{d->B, d->F_s, d->L, d->G, d->F_in, d->dtype};
        if (haste::fwd_bce_mfma_supported(a, P)) need = haste::fwd_bce_mfma_ws(a, P);
    }
    if (need > kStaticScratchBytes)
        return haste::report(HASTE_ERR_UNSUPPORTED,
                            "haste_fwd_bce_static: this layer needs %zu bytes of scratch, more than the %zu the "
                            "library holds per device (use haste_fwd_bce with a workspace)",
                            need, kStaticScratchBytes);
    void *ws = nullptr;
    if (need) {
        const hipError_t e = scratch_ptr(&ws);
        if (e != hipSuccess)
            return haste::report(HASTE_ERR_HIP, "haste_fwd_bce_static: device address of the scratch array: %s",
                                hipGetErrorString(e));
    }
    // every byte of scratch the call reads it first writes (the X^T copy, padding rows included)
    return haste_fwd_bce(d, X, idx, W, bias, pos, P, dY, dW, dbias, beta, ws, need ? kStaticScratchBytes : 0, stream);
}

}  // extern "C"
