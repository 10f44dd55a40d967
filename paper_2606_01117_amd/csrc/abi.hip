// C ABI of libhaste.so: argument validation, kernel selection and launch on the caller's stream.
// Nothing here allocates, frees or synchronises; scratch comes only from the caller's workspace.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "common.hpp"

namespace {

thread_local char g_err[512];

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = 0;
    return HASTE_OK;
}

int hip_status(hipError_t e, const char *what) {
    if (e == hipSuccess) return ok();
    return fail(HASTE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int check_desc(const haste_desc_t *d) {
    if (!d) return fail(HASTE_ERR_INVALID, "desc is NULL");
    if (d->reserved != 0) return fail(HASTE_ERR_INVALID, "desc.reserved must be 0");
    if (d->dtype != HASTE_DTYPE_F32 && d->dtype != HASTE_DTYPE_BF16)
        return fail(HASTE_ERR_INVALID, "dtype %d is neither HASTE_DTYPE_F32 nor HASTE_DTYPE_BF16", d->dtype);
    if (d->B < 0 || d->L < 0) return fail(HASTE_ERR_INVALID, "B and L must be >= 0");
    if (d->F_s <= 0 || d->F_s > INT32_MAX) return fail(HASTE_ERR_INVALID, "F_s must be in [1, 2^31)");
    if (d->G <= 0) return fail(HASTE_ERR_INVALID, "G must be > 0");
    if (d->L % d->G != 0) return fail(HASTE_ERR_INVALID, "L (%lld) must be a multiple of G (%lld)", (long long)d->L,
                                      (long long)d->G);
    if (d->F_in < 1 || d->F_in > d->F_s) return fail(HASTE_ERR_INVALID, "F_in must be in [1, F_s]");
    if (d->B > INT32_MAX || d->G > INT32_MAX) return fail(HASTE_ERR_INVALID, "B and G must be < 2^31");
    if (d->F_s > kMaxFs)
        return fail(HASTE_ERR_UNSUPPORTED, "F_s = %lld exceeds the supported maximum %d", (long long)d->F_s, kMaxFs);
    return HASTE_OK;
}

int need_ptr(const void *p, const char *name) {
    if (!p) return fail(HASTE_ERR_INVALID, "%s is NULL", name);
    if (!aligned16(p)) return fail(HASTE_ERR_INVALID, "%s is not 16-byte aligned", name);
    return HASTE_OK;
}

haste::TailArgs targs(const haste_desc_t *d) { return haste::TailArgs{d->B, d->F_s, d->L, d->G, d->F_in, d->dtype}; }

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

namespace haste {
int report(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}
}  // namespace haste

namespace {

// the forward kernel for a layer: small groups (G = 1, 2, 4, 8) on their own matrix-core kernel,
// larger ones on the gather-once kernel, the rest (fp32, other G) on the vector ALUs
bool fwd_kernel_exists(const haste::TailArgs &a) {
    return haste::fwd_dn_supported(a) || haste::fwd_sg_supported(a) || haste::fwd_mfma_supported(a) ||
           haste::valu_supported(a);
}

// the small-group forward kernels form the loss gradient as they store (given the sorted positives)
bool fwd_small_bce(const haste::TailArgs &a, int P) {
    return P <= haste::kSortPosMax && (haste::fwd_dn_supported(a) || haste::fwd_sg_supported(a));
}

hipError_t fwd_small(const haste::TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                     void *Y, hipStream_t s, const int32_t *spos, int P) {
    if (haste::fwd_dn_supported(a)) return haste::fwd_dn(a, X, idx, W, bias, Y, s, spos, P);
    return haste::fwd_sg(a, X, idx, W, bias, Y, s, spos, P);
}

hipError_t fwd_any(const haste::TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                   void *Y, hipStream_t s) {
    if (haste::fwd_dn_supported(a)) return haste::fwd_dn(a, X, idx, W, bias, Y, s);
    if (haste::fwd_sg_supported(a)) return haste::fwd_sg(a, X, idx, W, bias, Y, s);
    if (haste::fwd_mfma_supported(a)) return haste::fwd_mfma(a, X, idx, W, bias, Y, s);
    return haste::fwd_valu(a, X, idx, W, bias, Y, s);
}

// the backward-weight kernel for a layer: small groups (G = 1, 2, 4, 8) and larger ones on the matrix
// cores (both on the workspace's X^T copy), the rest on the vector ALUs
// backward-feature: small-group kernel, else the general matrix-core kernel, else the VALU kernel
size_t bwd_x_ws(const haste::TailArgs &a) {
    if (haste::bwd_x_dn_supported(a)) return haste::bwd_x_dn_ws(a);
    if (haste::bwd_x_sg_supported(a)) return haste::bwd_x_sg_ws(a);
    return haste::bwd_x_mfma_supported(a) ? haste::bwd_x_mfma_ws(a) : haste::bwd_x_valu_ws(a);
}

bool bwd_w_uses_xt(const haste::TailArgs &a) {
    return haste::bwd_w_dn_supported(a) || haste::bwd_w_sg_supported(a) || haste::bwd_w_mfma_supported(a);
}

hipError_t bwd_w_any(const haste::TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                     float *dbias, int beta, void *ws, hipStream_t s) {
    if (haste::bwd_w_dn_supported(a)) return haste::bwd_w_dn(a, X, idx, dY, dW, dbias, beta, ws, s);
    if (haste::bwd_w_sg_supported(a)) return haste::bwd_w_sg(a, X, idx, dY, dW, dbias, beta, ws, s);
    if (haste::bwd_w_mfma_supported(a)) return haste::bwd_w_mfma(a, X, idx, dY, dW, dbias, beta, ws, s);
    return haste::bwd_w_valu(a, X, idx, dY, dW, dbias, beta, s);
}

#define TRY(x)                      \
    do {                            \
        int _rc = (x);              \
        if (_rc != HASTE_OK) return _rc; \
    } while (0)

}  // namespace

extern "C" {

const char *haste_version(void) { return "haste-mi355x 0.1 (gfx950)"; }

const char *haste_status_str(int status) {
    switch (status) {
        case HASTE_OK: return "ok";
        case HASTE_ERR_INVALID: return "invalid argument";
        case HASTE_ERR_UNSUPPORTED: return "unsupported";
        case HASTE_ERR_WORKSPACE: return "workspace too small";
        case HASTE_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char *haste_last_error(void) { return g_err; }

size_t haste_workspace_bytes(const haste_desc_t *d, int op) {
    if (check_desc(d) != HASTE_OK) return 0;
    const haste::TailArgs a = targs(d);
    if (op == HASTE_OP_REWIRE) return a.L > 0 && haste::rewire_supported(a) ? haste::rewire_ws(a) : 0;
    if (a.B == 0 || a.L == 0) return 0;
    switch (op) {
        case HASTE_OP_FWD: return 0;
        case HASTE_OP_BWD_W: return bwd_w_uses_xt(a) ? haste::bwd_w_mfma_ws(a) : 0;
        case HASTE_OP_BWD_X: return bwd_x_ws(a);
        // the fused kernel and the backward-weight kernel stage the same X^T copy; the fused kernel
        // also buckets rows of many positives (provided for up to kFusedPosWs per row)
        // small groups: the sorted positives (for rows of up to kSortPosMax) after the X^T copy
        case HASTE_OP_FWD_BCE: {
            if (haste::fwd_bce_mfma_supported(a, haste::kFusedPosWs)) return haste::fwd_bce_mfma_ws(a, haste::kFusedPosWs);
            const size_t xws = bwd_w_uses_xt(a) ? haste::bwd_w_mfma_ws(a) : 0;
            if (!fwd_small_bce(a, 0)) return xws;
            return (size_t)haste::round_up((int64_t)xws, 256) +
                   (size_t)haste::round_up(a.B * haste::kSortPosMax * 4, 256);
        }
        // the composed form also keeps dW in the workspace (after the X^T copy)
        case HASTE_OP_REWIRE: return haste::rewire_supported(a) ? haste::rewire_ws(a) : 0;
        // backward-feature's region (partials, transposed weights, supports), then the fused kernel's
        case HASTE_OP_TAIL_STEP:
            return (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_BWD_X), 256) +
                   haste_workspace_bytes(d, HASTE_OP_FWD_BCE);
        case HASTE_OP_TAIL_STEP_SGD:
            return (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_BWD_X), 256) +
                   haste_workspace_bytes(d, HASTE_OP_FWD_BCE_SGD);
        // composed: haste_fwd_bce's region, then dW
        case HASTE_OP_FWD_BCE_SGD:
            if (haste::fwd_bce_mfma_supported(a, haste::kFusedPosWs)) return haste::fwd_bce_mfma_ws(a, haste::kFusedPosWs);
            return (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_FWD_BCE), 256) +
                   (size_t)haste::round_up(a.L * a.F_in * 4, 256);
    }
    return 0;
}

size_t haste_head_workspace_bytes(int64_t B, int64_t F_s, int64_t H, int32_t dtype) {
    if (B <= 0 || F_s <= 0 || H <= 0) return 0;
    return haste::head_ws(B, F_s, H, dtype);
}

int haste_fwd(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias, void *Y,
              void *ws, size_t ws_bytes, void *stream) {
    (void)ws;
    (void)ws_bytes;
    TRY(check_desc(d));
    const haste::TailArgs a = targs(d);
    if (a.B == 0 || a.L == 0) return ok();
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(W, "W"));
    TRY(need_ptr(Y, "Y"));
    if (bias && !aligned16(bias)) return fail(HASTE_ERR_INVALID, "bias is not 16-byte aligned");
    if (!fwd_kernel_exists(a)) return fail(HASTE_ERR_UNSUPPORTED, "no forward kernel for this shape");
    return hip_status(fwd_any(a, X, idx, W, bias, Y, as_stream(stream)), "haste_fwd");
}

int haste_bwd_w(const haste_desc_t *d, const void *X, const int32_t *idx, const void *dY, float *dW, float *dbias,
                int beta, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    if (beta != 0 && beta != 1) return fail(HASTE_ERR_INVALID, "beta must be 0 or 1");
    const haste::TailArgs a = targs(d);
    hipStream_t s = as_stream(stream);
    if (a.L == 0) return ok();
    TRY(need_ptr(dW, "dW"));
    if (dbias && !aligned16(dbias)) return fail(HASTE_ERR_INVALID, "dbias is not 16-byte aligned");
    if (a.B == 0) {  // empty batch: the sum is zero
        if (beta) return ok();
        hipError_t e = haste::fill_f32(dW, a.L * a.F_in, 0.0f, s);
        if (e == hipSuccess && dbias) e = haste::fill_f32(dbias, a.L, 0.0f, s);
        return hip_status(e, "haste_bwd_w");
    }
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(dY, "dY"));
    if (bwd_w_uses_xt(a)) {
        const size_t need = haste::bwd_w_mfma_ws(a);
        if (!ws || ws_bytes < need)
            return fail(HASTE_ERR_WORKSPACE, "haste_bwd_w needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
        TRY(need_ptr(ws, "ws"));
        return hip_status(bwd_w_any(a, X, idx, dY, dW, dbias, beta, ws, s), "haste_bwd_w");
    }
    if (!haste::valu_supported(a)) return fail(HASTE_ERR_UNSUPPORTED, "no backward-weight kernel for this shape");
    return hip_status(haste::bwd_w_valu(a, X, idx, dY, dW, dbias, beta, s), "haste_bwd_w");
}

int haste_bwd_x(const haste_desc_t *d, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    if (beta != 0 && beta != 1) return fail(HASTE_ERR_INVALID, "beta must be 0 or 1");
    const haste::TailArgs a = targs(d);
    hipStream_t s = as_stream(stream);
    if (a.B == 0) return ok();
    TRY(need_ptr(dX, "dX"));
    if (a.L == 0) {  // no labels: nothing flows back
        if (beta) return ok();
        return hip_status(haste::fill_f32(dX, a.B * a.F_s, 0.0f, s), "haste_bwd_x");
    }
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(W, "W"));
    TRY(need_ptr(dY, "dY"));
    if (!haste::bwd_x_dn_supported(a) && !haste::bwd_x_sg_supported(a) && !haste::bwd_x_mfma_supported(a) &&
        !haste::valu_supported(a))
        return fail(HASTE_ERR_UNSUPPORTED, "no backward-feature kernel for this shape");
    const size_t need = bwd_x_ws(a);
    if (!ws || ws_bytes < need)
        return fail(HASTE_ERR_WORKSPACE, "haste_bwd_x needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
    TRY(need_ptr(ws, "ws"));
    if (haste::bwd_x_dn_supported(a)) return hip_status(haste::bwd_x_dn(a, idx, W, dY, dX, beta, ws, s), "haste_bwd_x");
    if (haste::bwd_x_sg_supported(a)) return hip_status(haste::bwd_x_sg(a, idx, W, dY, dX, beta, ws, s), "haste_bwd_x");
    if (haste::bwd_x_mfma_supported(a)) return hip_status(haste::bwd_x_mfma(a, idx, W, dY, dX, beta, ws, s), "haste_bwd_x");
    return hip_status(haste::bwd_x_valu(a, idx, W, dY, dX, beta, ws, s), "haste_bwd_x");
}

int haste_tail_step(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias,
                    const int32_t *pos, int32_t P, void *dY, float *dW, float *dbias, int beta, float *dX, int beta_dx,
                    void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    if (beta != 0 && beta != 1) return fail(HASTE_ERR_INVALID, "beta must be 0 or 1");
    if (beta_dx != 0 && beta_dx != 1) return fail(HASTE_ERR_INVALID, "beta_dx must be 0 or 1");
    if (P < 0) return fail(HASTE_ERR_INVALID, "P must be >= 0");
    const haste::TailArgs a = targs(d);
    const size_t need = haste_workspace_bytes(d, HASTE_OP_TAIL_STEP);
    if (need && (!ws || ws_bytes < need))
        return fail(HASTE_ERR_WORKSPACE, "haste_tail_step needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
    const size_t xoff = (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_BWD_X), 256);
    if (a.L > 0 && a.B > 0 && dW && dX && haste::tail_step_fused(a, P) && ws_bytes >= haste::tail_step_ws(a, P)) {
        TRY(need_ptr(X, "X"));
        TRY(need_ptr(idx, "idx"));
        TRY(need_ptr(W, "W"));
        TRY(need_ptr(dY, "dY"));
        TRY(need_ptr(dW, "dW"));
        TRY(need_ptr(dX, "dX"));
        TRY(need_ptr(ws, "ws"));
        if (P > 0) TRY(need_ptr(pos, "pos"));
        if (bias && !aligned16(bias)) return fail(HASTE_ERR_INVALID, "bias is not 16-byte aligned");
        if (dbias && !aligned16(dbias)) return fail(HASTE_ERR_INVALID, "dbias is not 16-byte aligned");
        if (a.B * haste::cdiv(a.L, 2048) >= ((int64_t)1 << 31))
            return fail(HASTE_ERR_UNSUPPORTED, "B * L too large for the gradient kernel's grid");
        return hip_status(haste::tail_step_mfma(a, X, idx, W, bias, P > 0 ? pos : nullptr, P, dY, dW, dbias, beta, dX,
                                                beta_dx, ws, as_stream(stream)),
                          "haste_tail_step");
    }
    // composed: the two calls, each in its own part of the workspace
    TRY(haste_fwd_bce(d, X, idx, W, bias, pos, P, dY, dW, dbias, beta, ws ? (char *)ws + xoff : nullptr,
                      ws ? ws_bytes - xoff : 0, stream));
    if (!dX) return ok();
    return haste_bwd_x(d, idx, W, dY, dX, beta_dx, ws, xoff, stream);
}

int haste_fwd_bce(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias,
                  const int32_t *pos, int32_t P, void *dY, float *dW, float *dbias, int beta, void *ws, size_t ws_bytes,
                  void *stream) {
    TRY(check_desc(d));
    if (beta != 0 && beta != 1) return fail(HASTE_ERR_INVALID, "beta must be 0 or 1");
    if (P < 0) return fail(HASTE_ERR_INVALID, "P must be >= 0");
    if (dbias && !dW) return fail(HASTE_ERR_INVALID, "dbias needs dW (both come from the backward-weight product)");
    const haste::TailArgs a = targs(d);
    hipStream_t s = as_stream(stream);
    if (a.L == 0) return ok();
    if (dW) TRY(need_ptr(dW, "dW"));
    if (dbias && !aligned16(dbias)) return fail(HASTE_ERR_INVALID, "dbias is not 16-byte aligned");
    if (a.B == 0) {  // no rows: dY is empty and the sums are zero
        if (!dW || beta) return ok();
        hipError_t e = haste::fill_f32(dW, a.L * a.F_in, 0.0f, s);
        if (e == hipSuccess && dbias) e = haste::fill_f32(dbias, a.L, 0.0f, s);
        return hip_status(e, "haste_fwd_bce");
    }
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(W, "W"));
    TRY(need_ptr(dY, "dY"));
    if (P > 0) TRY(need_ptr(pos, "pos"));
    if (bias && !aligned16(bias)) return fail(HASTE_ERR_INVALID, "bias is not 16-byte aligned");
    if (a.B * haste::cdiv(a.L, 2048) >= ((int64_t)1 << 31))
        return fail(HASTE_ERR_UNSUPPORTED, "B * L too large for the gradient kernel's grid");
    const bool bw_mfma = bwd_w_uses_xt(a);
    const size_t need = bw_mfma ? haste::bwd_w_mfma_ws(a) : 0;
    if (need && (!ws || ws_bytes < need))
        return fail(HASTE_ERR_WORKSPACE, "haste_fwd_bce needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
    if (need) TRY(need_ptr(ws, "ws"));
    // fused where the shape allows it and the workspace also holds the bucketed positives of long
    // rows (the query's size does for up to kFusedPosWs per row)
    if (haste::fwd_bce_mfma_supported(a, P) && ws_bytes >= haste::fwd_bce_mfma_ws(a, P))
        return hip_status(haste::fwd_bce_mfma(a, X, idx, W, bias, P > 0 ? pos : nullptr, P, dY, dW, dbias, beta, ws, s),
                          "haste_fwd_bce");
    // small groups: the forward stores the gradient of its rounded logits (bit for bit what the
    // separate gradient pass computes), given each row's positives sorted after the X^T copy
    const size_t spos_at = (size_t)haste::round_up((int64_t)need, 256);
    hipError_t e = hipSuccess;
    if (fwd_small_bce(a, P) && ws && ws_bytes >= spos_at + (size_t)a.B * P * 4) {
        int32_t *spos = reinterpret_cast<int32_t *>(static_cast<char *>(ws) + spos_at);
        if (P > 0) e = haste::sort_positives(a.B, a.L, pos, P, spos, s);
        // with no positives the kernels never read the list, but need a non-null one to form the gradient
        if (e == hipSuccess) e = fwd_small(a, X, idx, W, bias, dY, s, P > 0 ? spos : reinterpret_cast<int32_t *>(dY), P);
    } else {
        // composed: logits into dY, the gradient in place
        if (!fwd_kernel_exists(a)) return fail(HASTE_ERR_UNSUPPORTED, "no forward kernel for this shape");
        e = fwd_any(a, X, idx, W, bias, dY, s);
        if (e == hipSuccess) e = haste::bce_grad(a.B, a.L, a.dtype, dY, P > 0 ? pos : nullptr, P, dY, s);
    }
    if (e == hipSuccess && dW)
        e = bwd_w_any(a, X, idx, dY, dW, dbias, beta, ws, s);
    return hip_status(e, "haste_fwd_bce");
}

static int check_sgd(const haste_sgd_t *o) {
    if (!o) return fail(HASTE_ERR_INVALID, "opt is NULL");
    if (o->reserved != 0) return fail(HASTE_ERR_INVALID, "opt.reserved must be 0");
    if (!(o->momentum >= 0.0f && o->momentum < 1.0f)) return fail(HASTE_ERR_INVALID, "momentum must be in [0, 1)");
    if (!(o->lr == o->lr) || !(o->weight_decay == o->weight_decay))
        return fail(HASTE_ERR_INVALID, "lr and weight_decay must be numbers");
    return HASTE_OK;
}

int haste_sgd_momentum(int64_t n, int32_t dtype, const void *W, const float *grad, float *m, const haste_sgd_t *opt,
                       void *W_next, void *stream) {
    if (dtype != HASTE_DTYPE_F32 && dtype != HASTE_DTYPE_BF16) return fail(HASTE_ERR_INVALID, "bad dtype %d", dtype);
    if (n < 0) return fail(HASTE_ERR_INVALID, "n must be >= 0");
    TRY(check_sgd(opt));
    if (n == 0) return ok();
    TRY(need_ptr(W, "W"));
    if (grad) TRY(need_ptr(grad, "grad"));
    TRY(need_ptr(m, "m"));
    TRY(need_ptr(W_next, "W_next"));
    if (haste::cdiv(n, 256) >= ((int64_t)1 << 31)) return fail(HASTE_ERR_UNSUPPORTED, "n too large");
    return hip_status(haste::sgd_momentum(n, dtype, W, grad, m, *opt, W_next, as_stream(stream)), "haste_sgd_momentum");
}

int haste_fwd_bce_sgd(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias,
                      const int32_t *pos, int32_t P, void *dY, float *dbias, const haste_sgd_t *opt, float *m,
                      void *W_next, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    TRY(check_sgd(opt));
    if (P < 0) return fail(HASTE_ERR_INVALID, "P must be >= 0");
    const haste::TailArgs a = targs(d);
    hipStream_t s = as_stream(stream);
    if (a.L == 0) return ok();
    TRY(need_ptr(W, "W"));
    TRY(need_ptr(m, "m"));
    TRY(need_ptr(W_next, "W_next"));
    if (dbias && !aligned16(dbias)) return fail(HASTE_ERR_INVALID, "dbias is not 16-byte aligned");
    const int64_t wbytes = a.L * a.F_in * (a.dtype == HASTE_DTYPE_BF16 ? 2 : 4);
    {
        const char *w0 = static_cast<const char *>(W), *n0 = static_cast<const char *>(W_next);
        if (n0 < w0 + wbytes && w0 < n0 + wbytes)
            return fail(HASTE_ERR_INVALID, "W_next overlaps W (the backward-feature call still reads W)");
    }
    if (a.B > 0) {
        TRY(need_ptr(X, "X"));
        TRY(need_ptr(idx, "idx"));
        TRY(need_ptr(dY, "dY"));
        if (P > 0) TRY(need_ptr(pos, "pos"));
    }
    if (bias && !aligned16(bias)) return fail(HASTE_ERR_INVALID, "bias is not 16-byte aligned");
    if (a.B * haste::cdiv(a.L, 2048) >= ((int64_t)1 << 31))
        return fail(HASTE_ERR_UNSUPPORTED, "B * L too large for the gradient kernel's grid");
    // the fused kernel's shapes need the X^T copy (and the bucketed positives of rows of more than
    // 64); others keep dW in the workspace too
    const bool fused_shape = haste::fwd_bce_mfma_supported(a, P);
    // composed: haste_fwd_bce's region (the X^T copy and sorted positives), then dW
    const size_t xws = (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_FWD_BCE), 256);
    const size_t need = fused_shape ? haste::fwd_bce_mfma_ws(a, P) : xws + (size_t)haste::round_up(a.L * a.F_in * 4, 256);
    if (a.B == 0) {  // no rows: a zero gradient, the step still decays the velocity and the weights
        if (dbias) TRY(hip_status(haste::fill_f32(dbias, a.L, 0.0f, s), "haste_fwd_bce_sgd"));
        return hip_status(haste::sgd_momentum(a.L * a.F_in, a.dtype, W, nullptr, m, *opt, W_next, s),
                          "haste_fwd_bce_sgd");
    }
    if (need && (!ws || ws_bytes < need))
        return fail(HASTE_ERR_WORKSPACE, "haste_fwd_bce_sgd needs %zu workspace bytes for rows of %d positives, got %zu",
                    need, (int)P, ws ? ws_bytes : 0);
    if (need) TRY(need_ptr(ws, "ws"));
    if (fused_shape) {
        return hip_status(haste::fwd_bce_sgd_mfma(a, X, idx, W, bias, P > 0 ? pos : nullptr, P, dY, dbias, *opt, m,
                                                  W_next, ws, s),
                          "haste_fwd_bce_sgd");
    }
    // composed: dW into the workspace after the X^T copy, then the momentum step
    float *dW = reinterpret_cast<float *>(static_cast<char *>(ws) + xws);
    const int rc = haste_fwd_bce(d, X, idx, W, bias, pos, P, dY, dW, dbias, 0, ws, xws, stream);
    if (rc != HASTE_OK) return rc;
    return hip_status(haste::sgd_momentum(a.L * a.F_in, a.dtype, W, dW, m, *opt, W_next, s), "haste_fwd_bce_sgd");
}

int haste_rewire(const haste_desc_t *d, int32_t *idx, void *W, float *m, double rho, int32_t init_random,
                 uint64_t seed, int64_t *n_pruned, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    if (!(rho >= 0.0 && rho < 1.0)) return fail(HASTE_ERR_INVALID, "rho must be in [0, 1)");
    if (init_random != 0 && init_random != 1) return fail(HASTE_ERR_INVALID, "init_random must be 0 or 1");
    const haste::TailArgs a = targs(d);
    if (!haste::rewire_supported(a)) return fail(HASTE_ERR_UNSUPPORTED, "rewiring takes at most 256 slots per group and 1024 features");
    const int64_t K = a.L / a.G;
    const int64_t npr = (int64_t)floor((double)K * (double)a.F_in * rho);
    if (n_pruned) *n_pruned = npr;
    if (npr == 0) return ok();
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(W, "W"));
    if (m) TRY(need_ptr(m, "m"));
    const size_t need = haste::rewire_ws(a);
    if (!ws || ws_bytes < need)
        return fail(HASTE_ERR_WORKSPACE, "haste_rewire needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
    TRY(need_ptr(ws, "ws"));
    if (K * a.F_in >= ((int64_t)1 << 31) / 4) return fail(HASTE_ERR_UNSUPPORTED, "K * F_in too large");
    return hip_status(haste::rewire(a, idx, W, m, npr, init_random, seed, ws, as_stream(stream)), "haste_rewire");
}

static int check_group(int64_t N, int64_t D, const haste_group_opts_t *o) {
    if (!o) return fail(HASTE_ERR_INVALID, "opts is NULL");
    if (o->beta < 1 || o->iters < 0) return fail(HASTE_ERR_INVALID, "beta must be >= 1 and iters >= 0");
    if (!haste::group_supported(N, D, o->G, o->beta))
        return fail(HASTE_ERR_UNSUPPORTED, "grouping needs 0 < N < 2^24, D a multiple of 16 up to 1024, 1 <= G <= 256, "
                                           "N D < 2^31 and 4 C D < 2^31");
    return HASTE_OK;
}

size_t haste_group_workspace_bytes(int64_t N, int64_t D, const haste_group_opts_t *o) {
    if (check_group(N, D, o) != HASTE_OK) return 0;
    return haste::group_ws(N, D, o->G, o->beta);
}

int haste_group_labels(int64_t N, int64_t D, const int8_t *E, const haste_group_opts_t *o, int32_t *order,
                       int32_t *gsize, int64_t *n_groups, int32_t *cluster, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_group(N, D, o));
    TRY(need_ptr(E, "E"));
    TRY(need_ptr(order, "order"));
    TRY(need_ptr(gsize, "gsize"));
    if (!n_groups) return fail(HASTE_ERR_INVALID, "n_groups is NULL");
    if (cluster) TRY(need_ptr(cluster, "cluster"));
    const size_t need = haste::group_ws(N, D, o->G, o->beta);
    if (!ws || ws_bytes < need)
        return fail(HASTE_ERR_WORKSPACE, "haste_group_labels needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
    TRY(need_ptr(ws, "ws"));
    return hip_status(haste::group_labels(N, D, E, o->G, o->beta, o->iters, o->seed, order, gsize, n_groups, cluster,
                                          ws, as_stream(stream)),
                      "haste_group_labels");
}

int haste_bce_grad(int64_t B, int64_t N, int32_t dtype, const void *Y, const int32_t *pos, int32_t P, void *dY,
                   void *stream) {
    if (dtype != HASTE_DTYPE_F32 && dtype != HASTE_DTYPE_BF16) return fail(HASTE_ERR_INVALID, "bad dtype %d", dtype);
    if (B < 0 || N < 0 || P < 0) return fail(HASTE_ERR_INVALID, "B, N and P must be >= 0");
    if (B == 0 || N == 0) return ok();
    TRY(need_ptr(Y, "Y"));
    TRY(need_ptr(dY, "dY"));
    if (P > 0) TRY(need_ptr(pos, "pos"));
    if (B * haste::cdiv(N, 2048) >= ((int64_t)1 << 31)) return fail(HASTE_ERR_UNSUPPORTED, "B * N too large");
    return hip_status(haste::bce_grad(B, N, dtype, Y, P > 0 ? pos : nullptr, P, dY, as_stream(stream)),
                      "haste_bce_grad");
}

static int check_head(int64_t B, int64_t F_s, int64_t H, int32_t dtype) {
    if (dtype != HASTE_DTYPE_F32 && dtype != HASTE_DTYPE_BF16) return fail(HASTE_ERR_INVALID, "bad dtype %d", dtype);
    if (B < 0 || F_s <= 0 || H < 0) return fail(HASTE_ERR_INVALID, "head needs B >= 0, F_s > 0, H >= 0");
    if (B > INT32_MAX || F_s > INT32_MAX) return fail(HASTE_ERR_INVALID, "B and F_s must be < 2^31");
    return HASTE_OK;
}

int haste_head_fwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *W_head,
                   const float *bias_h, void *Y_h, void *stream) {
    TRY(check_head(B, F_s, H, dtype));
    if (B == 0 || H == 0) return ok();
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(W_head, "W_head"));
    TRY(need_ptr(Y_h, "Y_h"));
    if (bias_h && !aligned16(bias_h)) return fail(HASTE_ERR_INVALID, "bias_h is not 16-byte aligned");
    return hip_status(haste::head_fwd(B, F_s, H, dtype, X, W_head, bias_h, Y_h, as_stream(stream)), "haste_head_fwd");
}

int haste_head_fwd_bce(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *W_head,
                       const float *bias_h, const int32_t *pos, int32_t P, void *dY_h, void *stream) {
    TRY(check_head(B, F_s, H, dtype));
    if (P < 0) return fail(HASTE_ERR_INVALID, "P must be >= 0");
    if (B == 0 || H == 0) return ok();
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(W_head, "W_head"));
    TRY(need_ptr(dY_h, "dY_h"));
    if (P > 0) TRY(need_ptr(pos, "pos"));
    if (bias_h && !aligned16(bias_h)) return fail(HASTE_ERR_INVALID, "bias_h is not 16-byte aligned");
    if (B * haste::cdiv(H, 2048) >= ((int64_t)1 << 31)) return fail(HASTE_ERR_UNSUPPORTED, "B * H too large");
    return hip_status(haste::head_fwd_bce(B, F_s, H, dtype, X, W_head, bias_h, P > 0 ? pos : nullptr, P, dY_h,
                                          as_stream(stream)),
                      "haste_head_fwd_bce");
}

int haste_head_bwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *W_head,
                   const void *dY_h, float *dW_h, float *dX, int beta_dx, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_head(B, F_s, H, dtype));
    if (beta_dx != 0 && beta_dx != 1) return fail(HASTE_ERR_INVALID, "beta_dx must be 0 or 1");
    hipStream_t s = as_stream(stream);
    if (dW_h) TRY(need_ptr(dW_h, "dW_h"));
    if (dX) TRY(need_ptr(dX, "dX"));
    if (H == 0) {
        if (dX && !beta_dx) return hip_status(haste::fill_f32(dX, B * F_s, 0.0f, s), "haste_head_bwd");
        return ok();
    }
    if (B == 0) {
        if (dW_h) return hip_status(haste::fill_f32(dW_h, H * F_s, 0.0f, s), "haste_head_bwd");
        return ok();
    }
    TRY(need_ptr(dY_h, "dY_h"));
    if (dW_h) TRY(need_ptr(X, "X"));
    if (dX) {
        TRY(need_ptr(W_head, "W_head"));
        const size_t need = haste::head_ws(B, F_s, H, dtype);
        if (!ws || ws_bytes < need)
            return fail(HASTE_ERR_WORKSPACE, "haste_head_bwd needs %zu workspace bytes, got %zu", need, ws ? ws_bytes : 0);
        TRY(need_ptr(ws, "ws"));
    }
    return hip_status(haste::head_bwd(B, F_s, H, dtype, X, W_head, dY_h, dW_h, dX, beta_dx, ws, s), "haste_head_bwd");
}

int haste_validate_idx(const haste_desc_t *d, const int32_t *idx, int32_t *n_bad_rows, void *stream) {
    TRY(check_desc(d));
    if (!n_bad_rows) return fail(HASTE_ERR_INVALID, "n_bad_rows is NULL");
    const int64_t rows = d->L / d->G;
    if (rows > 0) TRY(need_ptr(idx, "idx"));
    return hip_status(haste::validate_idx(idx, rows, d->F_in, d->F_s, n_bad_rows, as_stream(stream)),
                      "haste_validate_idx");
}

int haste_debug_gather(const haste_desc_t *d, const void *X, const int32_t *idx, int64_t k0, int64_t nk, void *out,
                       void *stream) {
    TRY(check_desc(d));
    const int64_t K = d->L / d->G;
    if (k0 < 0 || nk < 0 || k0 + nk > K) return fail(HASTE_ERR_INVALID, "group range [k0, k0+nk) outside [0, L/G)");
    if (nk == 0 || d->B == 0) return ok();
    TRY(need_ptr(X, "X"));
    TRY(need_ptr(idx, "idx"));
    TRY(need_ptr(out, "out"));
    return hip_status(haste::debug_gather(X, d->dtype, idx, d->B, d->F_s, d->F_in, k0, nk, out, as_stream(stream)),
                      "haste_debug_gather");
}

}  // extern "C"

int haste_tail_step_sgd(const haste_desc_t *d, const void *X, const int32_t *idx, const void *W, const float *bias,
                        const int32_t *pos, int32_t P, void *dY, float *dbias, const haste_sgd_t *opt, float *m,
                        void *W_next, float *dX, int beta_dx, void *ws, size_t ws_bytes, void *stream) {
    TRY(check_desc(d));
    TRY(check_sgd(opt));
    if (beta_dx != 0 && beta_dx != 1) return fail(HASTE_ERR_INVALID, "beta_dx must be 0 or 1");
    if (P < 0) return fail(HASTE_ERR_INVALID, "P must be >= 0");
    const haste::TailArgs a = targs(d);
    const size_t need = haste_workspace_bytes(d, HASTE_OP_TAIL_STEP_SGD);
    if (need && (!ws || ws_bytes < need))
        return fail(HASTE_ERR_WORKSPACE, "haste_tail_step_sgd needs %zu workspace bytes, got %zu", need,
                    ws ? ws_bytes : 0);
    const size_t xoff = (size_t)haste::round_up((int64_t)haste_workspace_bytes(d, HASTE_OP_BWD_X), 256);
    if (a.L > 0 && a.B > 0 && dX && haste::tail_step_fused(a, P) && ws_bytes >= haste::tail_step_ws(a, P)) {
        TRY(need_ptr(X, "X"));
        TRY(need_ptr(idx, "idx"));
        TRY(need_ptr(W, "W"));
        TRY(need_ptr(dY, "dY"));
        TRY(need_ptr(m, "m"));
        TRY(need_ptr(W_next, "W_next"));
        TRY(need_ptr(dX, "dX"));
        TRY(need_ptr(ws, "ws"));
        if (P > 0) TRY(need_ptr(pos, "pos"));
        if (bias && !aligned16(bias)) return fail(HASTE_ERR_INVALID, "bias is not 16-byte aligned");
        if (dbias && !aligned16(dbias)) return fail(HASTE_ERR_INVALID, "dbias is not 16-byte aligned");
        const uintptr_t wb = (uintptr_t)W, nb = (uintptr_t)W_next, len = (uintptr_t)(a.L * a.F_in * 2);
        if (wb < nb + len && nb < wb + len)
            return fail(HASTE_ERR_INVALID, "W_next overlaps W (the backward-feature pass still reads W)");
        if (a.B * haste::cdiv(a.L, 2048) >= ((int64_t)1 << 31))
            return fail(HASTE_ERR_UNSUPPORTED, "B * L too large for the gradient kernel's grid");
        return hip_status(haste::tail_step_sgd_mfma(a, X, idx, W, bias, P > 0 ? pos : nullptr, P, dY, dbias, *opt, m,
                                                    W_next, dX, beta_dx, ws, ws_bytes - xoff, as_stream(stream)),
                          "haste_tail_step_sgd");
    }
    // composed: the two calls, each in its own part of the workspace
    TRY(haste_fwd_bce_sgd(d, X, idx, W, bias, pos, P, dY, dbias, opt, m, W_next, ws ? (char *)ws + xoff : nullptr,
                          ws ? ws_bytes - xoff : 0, stream));
    if (!dX) return ok();
    return haste_bwd_x(d, idx, W, dY, dX, beta_dx, ws, xoff, stream);
}
