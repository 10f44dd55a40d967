// Group-shared fixed fan-in tail on the vector ALUs (fp32 FMA), for any G including G = 1.
//
// Used for fp32 layers (the paper's logit definition, Section 3.1, evaluated with true fp32
// products: gfx950 has no reduced-precision fp32 matrix path to fall into) and as the standard
// per-label fixed fan-in comparator (G = 1, Section 3.1 / Fig. 2(c)): every label gathers its own
// F_in features, so there is no shared tile and the work is thin dot products.
//
// A batch tile of TB rows of X is kept transposed in LDS as fp32 (xs[f][b], row stride TB+4
// floats so 16-byte reads stay aligned).  One thread owns one label.
#include "common.hpp"

namespace {

constexpr int TB = 16;        // batch rows per tile
constexpr int XS = TB + 4;    // LDS row stride (floats) of the transposed tile

template <typename T>
__device__ __forceinline__ void load_slab(float *xs, const T *__restrict__ X, int b0, int B, int F_s) {
    for (int e = threadIdx.x; e < TB * F_s; e += blockDim.x) {
        const int r = e / F_s, f = e - r * F_s;
        const int b = b0 + r;
        xs[f * XS + r] = (b < B) ? load_f32(X, (int64_t)b * F_s + f) : 0.0f;
    }
}

// Y[b, l] = bias[l] + sum_t X[b, idx[l/G, t]] * W[l, t]
template <typename T>
__global__ __launch_bounds__(256) void k_fwd_valu(const T *__restrict__ X, const int32_t *__restrict__ idx,
                                                  const T *__restrict__ W, const float *__restrict__ bias,
                                                  T *__restrict__ Y, int B, int F_s, int64_t L, int G, int F_in,
                                                  int64_t nlt) {
    extern __shared__ __align__(16) float xs[];
    const int b0 = blockIdx.y * TB;
    load_slab(xs, X, b0, B, F_s);
    __syncthreads();
    for (int64_t lt = blockIdx.x; lt < nlt; lt += gridDim.x) {
        const int64_t l = lt * blockDim.x + threadIdx.x;
        if (l >= L) continue;
        const int64_t g = l / G;
        float acc[TB];
#pragma unroll
        for (int b = 0; b < TB; ++b) acc[b] = 0.0f;
        const int32_t *ip = idx + g * F_in;
        const T *wp = W + l * F_in;
        for (int t = 0; t < F_in; ++t) {
            const int f = ip[t];
            const float w = load_f32(wp, t);
            const float4 *xr = reinterpret_cast<const float4 *>(xs + f * XS);
#pragma unroll
            for (int q = 0; q < TB / 4; ++q) {
                const float4 x = xr[q];
                acc[4 * q + 0] = fmaf(x.x, w, acc[4 * q + 0]);
                acc[4 * q + 1] = fmaf(x.y, w, acc[4 * q + 1]);
                acc[4 * q + 2] = fmaf(x.z, w, acc[4 * q + 2]);
                acc[4 * q + 3] = fmaf(x.w, w, acc[4 * q + 3]);
            }
        }
        const float bv = bias ? bias[l] : 0.0f;
#pragma unroll
        for (int b = 0; b < TB; ++b)
            if (b0 + b < B) store_out(Y, (int64_t)(b0 + b) * L + l, acc[b] + bv);
    }
}

// dW[l, t] = beta*dW + sum_b dY[b, l] * X[b, idx[l/G, t]];  dbias[l] = beta*dbias + sum_b dY[b, l]
template <typename T>
__global__ __launch_bounds__(256) void k_bwd_w_valu(const T *__restrict__ X, const int32_t *__restrict__ idx,
                                                    const T *__restrict__ dY, float *__restrict__ dW,
                                                    float *__restrict__ dbias, int beta, int B, int F_s, int64_t L,
                                                    int G, int F_in) {
    extern __shared__ __align__(16) float xs[];
    const int64_t l = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool valid = l < L;
    const int64_t g = valid ? l / G : 0;
    constexpr int TC = 32;  // support slots per pass (register accumulators)
    for (int tc = 0; tc < F_in; tc += TC) {
        float acc[TC];
#pragma unroll
        for (int t = 0; t < TC; ++t) acc[t] = 0.0f;
        float db = 0.0f;
        const int nt = F_in - tc < TC ? F_in - tc : TC;
        // the pass's supports, once for the whole batch (lanes sit a label's support apart)
        int fs[TC];
#pragma unroll
        for (int t = 0; t < TC; ++t) fs[t] = valid && t < nt ? idx[g * F_in + tc + t] : 0;
        for (int b0 = 0; b0 < B; b0 += TB) {
            __syncthreads();
            load_slab(xs, X, b0, B, F_s);
            __syncthreads();
            if (valid) {
                float dy[TB];
#pragma unroll
                for (int b = 0; b < TB; ++b) dy[b] = (b0 + b < B) ? load_f32(dY, (int64_t)(b0 + b) * L + l) : 0.0f;
                if (tc == 0) {
#pragma unroll
                    for (int b = 0; b < TB; ++b) db += dy[b];
                }
#pragma unroll
                for (int t = 0; t < TC; ++t) {
                    if (t < nt) {
                        const float4 *xr = reinterpret_cast<const float4 *>(xs + fs[t] * XS);
                        float s = 0.0f;
#pragma unroll
                        for (int q = 0; q < TB / 4; ++q) {
                            const float4 x = xr[q];
                            s = fmaf(x.x, dy[4 * q + 0], s);
                            s = fmaf(x.y, dy[4 * q + 1], s);
                            s = fmaf(x.z, dy[4 * q + 2], s);
                            s = fmaf(x.w, dy[4 * q + 3], s);
                        }
                        acc[t] += s;
                    }
                }
            }
        }
        if (valid) {
#pragma unroll
            for (int t = 0; t < TC; ++t)
                if (t < nt) {
                    float *p = dW + l * F_in + tc + t;
                    *p = beta ? *p + acc[t] : acc[t];
                }
            if (tc == 0 && dbias) dbias[l] = beta ? dbias[l] + db : db;
        }
    }
}

// Partial dX^T over one label segment and one 32-row batch tile: part[seg][f][b0 + b].
//
// The accumulator dX^T[F_s][32] (fp32, rows of kOwnAS floats) lives in LDS.  Wave w owns rows
// 4w .. 4w + 3 of the tile, so no two waves touch the same cell, and within a wave the lanes run
// over one label's support slots, whose rows are distinct: every update is a plain float4
// read-add-write in the wave's program order (LDS operations of a wave execute in order), with
// no atomics, and dX is bit-reproducible.  The supports and weights of a block of LB labels are
// staged in LDS once per workgroup (LB F_in = 4096), and the wave's dY values for the block are
// read with one coalesced load per row and handed to the lanes label by label.
constexpr int kOwnWaves = 8;
constexpr int kOwnAS = 36;        // accumulator row stride (floats): 32 rows + 4 pad

template <typename T>
__global__ __launch_bounds__(kOwnWaves * 64) void k_bwd_x_valu(const int32_t *__restrict__ idx,
                                                                const T *__restrict__ W, const T *__restrict__ dY,
                                                                float *__restrict__ part, int B, int Bp, int F_s,
                                                                int64_t L, int G, int F_in, int64_t lps) {
    extern __shared__ __align__(16) float accs[];   // [F_s][kOwnAS], then the staged block
    const int LB = 4096 / F_in;                      // labels per staged block
    int2 *sfw = reinterpret_cast<int2 *>(accs + F_s * kOwnAS);   // [LB][F_in] (support, weight bits)
    const int64_t seg = blockIdx.x;
    const int b0 = blockIdx.y * 32;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int nthr = kOwnWaves * 64;
    for (int e = tid; e < F_s * kOwnAS; e += nthr) accs[e] = 0.0f;
    const int64_t l_begin = seg * lps;
    const int64_t l_end = l_begin + lps < L ? l_begin + lps : L;
    float *accw = accs + 4 * w;                      // this wave's 4 columns of a row
    for (int64_t lb = l_begin; lb < l_end; lb += LB) {
        const int nl = l_end - lb < LB ? (int)(l_end - lb) : LB;
        __syncthreads();                             // the previous block is no longer read
        for (int e = tid; e < nl * F_in; e += nthr) {
            const int j = e / F_in, t = e - j * F_in;
            const int64_t l = lb + j;
            sfw[e] = make_int2(idx[(l / G) * F_in + t], __float_as_int(load_f32(W, l * F_in + t)));
        }
        __syncthreads();
        // dY of this wave's 4 rows for labels lb + 64c + lane (c < LB / 64 chunks of the block)
        for (int c = 0; c * 64 < nl; ++c) {
            float dyr[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int b = b0 + 4 * w + i;
                const int j = 64 * c + lane;
                dyr[i] = (b < B && j < nl) ? load_f32(dY, (int64_t)b * L + lb + j) : 0.0f;
            }
            const int ncl = nl - 64 * c < 64 ? nl - 64 * c : 64;
            for (int jj = 0; jj < ncl; ++jj) {
                const int j = 64 * c + jj;
                float dy[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) dy[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dyr[i]), jj));
                for (int t = lane; t < F_in; t += 64) {
                    const int2 fw = sfw[j * F_in + t];   // one 8-byte read: the slot's feature and weight
                    const int f = fw.x;
                    const float wv = __int_as_float(fw.y);
                    float4 *p = reinterpret_cast<float4 *>(accw + f * kOwnAS);
                    float4 v = *p;
                    v.x = fmaf(dy[0], wv, v.x);
                    v.y = fmaf(dy[1], wv, v.y);
                    v.z = fmaf(dy[2], wv, v.z);
                    v.w = fmaf(dy[3], wv, v.w);
                    *p = v;
                }
            }
        }
    }
    __syncthreads();
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    for (int e = tid; e < F_s * 32; e += nthr) {
        const int f = e >> 5, b = e & 31;
        pp[(size_t)f * Bp + b] = accs[f * kOwnAS + b];
    }
}

size_t bwd_x_valu_lds(const haste::TailArgs &a) {
    return (size_t)a.F_s * kOwnAS * 4 + 2 * 4096 * 4;
}

int64_t bwd_x_valu_segments(const haste::TailArgs &a) {
    const int64_t nbt = haste::cdiv(a.B, 32);
    int64_t S = 512 / (nbt < 1 ? 1 : nbt);
    const int64_t maxS = haste::cdiv(a.L, 64);
    if (S > maxS) S = maxS;
    return S < 1 ? 1 : S;
}

}  // namespace

namespace haste {

bool valu_supported(const TailArgs &a) {
    return a.F_s <= kMaxFs && (size_t)a.F_s * XS * 4 <= 150 * 1024 && bwd_x_valu_lds(a) <= 160 * 1024;
}

hipError_t fwd_valu(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s) {
    const int64_t nbt = cdiv(a.B, TB);
    const int64_t nlt = cdiv(a.L, 256);
    int64_t gx = 2048 / nbt;
    if (gx < 1) gx = 1;
    if (gx > nlt) gx = nlt;
    const size_t lds = (size_t)a.F_s * XS * 4;
    const dim3 grid((unsigned)gx, (unsigned)nbt);
    if (a.dtype == HASTE_DTYPE_F32) {
        hipFuncSetAttribute((const void *)k_fwd_valu<float>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_fwd_valu<float>, grid, dim3(256), lds, s, (const float *)X, idx, (const float *)W, bias,
                           (float *)Y, (int)a.B, (int)a.F_s, a.L, (int)a.G, (int)a.F_in, nlt);
    } else {
        hipFuncSetAttribute((const void *)k_fwd_valu<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_fwd_valu<bf16_t>, grid, dim3(256), lds, s, (const bf16_t *)X, idx, (const bf16_t *)W,
                           bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, a.L, (int)a.G, (int)a.F_in, nlt);
    }
    return hipGetLastError();
}

hipError_t bwd_w_valu(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, hipStream_t s) {
    const size_t lds = (size_t)a.F_s * XS * 4;
    const dim3 grid((unsigned)cdiv(a.L, 256));
    if (a.dtype == HASTE_DTYPE_F32) {
        hipFuncSetAttribute((const void *)k_bwd_w_valu<float>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_bwd_w_valu<float>, grid, dim3(256), lds, s, (const float *)X, idx, (const float *)dY, dW,
                           dbias, beta, (int)a.B, (int)a.F_s, a.L, (int)a.G, (int)a.F_in);
    } else {
        hipFuncSetAttribute((const void *)k_bwd_w_valu<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_bwd_w_valu<bf16_t>, grid, dim3(256), lds, s, (const bf16_t *)X, idx, (const bf16_t *)dY,
                           dW, dbias, beta, (int)a.B, (int)a.F_s, a.L, (int)a.G, (int)a.F_in);
    }
    return hipGetLastError();
}

size_t bwd_x_valu_ws(const TailArgs &a) {
    const int64_t S = bwd_x_valu_segments(a);
    return (size_t)S * (size_t)a.F_s * (size_t)(cdiv(a.B, 32) * 32) * 4 + 256;
}

hipError_t bwd_x_valu(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s) {
    const int64_t nbt = cdiv(a.B, 32);
    const int64_t S = bwd_x_valu_segments(a);
    const int64_t lps = cdiv(a.L, S);
    const int Bp = (int)(nbt * 32);
    const size_t lds = bwd_x_valu_lds(a);
    float *part = reinterpret_cast<float *>(ws);
    const dim3 grid((unsigned)S, (unsigned)nbt);
    if (a.dtype == HASTE_DTYPE_F32) {
        hipFuncSetAttribute((const void *)k_bwd_x_valu<float>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_bwd_x_valu<float>, grid, dim3(kOwnWaves * 64), lds, s, idx, (const float *)W,
                           (const float *)dY, part, (int)a.B, Bp, (int)a.F_s, a.L, (int)a.G, (int)a.F_in, lps);
    } else {
        hipFuncSetAttribute((const void *)k_bwd_x_valu<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k_bwd_x_valu<bf16_t>, grid, dim3(kOwnWaves * 64), lds, s, idx, (const bf16_t *)W,
                           (const bf16_t *)dY, part, (int)a.B, Bp, (int)a.F_s, a.L, (int)a.G, (int)a.F_in, lps);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)S, Bp, a.B, a.F_s, dX, beta, s);
}

}  // namespace haste
