// Dense head over the frequent labels (paper Section 3.3, a^H = W_head h_head) and its backward.
//
// All three products are plain GEMMs C[M,N] = A[M,K] B[K,N] whose operands arrive in different
// layouts:
//   forward   Y_h  = X  W_head^T    A = X      (K contiguous), B = W_head^T (K contiguous)
//   dW_head   dW_h = dY_h^T X       A = dY_h^T (M contiguous), B = X        (N contiguous)
//   dX        dX  += dY_h W_head    A = dY_h   (K contiguous), B = W_head   (N contiguous), K = H
// The bf16 kernel stages 128x32 tiles of both operands in LDS with K contiguous (operands that
// are contiguous along M/N are transposed while being written to LDS) and runs
// v_mfma_f32_32x32x16_bf16 on a 2x2 grid of waves, each owning a 64x64 block.  dX contracts over
// the H head labels, so it is split over K and the partials are reduced in a fixed order.
#include "common.hpp"

namespace {

enum { EPI_BF16_BIAS = 0, EPI_F32 = 1, EPI_F32_PART = 2 };

constexpr int TM = 128, TN = 128, TK = 32;
constexpr int LS = TK + 8;  // LDS row stride (bf16): 80 bytes keeps 16-byte rows aligned

// 8 consecutive elements along the operand's contiguous dimension, zero outside [0, lim)
__device__ __forceinline__ uint4 load8(const bf16_t *__restrict__ p, int64_t pos, int64_t lim) {
    if (pos + 8 <= lim && ((reinterpret_cast<uintptr_t>(p) & 15) == 0)) return *reinterpret_cast<const uint4 *>(p);
    bf16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = (pos + i < lim) ? p[i] : (bf16_t)0;
    return make_uint4(pack2(e[0], e[1]), pack2(e[2], e[3]), pack2(e[4], e[5]), pack2(e[6], e[7]));
}

// Stage a 128 x 32 operand tile into LDS as tile[r][k] (k contiguous).  Element (r, k) of the
// operand lives at base + r*sr + k*sk; exactly one of sr, sk is 1 (KC: k contiguous).
template <bool KC>
__device__ __forceinline__ void stage(bf16_t *tile, const bf16_t *__restrict__ base, int64_t sr, int64_t sk,
                                      int64_t r0, int64_t rlim, int64_t k0, int64_t klim) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int c = threadIdx.x + 256 * q;
        if (KC) {
            const int r = c >> 2, kc = (c & 3) * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (r0 + r < rlim) v = load8(base + (r0 + r) * sr + (k0 + kc), k0 + kc, klim);
            *reinterpret_cast<uint4 *>(tile + r * LS + kc) = v;
        } else {
            const int k = c >> 4, rc = (c & 15) * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (k0 + k < klim) v = load8(base + (k0 + k) * sk + (r0 + rc), r0 + rc, rlim);
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                tile[(rc + 2 * h) * LS + k] = (bf16_t)(u[h] & 0xffffu);
                tile[(rc + 2 * h + 1) * LS + k] = (bf16_t)(u[h] >> 16);
            }
        }
    }
}

template <bool AK, bool BK, int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(const bf16_t *__restrict__ A, int64_t sam, int64_t sak,
                                                   const bf16_t *__restrict__ Bm, int64_t sbk, int64_t sbn,
                                                   void *__restrict__ C, int64_t ldc, const float *__restrict__ bias,
                                                   int64_t M, int64_t N, int64_t K, int64_t kchunk) {
    __shared__ __align__(16) bf16_t As[TM * LS];
    __shared__ __align__(16) bf16_t Bs[TN * LS];
    const int64_t n0 = (int64_t)blockIdx.x * TN, m0 = (int64_t)blockIdx.y * TM;
    const int64_t kb = (int64_t)blockIdx.z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ln = lane & 31, hh = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{0};

    for (int64_t k0 = kb; k0 < ke; k0 += TK) {
        // A(m, k) at A + m*sam + k*sak ; B(k, n) at Bm + k*sbk + n*sbn
        stage<AK>(As, A, sam, sak, m0, M, k0, ke);
        stage<BK>(Bs, Bm, sbn, sbk, n0, N, k0, ke);
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < TK / 16; ++ks) {
            uint4 av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *reinterpret_cast<const uint4 *>(As + (wm * 64 + i * 32 + ln) * LS + ks * 16 + 8 * hh);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bv[j] = *reinterpret_cast<const uint4 *>(Bs + (wn * 64 + j * 32 + ln) * LS + ks * 16 + 8 * hh);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x16(as_bf16x8(av[i]), as_bf16x8(bv[j]), acc[i][j]);
        }
        __syncthreads();
    }
    // D[m = 8r + 4hh + q][n = ln] per 32x32 block
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 64 + j * 32 + ln;
            if (n >= N) continue;
            const float bv = (EPI == EPI_BF16_BIAS && bias) ? bias[n] : 0.0f;
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t m = m0 + wm * 64 + i * 32 + 8 * r + 4 * hh + q;
                    if (m >= M) continue;
                    const float v = acc[i][j][4 * r + q];
                    if (EPI == EPI_BF16_BIAS) {
                        reinterpret_cast<bf16_t *>(C)[m * ldc + n] = f32_to_bf16(v + bv);
                    } else if (EPI == EPI_F32) {
                        reinterpret_cast<float *>(C)[m * ldc + n] = v;
                    } else {
                        reinterpret_cast<float *>(C)[(int64_t)blockIdx.z * M * N + m * N + n] = v;
                    }
                }
        }
}

// fp32 GEMM on the vector ALUs (fp32 heads): 64x64 tiles, 4x4 outputs per thread.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float *__restrict__ A, int64_t sam, int64_t sak,
                                                  const float *__restrict__ Bm, int64_t sbk, int64_t sbn,
                                                  void *__restrict__ C, int64_t ldc, const float *__restrict__ bias,
                                                  int64_t M, int64_t N, int64_t K, int64_t kchunk) {
    __shared__ float As[16][64 + 4];
    __shared__ float Bs[16][64 + 4];
    const int64_t n0 = (int64_t)blockIdx.x * 64, m0 = (int64_t)blockIdx.y * 64;
    const int64_t kb = (int64_t)blockIdx.z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float acc[4][4] = {};
    for (int64_t k0 = kb; k0 < ke; k0 += 16) {
        for (int e = threadIdx.x; e < 16 * 64; e += 256) {
            const int k = e >> 6, r = e & 63;
            As[k][r] = (m0 + r < M && k0 + k < ke) ? A[(m0 + r) * sam + (k0 + k) * sak] : 0.0f;
            Bs[k][r] = (n0 + r < N && k0 + k < ke) ? Bm[(k0 + k) * sbk + (n0 + r) * sbn] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m >= M || n >= N) continue;
            const float v = acc[i][j];
            if (EPI == EPI_BF16_BIAS) {
                reinterpret_cast<float *>(C)[m * ldc + n] = v + (bias ? bias[n] : 0.0f);
            } else if (EPI == EPI_F32) {
                reinterpret_cast<float *>(C)[m * ldc + n] = v;
            } else {
                reinterpret_cast<float *>(C)[(int64_t)blockIdx.z * M * N + m * N + n] = v;
            }
        }
}

// split of the H contraction of dX: enough workgroups to cover the chip, never below 256 per chunk
int64_t head_splits(int64_t B, int64_t F_s, int64_t H, int32_t dtype) {
    const int64_t tm = dtype == HASTE_DTYPE_BF16 ? TM : 64, tn = dtype == HASTE_DTYPE_BF16 ? TN : 64;
    const int64_t tiles = haste::cdiv(B, tm) * haste::cdiv(F_s, tn);
    int64_t S = haste::cdiv(512, tiles < 1 ? 1 : tiles);
    const int64_t maxS = haste::cdiv(H, 256);
    if (S > maxS) S = maxS;
    return S < 1 ? 1 : S;
}

}  // namespace

namespace haste {

size_t head_ws(int64_t B, int64_t F_s, int64_t H, int32_t dtype) {
    return (size_t)head_splits(B, F_s, H, dtype) * (size_t)B * (size_t)F_s * 4 + 256;
}

hipError_t head_fwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const float *bias_h, void *Yh, hipStream_t s) {
    // M = B, N = H, K = F_s;  A(m,k) = X[m*F_s + k];  B(k,n) = Wh[n*F_s + k]
    if (dtype == HASTE_DTYPE_BF16) {
        const dim3 grid((unsigned)cdiv(H, TN), (unsigned)cdiv(B, TM), 1);
        hipLaunchKernelGGL((k_gemm_bf16<true, true, EPI_BF16_BIAS>), grid, dim3(256), 0, s, (const bf16_t *)X, F_s,
                           (int64_t)1, (const bf16_t *)Wh, (int64_t)1, F_s, Yh, H, bias_h, B, H, F_s, F_s);
    } else {
        const dim3 grid((unsigned)cdiv(H, 64), (unsigned)cdiv(B, 64), 1);
        hipLaunchKernelGGL((k_gemm_f32<EPI_BF16_BIAS>), grid, dim3(256), 0, s, (const float *)X, F_s, (int64_t)1,
                           (const float *)Wh, (int64_t)1, F_s, Yh, H, bias_h, B, H, F_s, F_s);
    }
    return hipGetLastError();
}

hipError_t head_bwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const void *dYh, float *dWh, float *dX, int beta_dx, void *ws, hipStream_t s) {
    const bool bf = dtype == HASTE_DTYPE_BF16;
    if (dWh) {
        // M = H, N = F_s, K = B;  A(m,k) = dYh[k*H + m];  B(k,n) = X[k*F_s + n]
        if (bf) {
            const dim3 grid((unsigned)cdiv(F_s, TN), (unsigned)cdiv(H, TM), 1);
            hipLaunchKernelGGL((k_gemm_bf16<false, false, EPI_F32>), grid, dim3(256), 0, s, (const bf16_t *)dYh,
                               (int64_t)1, H, (const bf16_t *)X, F_s, (int64_t)1, (void *)dWh, F_s,
                               (const float *)nullptr, H, F_s, B, B);
        } else {
            const dim3 grid((unsigned)cdiv(F_s, 64), (unsigned)cdiv(H, 64), 1);
            hipLaunchKernelGGL((k_gemm_f32<EPI_F32>), grid, dim3(256), 0, s, (const float *)dYh, (int64_t)1, H,
                               (const float *)X, F_s, (int64_t)1, (void *)dWh, F_s, (const float *)nullptr, H, F_s,
                               B, B);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dX) {
        // M = B, N = F_s, K = H;  A(m,k) = dYh[m*H + k];  B(k,n) = Wh[k*F_s + n]; split over K
        const int64_t S = head_splits(B, F_s, H, dtype);
        const int64_t kchunk = round_up(cdiv(H, S), 32);
        const int64_t Sx = cdiv(H, kchunk);
        float *part = reinterpret_cast<float *>(ws);
        if (bf) {
            const dim3 grid((unsigned)cdiv(F_s, TN), (unsigned)cdiv(B, TM), (unsigned)Sx);
            hipLaunchKernelGGL((k_gemm_bf16<true, false, EPI_F32_PART>), grid, dim3(256), 0, s, (const bf16_t *)dYh,
                               H, (int64_t)1, (const bf16_t *)Wh, F_s, (int64_t)1, (void *)part, F_s,
                               (const float *)nullptr, B, F_s, H, kchunk);
        } else {
            const dim3 grid((unsigned)cdiv(F_s, 64), (unsigned)cdiv(B, 64), (unsigned)Sx);
            hipLaunchKernelGGL((k_gemm_f32<EPI_F32_PART>), grid, dim3(256), 0, s, (const float *)dYh, H, (int64_t)1,
                               (const float *)Wh, F_s, (int64_t)1, (void *)part, F_s, (const float *)nullptr, B, F_s,
                               H, kchunk);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return reduce_rmajor(part, (int)Sx, B, F_s, dX, beta_dx, s);
    }
    return hipSuccess;
}

}  // namespace haste
