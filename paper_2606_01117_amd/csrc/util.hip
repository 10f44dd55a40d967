// Small helper kernels: fills, fixed-order partial reductions, idx validation, gather export.
#include "common.hpp"

namespace {

__global__ void k_fill(float *__restrict__ p, int64_t n, float v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_scale(float *__restrict__ p, int64_t n, float beta) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] *= beta;
}

// dX[b, f] = beta*dX[b, f] + sum_{s in order} part[s][f][b]; 32x32 tiles transposed through LDS
__global__ __launch_bounds__(256) void k_reduce_fmajor(const float *__restrict__ part, int S, int64_t ldp,
                                                       int64_t B, int64_t F_s, float *__restrict__ dX, int beta) {
    __shared__ float tile[32][33];
    const int64_t f0 = (int64_t)blockIdx.x * 32, b0 = (int64_t)blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int r = ty; r < 32; r += 8) {
        const int64_t f = f0 + r, b = b0 + tx;
        float s = 0.0f;
        if (f < F_s && b < B) {
            const float *p = part + f * ldp + b;
            for (int k = 0; k < S; ++k) s += p[(int64_t)k * F_s * ldp];
        }
        tile[r][tx] = s;
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
        const int64_t b = b0 + r, f = f0 + tx;
        if (b < B && f < F_s) {
            float *q = dX + b * F_s + f;
            *q = beta ? *q + tile[tx][r] : tile[tx][r];
        }
    }
}

__global__ void k_reduce_rmajor(const float *__restrict__ part, int S, int64_t MN, float *__restrict__ C, int beta) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < MN; i += (int64_t)gridDim.x * blockDim.x) {
        float s = 0.0f;
        for (int k = 0; k < S; ++k) s += part[(int64_t)k * MN + i];
        C[i] = beta ? C[i] + s : s;
    }
}

__global__ void k_validate(const int32_t *__restrict__ idx, int64_t rows, int64_t F_in, int64_t F_s,
                           int32_t *__restrict__ n_bad) {
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < rows; r += (int64_t)gridDim.x * blockDim.x) {
        const int32_t *p = idx + r * F_in;
        bool ok = true;
        int64_t prev = -1;
        for (int64_t t = 0; t < F_in; ++t) {
            const int64_t v = p[t];
            if (v <= prev || v >= F_s) ok = false;
            prev = v;
        }
        if (!ok) atomicAdd(n_bad, 1);
    }
}

__global__ void k_zero_i32(int32_t *p) { *p = 0; }

template <typename T>
__global__ void k_gather(const T *__restrict__ X, const int32_t *__restrict__ idx, int64_t B, int64_t F_s,
                         int64_t F_in, int64_t k0, int64_t nk, T *__restrict__ out) {
    const int64_t n = nk * B * F_in;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t t = i % F_in, b = (i / F_in) % B, k = i / (F_in * B);
        out[i] = X[b * F_s + idx[(k0 + k) * F_in + t]];
    }
}

unsigned grid_for(int64_t n) {
    int64_t g = haste::cdiv(n, 256);
    if (g > 4096) g = 4096;
    return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

namespace haste {

hipError_t fill_f32(float *p, int64_t n, float v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill, dim3(grid_for(n)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t scale_f32(float *p, int64_t n, float beta, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_scale, dim3(grid_for(n)), dim3(256), 0, s, p, n, beta);
    return hipGetLastError();
}

hipError_t reduce_fmajor(const float *part, int S, int64_t ldp, int64_t B, int64_t F_s, float *dX, int beta,
                         hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_reduce_fmajor, dim3((unsigned)cdiv(F_s, 32), (unsigned)cdiv(B, 32)), dim3(256), 0, s, part,
                       S, ldp, B, F_s, dX, beta);
    return hipGetLastError();
}

hipError_t reduce_rmajor(const float *part, int S, int64_t M, int64_t N, float *C, int beta, hipStream_t s) {
    const int64_t MN = M * N;
    if (MN <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_reduce_rmajor, dim3(grid_for(MN)), dim3(256), 0, s, part, S, MN, C, beta);
    return hipGetLastError();
}

hipError_t validate_idx(const int32_t *idx, int64_t rows, int64_t F_in, int64_t F_s, int32_t *n_bad,
                        hipStream_t s) {
    hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(1), 0, s, n_bad);
    if (rows > 0) hipLaunchKernelGGL(k_validate, dim3(grid_for(rows)), dim3(256), 0, s, idx, rows, F_in, F_s, n_bad);
    return hipGetLastError();
}

hipError_t debug_gather(const void *X, int32_t dtype, const int32_t *idx, int64_t B, int64_t F_s, int64_t F_in,
                        int64_t k0, int64_t nk, void *out, hipStream_t s) {
    const int64_t n = nk * B * F_in;
    if (n <= 0) return hipSuccess;
    if (dtype == HASTE_DTYPE_BF16)
        hipLaunchKernelGGL(k_gather<bf16_t>, dim3(grid_for(n)), dim3(256), 0, s, (const bf16_t *)X, idx, B, F_s, F_in,
                           k0, nk, (bf16_t *)out);
    else
        hipLaunchKernelGGL(k_gather<float>, dim3(grid_for(n)), dim3(256), 0, s, (const float *)X, idx, B, F_s, F_in, k0,
                           nk, (float *)out);
    return hipGetLastError();
}

}  // namespace haste
