// Small helper kernels: fills, fixed-order partial reductions, idx validation, gather export.
#include "common.hpp"

namespace {

__global__ void k_fill(float *__restrict__ p, int64_t n, float v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// dX[b, f] = beta dX[b, f] + sum_{k < S} part[k][f][b], summed in ascending k.  A workgroup takes
// 8 features x 128 rows: each thread reads 4 consecutive rows (16 bytes, 512 contiguous bytes per
// feature and wave) of every partial, with the loads of 8 partials in flight, and the tile is
// transposed through LDS so that dX is written 16 bytes per thread.
__global__ __launch_bounds__(256) void k_reduce_fmajor(const float *__restrict__ part, int S, int64_t ldp,
                                                       int64_t B, int64_t F_s, float *__restrict__ dX, int beta) {
    __shared__ float tile[8][128 + 4];
    const int64_t f0 = (int64_t)blockIdx.x * 8, b0 = (int64_t)blockIdx.y * 128;
    const int t = threadIdx.x, bq = t & 31, fr = t >> 5;
    const int64_t f = f0 + fr, b = b0 + 4 * bq;
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (f < F_s && b < ldp) {
        const float4 *p = reinterpret_cast<const float4 *>(part + f * ldp + b);
        const int64_t ks = F_s * ldp / 4;   // float4 stride between partials
        int k = 0;
        for (; k + 8 <= S; k += 8) {
            float4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = p[(int64_t)(k + j) * ks];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc.x += v[j].x;
                acc.y += v[j].y;
                acc.z += v[j].z;
                acc.w += v[j].w;
            }
        }
        for (; k < S; ++k) {
            const float4 v = p[(int64_t)k * ks];
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
    }
    tile[fr][4 * bq + 0] = acc.x;
    tile[fr][4 * bq + 1] = acc.y;
    tile[fr][4 * bq + 2] = acc.z;
    tile[fr][4 * bq + 3] = acc.w;
    __syncthreads();
    // thread -> row b0 + t / 2, features f0 + 4 (t % 2) .. +3
    const int64_t ob = b0 + (t >> 1), of = f0 + 4 * (t & 1);
    if (ob < B) {
        const int r = t >> 1, c = 4 * (t & 1);
        float4 s4 = make_float4(tile[c][r], tile[c + 1][r], tile[c + 2][r], tile[c + 3][r]);
        float *q = dX + ob * F_s + of;
        if (of + 3 < F_s && ((F_s & 3) == 0)) {
            if (beta) {
                const float4 o = *reinterpret_cast<const float4 *>(q);
                s4.x += o.x;
                s4.y += o.y;
                s4.z += o.z;
                s4.w += o.w;
            }
            *reinterpret_cast<float4 *>(q) = s4;
        } else {
            const float v[4] = {s4.x, s4.y, s4.z, s4.w};
            for (int j = 0; j < 4; ++j)
                if (of + j < F_s) q[j] = beta ? q[j] + v[j] : v[j];
        }
    }
}

// C[i] (+)= sum_{k < S} part[k][i] in ascending k, four consecutive elements per thread (16-byte
// loads) with the loads of 16 partials in flight: the partial sums are read once, at a rate the
// one-float-per-thread loop below does not reach (its loads wait one by one).  MN % 4 == 0 and
// 16-byte aligned arrays.
__global__ __launch_bounds__(256) void k_reduce_rmajor4(const float4 *__restrict__ part, int S, int64_t MN4,
                                                        float4 *__restrict__ C, int beta) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= MN4) return;
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    int k = 0;
    for (; k + 16 <= S; k += 16) {
        float4 v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = part[(int64_t)(k + j) * MN4 + i];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            acc.x += v[j].x;
            acc.y += v[j].y;
            acc.z += v[j].z;
            acc.w += v[j].w;
        }
    }
    for (; k < S; ++k) {
        const float4 v = part[(int64_t)k * MN4 + i];
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
    }
    if (beta) {
        const float4 o = C[i];
        acc.x = o.x + acc.x;
        acc.y = o.y + acc.y;
        acc.z = o.z + acc.z;
        acc.w = o.w + acc.w;
    }
    C[i] = acc;
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


// BCE gradient of stored logits (Section 3.3 objective): dY[b, n] = sigmoid(Y[b, n]) - T[b, n], with
// T[b, n] = 1 where n occurs in pos[b, 0..P-1].  A workgroup takes 2048 columns of one row and a
// thread 8 consecutive columns; the row's positives are workgroup-uniform reads.  Y and dY may be
// the same buffer (each element is read before it is written, by the same thread).
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void k_bce_grad(const T *Y, const int32_t *__restrict__ pos, int P, T *dY,
                                                  int64_t N, int64_t nchunk) {
    const int64_t b = blockIdx.x / nchunk;
    const int64_t c0 = (blockIdx.x - b * nchunk) * 2048 + 8 * (int64_t)threadIdx.x;
    if (c0 >= N) return;
    uint32_t t = 0;
    for (int p = 0; p < P; ++p) {
        const int64_t d = (int64_t)pos[b * P + p] - c0;
        if (d >= 0 && d < 8) t |= 1u << d;
    }
    const T *y = Y + b * N + c0;
    T *o = dY + b * N + c0;
    if constexpr (VEC && sizeof(T) == 2) {   // bf16, whole 16-byte groups
        const uint4 v = *reinterpret_cast<const uint4 *>(y);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        uint32_t r[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
            r[i] = pack_bf16(bce_grad_f32(__uint_as_float(w[i] << 16), (t >> (2 * i)) & 1),
                             bce_grad_f32(__uint_as_float(w[i] & 0xffff0000u), (t >> (2 * i + 1)) & 1));
        *reinterpret_cast<uint4 *>(o) = make_uint4(r[0], r[1], r[2], r[3]);
    } else {
        const int n = N - c0 < 8 ? (int)(N - c0) : 8;
        for (int i = 0; i < n; ++i) store_out(o, i, bce_grad_f32(load_f32(y, i), (t >> i) & 1));
    }
}

// Each batch row's positives sorted ascending (one wave per row): element i goes to its rank
// #{j : v_j < v_i, or v_j == v_i and j < i}; ids outside [0, N) (the -1 padding) sort last as
// INT32_MAX.
__global__ __launch_bounds__(256) void k_sort_pos(const int32_t *__restrict__ pos, int P, int64_t B, int64_t N,
                                                  int32_t *__restrict__ spos) {
    __shared__ int32_t v[4][haste::kSortPosMax];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t b = (int64_t)blockIdx.x * 4 + w;
    if (b >= B) return;   // wave-uniform; no barrier follows
    for (int i = lane; i < P; i += 64) {
        const int32_t x = pos[b * P + i];
        v[w][i] = x >= 0 && x < N ? x : INT32_MAX;
    }
    __builtin_amdgcn_wave_barrier();
    for (int i = lane; i < P; i += 64) {
        const int32_t x = v[w][i];
        int r = 0;
        for (int j = 0; j < P; ++j) {
            const int32_t y = v[w][j];
            r += (y < x) || (y == x && j < i);
        }
        spos[b * P + r] = x;
    }
}

// One momentum step per weight (sgd_step), four consecutive weights per thread: 16-byte velocity and
// gradient accesses and 8- or 16-byte weight accesses when n is a multiple of 4 and the buffers are
// aligned (VEC), else one weight per thread.  W_next may be W: each weight is read before it is
// written, by the same thread.  g == NULL: a zero gradient.
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void k_sgd_momentum(const T *W, const float *__restrict__ g, float *__restrict__ m,
                                                      T *W_next, int64_t n, float lr, float momentum,
                                                      float weight_decay) {
    const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * (VEC ? 4 : 1);
    if (i0 >= n) return;
    if constexpr (VEC) {
        const float4 gv = g ? *reinterpret_cast<const float4 *>(g + i0) : make_float4(0.f, 0.f, 0.f, 0.f);
        float4 mv = *reinterpret_cast<const float4 *>(m + i0);
        float w[4], o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = load_f32(W, i0 + j);
        sgd_step(w[0], gv.x, mv.x, o[0], lr, momentum, weight_decay);
        sgd_step(w[1], gv.y, mv.y, o[1], lr, momentum, weight_decay);
        sgd_step(w[2], gv.z, mv.z, o[2], lr, momentum, weight_decay);
        sgd_step(w[3], gv.w, mv.w, o[3], lr, momentum, weight_decay);
        *reinterpret_cast<float4 *>(m + i0) = mv;
        if constexpr (sizeof(T) == 2)
            *reinterpret_cast<uint2 *>(W_next + i0) = make_uint2(pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3]));
        else
            *reinterpret_cast<float4 *>(W_next + i0) = make_float4(o[0], o[1], o[2], o[3]);
    } else {
        float mm = m[i0], o;
        sgd_step(load_f32(W, i0), g ? g[i0] : 0.0f, mm, o, lr, momentum, weight_decay);
        m[i0] = mm;
        store_out(W_next, i0, o);
    }
}
}  // namespace

namespace haste {

hipError_t fill_f32(float *p, int64_t n, float v, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill, dim3(grid_for(n)), dim3(256), 0, s, p, n, v);
    return hipGetLastError();
}

hipError_t reduce_fmajor(const float *part, int S, int64_t ldp, int64_t B, int64_t F_s, float *dX, int beta,
                         hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_reduce_fmajor, dim3((unsigned)cdiv(F_s, 8), (unsigned)cdiv(B, 128)), dim3(256), 0, s, part,
                       S, ldp, B, F_s, dX, beta);
    return hipGetLastError();
}

hipError_t reduce_rmajor(const float *part, int S, int64_t M, int64_t N, float *C, int beta, hipStream_t s) {
    const int64_t MN = M * N;
    if (MN <= 0) return hipSuccess;
    if (MN % 4 == 0 && (reinterpret_cast<uintptr_t>(part) & 15) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0) {
        hipLaunchKernelGGL(k_reduce_rmajor4, dim3((unsigned)cdiv(MN / 4, 256)), dim3(256), 0, s,
                           reinterpret_cast<const float4 *>(part), S, MN / 4, reinterpret_cast<float4 *>(C), beta);
        return hipGetLastError();
    }
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


hipError_t bce_grad(int64_t B, int64_t N, int32_t dtype, const void *Y, const int32_t *pos, int P, void *dY,
                    hipStream_t s) {
    const int64_t nchunk = cdiv(N, 2048);
    const dim3 grid((unsigned)(B * nchunk)), block(256);
    const bool vec = (N % 8) == 0 && ((reinterpret_cast<uintptr_t>(Y) | reinterpret_cast<uintptr_t>(dY)) & 15) == 0;
    if (dtype == HASTE_DTYPE_BF16) {
        if (vec)
            hipLaunchKernelGGL((k_bce_grad<bf16_t, true>), grid, block, 0, s, (const bf16_t *)Y, pos, P, (bf16_t *)dY, N, nchunk);
        else
            hipLaunchKernelGGL((k_bce_grad<bf16_t, false>), grid, block, 0, s, (const bf16_t *)Y, pos, P, (bf16_t *)dY, N, nchunk);
    } else {
        hipLaunchKernelGGL((k_bce_grad<float, false>), grid, block, 0, s, (const float *)Y, pos, P, (float *)dY, N, nchunk);
    }
    return hipGetLastError();
}


hipError_t sort_positives(int64_t B, int64_t N, const int32_t *pos, int P, int32_t *spos, hipStream_t s) {
    if (B <= 0 || P <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_sort_pos, dim3((unsigned)cdiv(B, 4)), dim3(256), 0, s, pos, P, B, N, spos);
    return hipGetLastError();
}

hipError_t sgd_momentum(int64_t n, int32_t dtype, const void *W, const float *g, float *m, const haste_sgd_t &opt,
                        void *W_next, hipStream_t s) {
    const uintptr_t al = reinterpret_cast<uintptr_t>(W) | reinterpret_cast<uintptr_t>(g) |
                         reinterpret_cast<uintptr_t>(m) | reinterpret_cast<uintptr_t>(W_next);
    const bool vec = (n % 4) == 0 && (al & 15) == 0;
    const dim3 grid((unsigned)cdiv(n, vec ? 1024 : 256)), block(256);
    if (dtype == HASTE_DTYPE_BF16) {
        if (vec)
            hipLaunchKernelGGL((k_sgd_momentum<bf16_t, true>), grid, block, 0, s, (const bf16_t *)W, g, m,
                               (bf16_t *)W_next, n, opt.lr, opt.momentum, opt.weight_decay);
        else
            hipLaunchKernelGGL((k_sgd_momentum<bf16_t, false>), grid, block, 0, s, (const bf16_t *)W, g, m,
                               (bf16_t *)W_next, n, opt.lr, opt.momentum, opt.weight_decay);
    } else {
        if (vec)
            hipLaunchKernelGGL((k_sgd_momentum<float, true>), grid, block, 0, s, (const float *)W, g, m,
                               (float *)W_next, n, opt.lr, opt.momentum, opt.weight_decay);
        else
            hipLaunchKernelGGL((k_sgd_momentum<float, false>), grid, block, 0, s, (const float *)W, g, m,
                               (float *)W_next, n, opt.lr, opt.momentum, opt.weight_decay);
    }
    return hipGetLastError();
}

}  // namespace haste
