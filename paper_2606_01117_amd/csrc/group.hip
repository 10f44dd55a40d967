// Semantic grouping of labels (Alg. 2): coarse spherical k-means into C = max(1, N / (beta G))
// clusters, then greedy groups of G inside each cluster (a random unassigned seed and its top-G
// unassigned labels by similarity).  Embeddings are unit vectors stored as int8 (x 127): every
// similarity is an exact integer dot product, so every assignment, seed and top-G decision is
// exact.  The assignment is a dense contraction [N, D] x [D, C] and runs on int8 MFMA.
// Draws: SplitMix64 (Steele, Lea and Flood, 2014) in counter form.
#include <climits>

#include "common.hpp"

namespace {

typedef int i32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint64_t splitmix64_at(uint64_t s, uint64_t i) {
    uint64_t z = s + (i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ void k_gl_iota(int32_t *__restrict__ a, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) a[i] = (int32_t)i;
}

// the first C entries of a partial Fisher-Yates shuffle of [0, N): swap partner of i is
// i + out(i) mod (N - i)
__global__ void k_gl_shuffle(int32_t *__restrict__ a, int64_t N, int64_t C, uint64_t seed) {
    if (threadIdx.x != 0) return;
    for (int64_t i = 0; i < C; ++i) {
        const int64_t j = i + (int64_t)(splitmix64_at(seed, (uint64_t)i) % (uint64_t)(N - i));
        const int32_t t = a[i];
        a[i] = a[j];
        a[j] = t;
    }
}

__global__ void k_gl_pick_centres(const int8_t *__restrict__ E, const int32_t *__restrict__ a, int64_t C, int D,
                                  int8_t *__restrict__ cen) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= C * D) return;
    const int64_t c = i / D;
    cen[i] = E[(int64_t)a[c] * D + (i - c * D)];
}

// cl[l] = argmax_c <E[l], cen[c]> (ties: the lower c).  A wave takes 16 labels, a workgroup of 8
// waves 128; centres pass through LDS 16 at a time.  v_mfma_i32_16x16x64_i8, M = 16 labels,
// N = 16 centres, K = 64 dimensions: both operands hold, per lane, 16 consecutive dimensions
// (16 q .. 16 q + 15 of the 64-chunk) of their row, so each lane group contracts the same
// dimensions; result lane (centre l16, q) holds labels 4q .. 4q+3 of the wave's 16.
constexpr int kGlWaves = 8;
constexpr int kGlMaxD = 1024;

__global__ __launch_bounds__(64 * kGlWaves) void k_gl_assign(const int8_t *__restrict__ E, int64_t N, int D,
                                                             const int8_t *__restrict__ cen, int64_t C,
                                                             int32_t *__restrict__ cl) {
    __shared__ __align__(16) int8_t tile[16 * kGlMaxD];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, q = lane >> 4;
    const int64_t l0 = (int64_t)blockIdx.x * (16 * kGlWaves) + 16 * wave;
    const int nk = (D + 63) / 64;
    // this lane's A rows: label l0 + l16, dims 64 kk + 16 q .. +15 (zero past D or past N)
    const Buf eb(E, (uint32_t)(N * D));
    i32x4_t a[kGlMaxD / 64];
#pragma unroll
    for (int kk = 0; kk < kGlMaxD / 64; ++kk) {
        const int d0 = 64 * kk + 16 * q;
        const bool ok = kk < nk && d0 < D && l0 + l16 < N;
        a[kk] = __builtin_bit_cast(i32x4_t, eb.ld16(ok ? (uint32_t)((l0 + l16) * D + d0) : kOob));
    }
    int bv[4], bi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bv[i] = INT32_MIN;
        bi[i] = 0;
    }
    const Buf cb(cen, (uint32_t)(C * D));
    for (int64_t c0 = 0; c0 < C; c0 += 16) {
        __syncthreads();   // the previous tile is no longer read
        for (int e = threadIdx.x; e < 16 * (D / 16); e += 64 * kGlWaves) {
            const int r = e / (D / 16), ch = e - r * (D / 16);
            const uint4 v = cb.ld16(c0 + r < C ? (uint32_t)((c0 + r) * D + 16 * ch) : kOob);
            *reinterpret_cast<uint4 *>(tile + r * kGlMaxD + 16 * ch) = v;
        }
        __syncthreads();
        i32x4_t acc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < kGlMaxD / 64; ++kk) {
            if (kk >= nk) break;
            const int d0 = 64 * kk + 16 * q;
            const i32x4_t b = d0 < D ? *reinterpret_cast<const i32x4_t *>(tile + l16 * kGlMaxD + d0) : i32x4_t{0, 0, 0, 0};
            acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[kk], b, acc, 0, 0, 0);
        }
        const int c = (int)(c0 + l16);
        if (c < C) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (acc[i] > bv[i]) {   // centres ascend per lane: ties keep the lower one
                    bv[i] = acc[i];
                    bi[i] = c;
                }
        }
    }
    // best over the 16 lanes of each row group: larger value, then lower centre
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        for (int off = 1; off < 16; off <<= 1) {
            const int ov = __shfl_xor(bv[i], off, 64), oi = __shfl_xor(bi[i], off, 64);
            if (ov > bv[i] || (ov == bv[i] && oi < bi[i])) {
                bv[i] = ov;
                bi[i] = oi;
            }
        }
        const int64_t l = l0 + 4 * q + i;
        if (l16 == 0 && l < N) cl[l] = bi[i];
    }
}

__global__ void k_gl_zero(int32_t *__restrict__ p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

__global__ void k_gl_count(const int32_t *__restrict__ cl, int64_t N, int32_t *__restrict__ cnt) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < N) atomicAdd(&cnt[cl[i]], 1);
}

// block-wide inclusive sum of one value per thread (256 threads)
__device__ __forceinline__ int32_t block_incl_scan(int32_t v, int32_t *s) {
    s[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int32_t a = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += a;
        __syncthreads();
    }
    const int32_t r = s[threadIdx.x];
    __syncthreads();
    return r;
}

// start[c] = sum of cnt[< c]; gstart[c] = sum of ceil(cnt[< c] / G); start[C], gstart[C] the totals
// (one workgroup)
__global__ __launch_bounds__(256) void k_gl_starts(const int32_t *__restrict__ cnt, int64_t C, int64_t G,
                                                   int32_t *__restrict__ start, int32_t *__restrict__ gstart,
                                                   int64_t *__restrict__ n_groups) {
    __shared__ int32_t s[256];
    __shared__ int32_t carry[2];
    if (threadIdx.x == 0) carry[0] = carry[1] = 0;
    __syncthreads();
    for (int64_t base = 0; base < C; base += 256) {
        const int64_t c = base + threadIdx.x;
        const int32_t v = c < C ? cnt[c] : 0;
        const int32_t g = (int32_t)((v + G - 1) / G);
        const int32_t iv = block_incl_scan(v, s);
        const int32_t ig = block_incl_scan(g, s);
        if (c < C) {
            start[c] = carry[0] + iv - v;
            gstart[c] = carry[1] + ig - g;
        }
        __syncthreads();
        if (threadIdx.x == 255) {
            carry[0] += iv;
            carry[1] += ig;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        start[C] = carry[0];
        gstart[C] = carry[1];
        *n_groups = carry[1];
    }
}

// members[start[c] ..] = the labels of cluster c in ascending order (one workgroup per cluster)
__global__ __launch_bounds__(256) void k_gl_collect(const int32_t *__restrict__ cl, int64_t N,
                                                    const int32_t *__restrict__ start, int32_t *__restrict__ members) {
    __shared__ int32_t s[256];
    const int c = blockIdx.x;
    int32_t pos = start[c];
    for (int64_t base = 0; base < N; base += 256) {
        const int64_t l = base + threadIdx.x;
        const int32_t f = (l < N && cl[l] == c) ? 1 : 0;
        const int32_t inc = block_incl_scan(f, s);
        if (f) members[pos + inc - 1] = (int32_t)l;
        pos += s[255];   // s still holds the scan: the block total
        __syncthreads();
    }
}

// cen[c] = round(127 sum / |sum|) over the cluster's members (one workgroup per cluster; an empty
// cluster or a zero sum keeps its centre)
__global__ __launch_bounds__(256) void k_gl_centroid(const int8_t *__restrict__ E, int D,
                                                     const int32_t *__restrict__ members,
                                                     const int32_t *__restrict__ start, int8_t *__restrict__ cen) {
    __shared__ long long red[256];
    const int c = blockIdx.x;
    const int32_t m0 = start[c], m1 = start[c + 1];
    if (m1 == m0) return;   // workgroup-uniform
    int32_t sum[kGlMaxD / 256];
#pragma unroll
    for (int t = 0; t < kGlMaxD / 256; ++t) sum[t] = 0;
    for (int32_t m = m0; m < m1; ++m) {
        const int8_t *e = E + (int64_t)members[m] * D;
#pragma unroll
        for (int t = 0; t < kGlMaxD / 256; ++t) {
            const int d = threadIdx.x + 256 * t;
            if (d < D) sum[t] += e[d];
        }
    }
    long long ss = 0;
#pragma unroll
    for (int t = 0; t < kGlMaxD / 256; ++t) ss += (long long)sum[t] * sum[t];
    red[threadIdx.x] = ss;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    const long long tot = red[0];
    if (tot == 0) return;   // workgroup-uniform
    const double norm = sqrt((double)tot);
#pragma unroll
    for (int t = 0; t < kGlMaxD / 256; ++t) {
        const int d = threadIdx.x + 256 * t;
        if (d < D) {
            double qv = rint(127.0 * (double)sum[t] / norm);
            qv = qv > 127.0 ? 127.0 : (qv < -127.0 ? -127.0 : qv);
            cen[(int64_t)c * D + d] = (int8_t)qv;
        }
    }
}

// Greedy groups inside each cluster (one workgroup per cluster): seed = the (out(N + c N + t) mod
// nu)-th unassigned member in ascending order; the group = its top-k unassigned members by
// similarity (k = min(G, nu), ties to the lower label), listed in ascending label order.
__global__ __launch_bounds__(256) void k_gl_greedy(const int8_t *__restrict__ E, int64_t N, int D,
                                                   const int32_t *__restrict__ members,
                                                   const int32_t *__restrict__ start,
                                                   const int32_t *__restrict__ gstart, int64_t G, uint64_t seed,
                                                   uint8_t *__restrict__ taken, int32_t *__restrict__ sims,
                                                   int32_t *__restrict__ order, int32_t *__restrict__ gsize) {
    __shared__ int32_t s[256];
    __shared__ long long rv[256];
    __shared__ int32_t sel[256];
    __shared__ int32_t bc;
    const int c = blockIdx.x;
    const int32_t m0 = start[c], n = start[c + 1] - m0;
    int32_t g = gstart[c], pos = m0;
    for (int32_t i = threadIdx.x; i < n; i += 256) taken[m0 + i] = 0;
    __syncthreads();
    for (int64_t t = 0, nu = n; nu > 0; ++t) {
        // the seed: the r-th unassigned member, by a block scan over the members in order
        const int64_t r = (int64_t)(splitmix64_at(seed, (uint64_t)(N + (int64_t)c * N + t)) % (uint64_t)nu);
        int32_t before = 0;
        if (threadIdx.x == 0) bc = -1;
        __syncthreads();
        for (int32_t base = 0; base < n; base += 256) {
            const int32_t i = base + threadIdx.x;
            const int32_t f = (i < n && !taken[m0 + i]) ? 1 : 0;
            const int32_t inc = block_incl_scan(f, s);
            if (f && before + inc - 1 == r) bc = members[m0 + i];
            before += s[255];
            __syncthreads();
            if (bc >= 0) break;   // workgroup-uniform after the barrier
        }
        if (bc < 0) break;   // cannot happen (r < nu unassigned members); never index E with it
        const int8_t *es = E + (int64_t)bc * D;
        // similarities of the unassigned members to the seed (exact integer dot products)
        for (int32_t i = threadIdx.x; i < n; i += 256) {
            if (taken[m0 + i]) continue;
            const int8_t *e = E + (int64_t)members[m0 + i] * D;
            int32_t acc = 0;
            for (int d = 0; d < D; d += 4)
                acc = __builtin_amdgcn_sdot4(*reinterpret_cast<const int32_t *>(e + d),
                                             *reinterpret_cast<const int32_t *>(es + d), acc, false);
            sims[m0 + i] = acc;
        }
        __syncthreads();
        // top-k by repeated block argmax (larger similarity, then lower label)
        const int32_t k = (int32_t)(nu < G ? nu : G);
        for (int32_t j = 0; j < k; ++j) {
            long long best = LLONG_MIN;
            for (int32_t i = threadIdx.x; i < n; i += 256) {
                if (taken[m0 + i]) continue;
                // key: similarity high, label low (labels < 2^31, similarities fit 32 bits)
                const long long key = (long long)sims[m0 + i] * 4294967296LL + (long long)(0x7FFFFFFF - members[m0 + i]);
                if (key > best) best = key;
            }
            rv[threadIdx.x] = best;
            __syncthreads();
            for (int off = 128; off > 0; off >>= 1) {
                if (threadIdx.x < off && rv[threadIdx.x + off] > rv[threadIdx.x]) rv[threadIdx.x] = rv[threadIdx.x + off];
                __syncthreads();
            }
            const int32_t lab = 0x7FFFFFFF - (int32_t)(rv[0] & 0xFFFFFFFFll);
            if (threadIdx.x == 0) sel[j] = lab;
            for (int32_t i = threadIdx.x; i < n; i += 256)
                if (members[m0 + i] == lab) taken[m0 + i] = 1;
            __syncthreads();
        }
        // the group, ascending (insertion sort of at most G <= 256 labels)
        if (threadIdx.x == 0) {
            for (int32_t i = 1; i < k; ++i) {
                const int32_t v = sel[i];
                int32_t j = i - 1;
                while (j >= 0 && sel[j] > v) {
                    sel[j + 1] = sel[j];
                    --j;
                }
                sel[j + 1] = v;
            }
            gsize[g] = k;
        }
        __syncthreads();
        for (int32_t i = threadIdx.x; i < k; i += 256) order[pos + i] = sel[i];
        __syncthreads();
        pos += k;
        ++g;
        nu -= k;
    }
}

}  // namespace

namespace haste {

bool group_supported(int64_t N, int64_t D, int64_t G) {
    // N < 2^24 keeps a cluster's int32 sums of unit int8 rows (|e| ~ 127) and their int64 squared
    // norm exact
    return N > 0 && N < ((int64_t)1 << 24) && D > 0 && D % 16 == 0 && D <= kGlMaxD && G >= 1 && G <= 256 &&
           N * D < ((int64_t)1 << 31);
}

static int64_t gl_clusters(int64_t N, int64_t G, int64_t beta) {
    const int64_t C = N / (beta * G);
    return C < 1 ? 1 : C;
}

size_t group_ws(int64_t N, int64_t D, int64_t G, int64_t beta) {
    const int64_t C = gl_clusters(N, G, beta);
    return (size_t)(round_up(N * 4, 256) * 4 + round_up(N, 256) + round_up(C * D, 256) + round_up((C + 1) * 4, 256) * 3 +
                    256);
}

hipError_t group_labels(int64_t N, int64_t D, const int8_t *E, int64_t G, int64_t beta, int64_t iters, uint64_t seed,
                        int32_t *order, int32_t *gsize, int64_t *n_groups, int32_t *cluster, void *ws, hipStream_t s) {
    const int64_t C = gl_clusters(N, G, beta);
    char *p = static_cast<char *>(ws);
    auto take = [&](int64_t bytes) {
        char *q = p;
        p += round_up(bytes, 256);
        return q;
    };
    int32_t *a = reinterpret_cast<int32_t *>(take(N * 4));
    int32_t *cl = cluster ? cluster : reinterpret_cast<int32_t *>(take(N * 4));
    if (cluster) take(N * 4);
    int32_t *members = reinterpret_cast<int32_t *>(take(N * 4));
    int32_t *sims = reinterpret_cast<int32_t *>(take(N * 4));
    uint8_t *taken = reinterpret_cast<uint8_t *>(take(N));
    int8_t *cen = reinterpret_cast<int8_t *>(take(C * D));
    int32_t *cnt = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    int32_t *start = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    int32_t *gstart = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    const int Di = (int)D;
    hipLaunchKernelGGL(k_gl_iota, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s, a, N);
    hipLaunchKernelGGL(k_gl_shuffle, dim3(1), dim3(64), 0, s, a, N, C, seed);
    hipLaunchKernelGGL(k_gl_pick_centres, dim3((unsigned)cdiv(C * D, 256)), dim3(256), 0, s, E, a, C, Di, cen);
    const dim3 ga((unsigned)cdiv(N, 16 * kGlWaves));
    auto assign_and_collect = [&]() {
        hipLaunchKernelGGL(k_gl_assign, ga, dim3(64 * kGlWaves), 0, s, E, N, Di, cen, C, cl);
        hipLaunchKernelGGL(k_gl_zero, dim3((unsigned)cdiv(C, 256)), dim3(256), 0, s, cnt, C);
        hipLaunchKernelGGL(k_gl_count, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s, cl, N, cnt);
        hipLaunchKernelGGL(k_gl_starts, dim3(1), dim3(256), 0, s, cnt, C, G, start, gstart, n_groups);
        hipLaunchKernelGGL(k_gl_collect, dim3((unsigned)C), dim3(256), 0, s, cl, N, start, members);
    };
    for (int64_t it = 0; it < iters; ++it) {
        assign_and_collect();
        hipLaunchKernelGGL(k_gl_centroid, dim3((unsigned)C), dim3(256), 0, s, E, Di, members, start, cen);
    }
    assign_and_collect();
    hipLaunchKernelGGL(k_gl_greedy, dim3((unsigned)C), dim3(256), 0, s, E, N, Di, members, start, gstart, G, seed,
                       taken, sims, order, gsize);
    return hipGetLastError();
}

}  // namespace haste
