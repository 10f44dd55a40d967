// Semantic grouping of labels (Alg. 2): coarse spherical k-means into C = max(1, N / (beta G))
// clusters, then greedy groups inside each cluster: a random unassigned seed together with its
// top-(G - 1) unassigned neighbours by cosine similarity (Section 3.1, "Label Grouping").
// Embeddings are int8 (unit vectors x 127).  A centre is the direction of its members' sum s, kept
// exactly as an int32 vector; a label goes to the centre maximising e.s / |s| (the cosine up to the
// label's own norm), where e.s is an exact integer and |s| the correctly rounded square root of
// the exact |s|^2, and the quotient is one fp64 division.  The products e.s run on int8 MFMA: s is
// split into balanced base-256 digit planes, s = sum_p 256^p d_p with d_p in [-128, 127], and the
// planes' exact int32 products are recombined in int64.  Greedy similarities are the fp64 cosine
// (e_i.e_s) / sqrt(|e_i|^2 |e_s|^2) of exact integers.
// Draws: SplitMix64 (Steele, Lea and Flood, 2014) in counter form.
#include <cfloat>
#include <climits>

#include "common.hpp"

namespace {

typedef int i32x4_t __attribute__((ext_vector_type(4)));

constexpr int kGlPlanes = 4;   // |s| < 2^31 (N < 2^24 members of |e_d| <= 127) needs four digits

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

// Centre c is the direction of the int32 vector s_c (a label's embedding at the start, then the
// sum of its members).  The assignment reads it as digit planes cp[p][c][D] (s_c = sum_p 256^p
// cp[p][c]), the number of planes it needs cnp[c] (higher planes are zero), and its norm cn[c].
constexpr int kGlWaves = 8;
constexpr int kGlMaxD = 1024;
constexpr int kGlThreads = 256;

// Writes centre c from the int32 vector held by the workgroup (sum[t] = s[threadIdx.x + 256 t]):
// the exact |s|^2 (128-bit), its correctly rounded square root, the digit planes and their count.
// A zero vector leaves the centre as it was (the caller's "keep" rule).  Workgroup-uniform.
__device__ void gl_store_centre(const int32_t (&sum)[kGlMaxD / kGlThreads], int D, int64_t C, int c,
                                int32_t *__restrict__ cs, int8_t *__restrict__ cp, double *__restrict__ cn,
                                int32_t *__restrict__ cnp) {
    __shared__ unsigned __int128 red[kGlThreads];
    __shared__ int32_t rmax[kGlThreads];
    uint64_t q = 0;   // at most four squares below 2^62 each: exact in 64 bits
    int need = 1;
#pragma unroll
    for (int t = 0; t < kGlMaxD / kGlThreads; ++t) {
        const int d = threadIdx.x + kGlThreads * t;
        if (d < D) {
            q += (uint64_t)((int64_t)sum[t] * (int64_t)sum[t]);
            int32_t r = sum[t];
            for (int p = 0; p < kGlPlanes && r != 0; ++p) {
                const int32_t dp = (int32_t)(int8_t)(r & 0xFF);   // balanced digit in [-128, 127]
                r = (r - dp) / 256;                                // exact
                need = p + 1 > need ? p + 1 : need;
            }
        }
    }
    red[threadIdx.x] = q;
    rmax[threadIdx.x] = need;
    __syncthreads();
    for (int off = kGlThreads / 2; off > 0; off >>= 1) {
        if (threadIdx.x < off) {
            red[threadIdx.x] += red[threadIdx.x + off];
            rmax[threadIdx.x] = rmax[threadIdx.x] > rmax[threadIdx.x + off] ? rmax[threadIdx.x] : rmax[threadIdx.x + off];
        }
        __syncthreads();
    }
    const unsigned __int128 tot = red[0];
    const int np = rmax[0];
    __syncthreads();   // red and rmax may be reused by the caller's next centre
    if (tot == 0) return;
#pragma unroll
    for (int t = 0; t < kGlMaxD / kGlThreads; ++t) {
        const int d = threadIdx.x + kGlThreads * t;
        if (d < D) {
            int32_t r = sum[t];
            cs[(int64_t)c * D + d] = r;
            for (int p = 0; p < kGlPlanes; ++p) {
                const int32_t dp = (int32_t)(int8_t)(r & 0xFF);
                r = (r - dp) / 256;
                cp[((int64_t)p * C + c) * D + d] = (int8_t)dp;
            }
        }
    }
    if (threadIdx.x == 0) {
        cn[c] = sqrt((double)tot);   // one rounding of the exact integer, one correctly rounded root
        cnp[c] = np;
    }
}

// initial centres: the embeddings of labels a[0 .. C) (one workgroup per centre)
__global__ __launch_bounds__(kGlThreads) void k_gl_pick_centres(const int8_t *__restrict__ E,
                                                                const int32_t *__restrict__ a, int64_t C, int D,
                                                                int32_t *__restrict__ cs, int8_t *__restrict__ cp,
                                                                double *__restrict__ cn, int32_t *__restrict__ cnp) {
    const int c = blockIdx.x;
    const int8_t *e = E + (int64_t)a[c] * D;
    int32_t sum[kGlMaxD / kGlThreads];
#pragma unroll
    for (int t = 0; t < kGlMaxD / kGlThreads; ++t) {
        const int d = threadIdx.x + kGlThreads * t;
        sum[t] = d < D ? (int32_t)e[d] : 0;
    }
    gl_store_centre(sum, D, C, c, cs, cp, cn, cnp);
}

// cl[l] = argmax_c (E[l].s_c) / |s_c| (ties: the lower c).  A wave takes 16 labels, a workgroup of
// 8 waves 128; centres pass through LDS 16 at a time, as many digit planes as the 16 need.
// v_mfma_i32_16x16x64_i8, M = 16 labels, N = 16 centres, K = 64 dimensions: both operands hold,
// per lane, 16 consecutive dimensions (16 q .. 16 q + 15 of the 64-chunk) of their row, so each
// lane group contracts the same dimensions; result lane (centre l16, q) holds labels 4q .. 4q+3.
__global__ __launch_bounds__(64 * kGlWaves) void k_gl_assign(const int8_t *__restrict__ E, int64_t N, int D,
                                                             const int8_t *__restrict__ cp,
                                                             const double *__restrict__ cn,
                                                             const int32_t *__restrict__ cnp, int64_t C,
                                                             int32_t *__restrict__ cl) {
    __shared__ __align__(16) int8_t tile[kGlPlanes][16 * kGlMaxD];
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
    double bv[4];
    int bi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        bv[i] = -DBL_MAX;
        bi[i] = INT_MAX;
    }
    const Buf cb(cp, (uint32_t)(kGlPlanes * C * D));
    for (int64_t c0 = 0; c0 < C; c0 += 16) {
        int npt = 1;   // planes of the 16 centres (workgroup-uniform)
        for (int r = 0; r < 16 && c0 + r < C; ++r) npt = cnp[c0 + r] > npt ? cnp[c0 + r] : npt;
        __syncthreads();   // the previous tile is no longer read
        for (int p = 0; p < npt; ++p)
            for (int e = threadIdx.x; e < 16 * (D / 16); e += 64 * kGlWaves) {
                const int r = e / (D / 16), ch = e - r * (D / 16);
                const uint4 v = cb.ld16(c0 + r < C ? (uint32_t)(((int64_t)p * C + c0 + r) * D + 16 * ch) : kOob);
                *reinterpret_cast<uint4 *>(&tile[p][r * kGlMaxD + 16 * ch]) = v;
            }
        __syncthreads();
        i32x4_t acc[kGlPlanes];
#pragma unroll
        for (int p = 0; p < kGlPlanes; ++p) {
            acc[p] = i32x4_t{0, 0, 0, 0};
            if (p >= npt) continue;
#pragma unroll
            for (int kk = 0; kk < kGlMaxD / 64; ++kk) {
                if (kk >= nk) break;
                const int d0 = 64 * kk + 16 * q;
                const i32x4_t b = d0 < D ? *reinterpret_cast<const i32x4_t *>(&tile[p][l16 * kGlMaxD + d0])
                                         : i32x4_t{0, 0, 0, 0};
                acc[p] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[kk], b, acc[p], 0, 0, 0);
            }
        }
        const int c = (int)(c0 + l16);
        if (c < C) {
            const double nc = cn[c];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t dot = (int64_t)acc[0][i] + (int64_t)acc[1][i] * 256 + (int64_t)acc[2][i] * 65536 +
                                    (int64_t)acc[3][i] * 16777216;
                const double v = (double)dot / nc;
                // centres ascend per lane: ties keep the lower one; a lane's first centre is always
                // taken, so a label always gets a valid centre (even from NaN scores of zero rows)
                if (v > bv[i] || bi[i] == INT_MAX) {
                    bv[i] = v;
                    bi[i] = c;
                }
            }
        }
    }
    // best over the 16 lanes of each row group: larger value, then lower centre
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        for (int off = 1; off < 16; off <<= 1) {
            const double ov = __shfl_xor(bv[i], off, 64);
            const int oi = __shfl_xor(bi[i], off, 64);
            if (oi != INT_MAX && (bi[i] == INT_MAX || ov > bv[i] || (ov == bv[i] && oi < bi[i]))) {
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

// s_c = the sum of the cluster's members, exactly (one workgroup per cluster; an empty cluster, or
// one whose members sum to zero, keeps its centre)
__global__ __launch_bounds__(kGlThreads) void k_gl_centroid(const int8_t *__restrict__ E, int D, int64_t C,
                                                            const int32_t *__restrict__ members,
                                                            const int32_t *__restrict__ start,
                                                            int32_t *__restrict__ cs, int8_t *__restrict__ cp,
                                                            double *__restrict__ cn, int32_t *__restrict__ cnp) {
    const int c = blockIdx.x;
    const int32_t m0 = start[c], m1 = start[c + 1];
    if (m1 == m0) return;   // workgroup-uniform
    int32_t sum[kGlMaxD / kGlThreads];
#pragma unroll
    for (int t = 0; t < kGlMaxD / kGlThreads; ++t) sum[t] = 0;
    for (int32_t m = m0; m < m1; ++m) {
        const int8_t *e = E + (int64_t)members[m] * D;
#pragma unroll
        for (int t = 0; t < kGlMaxD / kGlThreads; ++t) {
            const int d = threadIdx.x + kGlThreads * t;
            if (d < D) sum[t] += e[d];
        }
    }
    gl_store_centre(sum, D, C, c, cs, cp, cn, cnp);
}

// |e|^2 of every label (exact integers below 2^24)
__global__ void k_gl_norms(const int8_t *__restrict__ E, int64_t N, int D, int32_t *__restrict__ nrm) {
    const int64_t l = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (l >= N) return;
    const int8_t *e = E + l * D;
    int32_t acc = 0;
    for (int d = 0; d < D; d += 4) {
        const int32_t w = *reinterpret_cast<const int32_t *>(e + d);
        acc = __builtin_amdgcn_sdot4(w, w, acc, false);
    }
    nrm[l] = acc;
}

// Greedy groups inside each cluster (one workgroup per cluster): the seed is the (out(N + c N + t)
// mod nu)-th unassigned member in ascending order; the group is the seed and its top-(k - 1)
// unassigned members by cosine to it (k = min(G, nu), ties to the lower label), listed in ascending
// label order.
__global__ __launch_bounds__(kGlThreads) void k_gl_greedy(const int8_t *__restrict__ E, int64_t N, int D,
                                                          const int32_t *__restrict__ members,
                                                          const int32_t *__restrict__ start,
                                                          const int32_t *__restrict__ gstart, int64_t G,
                                                          uint64_t seed, const int32_t *__restrict__ nrm,
                                                          uint8_t *__restrict__ taken, double *__restrict__ sims,
                                                          int32_t *__restrict__ order, int32_t *__restrict__ gsize) {
    __shared__ int32_t s[kGlThreads];
    __shared__ double rv[kGlThreads];
    __shared__ int32_t ri[kGlThreads];
    __shared__ int32_t sel[256];
    __shared__ int32_t bpos;
    const int c = blockIdx.x;
    const int32_t m0 = start[c], n = start[c + 1] - m0;
    int32_t g = gstart[c], pos = m0;
    for (int32_t i = threadIdx.x; i < n; i += kGlThreads) taken[m0 + i] = 0;
    __syncthreads();
    for (int64_t t = 0, nu = n; nu > 0; ++t) {
        // the seed: the r-th unassigned member, by a block scan over the members in order
        const int64_t r = (int64_t)(splitmix64_at(seed, (uint64_t)(N + (int64_t)c * N + t)) % (uint64_t)nu);
        int32_t before = 0;
        if (threadIdx.x == 0) bpos = -1;
        __syncthreads();
        for (int32_t base = 0; base < n; base += kGlThreads) {
            const int32_t i = base + threadIdx.x;
            const int32_t f = (i < n && !taken[m0 + i]) ? 1 : 0;
            const int32_t inc = block_incl_scan(f, s);
            if (f && before + inc - 1 == r) bpos = i;
            before += s[kGlThreads - 1];
            __syncthreads();
            if (bpos >= 0) break;   // workgroup-uniform after the barrier
        }
        if (bpos < 0) break;   // cannot happen (r < nu unassigned members); never index E with it
        const int32_t sp = bpos, bc = members[m0 + sp];
        const int8_t *es = E + (int64_t)bc * D;
        const int64_t ns = nrm[bc];
        // cosines of the other unassigned members to the seed
        for (int32_t i = threadIdx.x; i < n; i += kGlThreads) {
            if (taken[m0 + i] || i == sp) continue;
            const int32_t lab = members[m0 + i];
            const int8_t *e = E + (int64_t)lab * D;
            int32_t acc = 0;
            for (int d = 0; d < D; d += 4)
                acc = __builtin_amdgcn_sdot4(*reinterpret_cast<const int32_t *>(e + d),
                                             *reinterpret_cast<const int32_t *>(es + d), acc, false);
            sims[m0 + i] = (double)acc / sqrt((double)((int64_t)nrm[lab] * ns));
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            sel[0] = bc;
            taken[m0 + sp] = 1;
        }
        __syncthreads();
        // the other k - 1 by repeated block argmax (larger cosine, then lower member position,
        // i.e. lower label: members ascend)
        const int32_t k = (int32_t)(nu < G ? nu : G);
        for (int32_t j = 1; j < k; ++j) {
            double best = -DBL_MAX;
            int32_t bi = INT_MAX;
            for (int32_t i = threadIdx.x; i < n; i += kGlThreads) {
                if (taken[m0 + i]) continue;
                const double v = sims[m0 + i];
                if (bi == INT_MAX || v > best || (v == best && i < bi)) {   // any unassigned member first
                    best = v;
                    bi = i;
                }
            }
            rv[threadIdx.x] = best;
            ri[threadIdx.x] = bi;
            __syncthreads();
            for (int off = kGlThreads / 2; off > 0; off >>= 1) {
                if (threadIdx.x < off) {
                    const double ov = rv[threadIdx.x + off];
                    const int32_t oi = ri[threadIdx.x + off];
                    if (oi != INT_MAX &&
                        (ri[threadIdx.x] == INT_MAX || ov > rv[threadIdx.x] || (ov == rv[threadIdx.x] && oi < ri[threadIdx.x]))) {
                        rv[threadIdx.x] = ov;
                        ri[threadIdx.x] = oi;
                    }
                }
                __syncthreads();
            }
            if (threadIdx.x == 0) {
                // k <= nu, so an unassigned member exists and ri[0] < n; never index past it
                const int32_t pick = ri[0] < n ? ri[0] : 0;
                sel[j] = members[m0 + pick];
                taken[m0 + pick] = 1;
            }
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
        for (int32_t i = threadIdx.x; i < k; i += kGlThreads) order[pos + i] = sel[i];
        __syncthreads();
        pos += k;
        ++g;
        nu -= k;
    }
}

}  // namespace

namespace haste {

static int64_t gl_clusters(int64_t N, int64_t G, int64_t beta) {
    const int64_t C = N / (beta * G);
    return C < 1 ? 1 : C;
}

bool group_supported(int64_t N, int64_t D, int64_t G, int64_t beta) {
    // N < 2^24 keeps a cluster's int32 sums of int8 rows (|e_d| <= 127) exact and inside four
    // balanced base-256 digits; the digit planes (4 C D bytes) stay addressable by 32-bit offsets
    if (!(N > 0 && N < ((int64_t)1 << 24) && D > 0 && D % 16 == 0 && D <= kGlMaxD && G >= 1 && G <= 256 &&
          beta >= 1 && N * D < ((int64_t)1 << 31)))
        return false;
    return kGlPlanes * gl_clusters(N, G, beta) * D < ((int64_t)1 << 31);
}

size_t group_ws(int64_t N, int64_t D, int64_t G, int64_t beta) {
    const int64_t C = gl_clusters(N, G, beta);
    return (size_t)(round_up(N * 4, 256) * 4 + round_up(N * 8, 256) + round_up(N, 256) + round_up(C * D * 4, 256) +
                    round_up(kGlPlanes * C * D, 256) + round_up(C * 8, 256) + round_up((C + 1) * 4, 256) * 4 + 256);
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
    int32_t *nrm = reinterpret_cast<int32_t *>(take(N * 4));
    double *sims = reinterpret_cast<double *>(take(N * 8));
    uint8_t *taken = reinterpret_cast<uint8_t *>(take(N));
    int32_t *cs = reinterpret_cast<int32_t *>(take(C * D * 4));
    int8_t *cp = reinterpret_cast<int8_t *>(take(kGlPlanes * C * D));
    double *cn = reinterpret_cast<double *>(take(C * 8));
    int32_t *cnp = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    int32_t *cnt = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    int32_t *start = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    int32_t *gstart = reinterpret_cast<int32_t *>(take((C + 1) * 4));
    const int Di = (int)D;
    hipLaunchKernelGGL(k_gl_iota, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s, a, N);
    hipLaunchKernelGGL(k_gl_shuffle, dim3(1), dim3(64), 0, s, a, N, C, seed);
    hipLaunchKernelGGL(k_gl_pick_centres, dim3((unsigned)C), dim3(kGlThreads), 0, s, E, a, C, Di, cs, cp, cn, cnp);
    const dim3 ga((unsigned)cdiv(N, 16 * kGlWaves));
    auto assign_and_collect = [&]() {
        hipLaunchKernelGGL(k_gl_assign, ga, dim3(64 * kGlWaves), 0, s, E, N, Di, cp, cn, cnp, C, cl);
        hipLaunchKernelGGL(k_gl_zero, dim3((unsigned)cdiv(C, 256)), dim3(256), 0, s, cnt, C);
        hipLaunchKernelGGL(k_gl_count, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s, cl, N, cnt);
        hipLaunchKernelGGL(k_gl_starts, dim3(1), dim3(256), 0, s, cnt, C, G, start, gstart, n_groups);
        hipLaunchKernelGGL(k_gl_collect, dim3((unsigned)C), dim3(256), 0, s, cl, N, start, members);
    };
    for (int64_t it = 0; it < iters; ++it) {
        assign_and_collect();
        hipLaunchKernelGGL(k_gl_centroid, dim3((unsigned)C), dim3(kGlThreads), 0, s, E, Di, C, members, start, cs, cp,
                           cn, cnp);
    }
    assign_and_collect();
    hipLaunchKernelGGL(k_gl_norms, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s, E, N, Di, nrm);
    hipLaunchKernelGGL(k_gl_greedy, dim3((unsigned)C), dim3(kGlThreads), 0, s, E, N, Di, members, start, gstart, G,
                       seed, nrm, taken, sims, order, gsize);
    return hipGetLastError();
}

}  // namespace haste
