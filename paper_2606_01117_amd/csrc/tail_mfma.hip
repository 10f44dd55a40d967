// Group-shared fixed fan-in tail on bf16 MFMA (gfx950, v_mfma_f32_32x32x16_bf16).
//
// The three products of the paper's Section 3.2, each run per label group k (labels kG..kG+G-1,
// support idx[k, 0..F_in-1]):
//   forward          Z_k  = H_k W_k^T            H_k = X[:, idx[k, :]]   (M = batch, N = labels, K = slots)
//   backward-weight  dW_k = dZ_k^T H_k                                   (M = labels, N = slots, K = batch)
//   backward-feature dH_k = dZ_k W_k, scattered to X's columns idx[k,:] (M = slots,  N = batch,  K = labels)
// Every contraction is a small dense GEMM once the group's support columns are gathered, which is
// what makes the group-shared format MFMA-friendly (one gather serves all G labels).
#include "common.hpp"

namespace {

constexpr int kSlabPadDw = 1;  // LDS row padding of the X slab (keeps row strides an odd dword count)

// --------------------------------------------------------------------------------------------
// Forward.
// A workgroup keeps BT rows of X resident in LDS (the "slab") and sweeps a contiguous stream of
// groups.  Each wave owns one group at a time: it gathers the group's support columns straight
// from the slab into A-operand registers (gathered once per group and batch tile, shared by all
// G labels through the MFMA N dimension), streams the group's weights as the B operand and
// writes bf16 logits.  The nbt workgroups of one stream (one per batch tile) carry the same
// blockIdx % 8, so they run on one XCD and W is fetched from HBM about once per stream.
// --------------------------------------------------------------------------------------------
template <int BT, int F_IN>
__global__ __launch_bounds__(512) void k_fwd(const bf16_t *__restrict__ X, const int32_t *__restrict__ idx,
                                             const bf16_t *__restrict__ W, const float *__restrict__ bias,
                                             bf16_t *__restrict__ Y, int B, int F_s, int S16, int64_t L, int G,
                                             int64_t K, int nbt, int64_t gps) {
    extern __shared__ __align__(16) bf16_t xs[];
    const int w = blockIdx.x;
    const int xcd = w % kXcds;
    const int jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t stream = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * BT;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;

    // slab: rows b0 .. b0+BT-1 of X, zero rows past B (F_s is even: copy in bf16 pairs)
    {
        const int half = F_s >> 1;
        const uint32_t *X32 = reinterpret_cast<const uint32_t *>(X);
        uint32_t *xs32 = reinterpret_cast<uint32_t *>(xs);
        const int rs32 = S16 >> 1;
        for (int e = tid; e < BT * half; e += nthr) {
            const int r = e / half, c = e - r * half;
            const int b = b0 + r;
            xs32[r * rs32 + c] = (b < B) ? X32[(int64_t)b * half + c] : 0u;
        }
    }
    __syncthreads();

    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int nwaves = nthr >> 6;
    const int ln = lane & 31;
    const int hh = lane >> 5;
    const int64_t g_begin = stream * gps;
    const int64_t g_end = g_begin + gps < K ? g_begin + gps : K;
    const int ntn = (G + 31) >> 5;
    constexpr int KS = F_IN / 16;   // MFMA K-steps over the support slots
    constexpr int MT = BT / 32;     // MFMA M-tiles over the batch rows

    for (int64_t k = g_begin + wave; k < g_end; k += nwaves) {
        // this lane's support slots: t = 16*s + 8*hh + i
        int32_t fi[KS * 8];
        const int32_t *ip = idx + k * F_IN + 8 * hh;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int4 v0 = *reinterpret_cast<const int4 *>(ip + 16 * s);
            const int4 v1 = *reinterpret_cast<const int4 *>(ip + 16 * s + 4);
            fi[8 * s + 0] = v0.x; fi[8 * s + 1] = v0.y; fi[8 * s + 2] = v0.z; fi[8 * s + 3] = v0.w;
            fi[8 * s + 4] = v1.x; fi[8 * s + 5] = v1.y; fi[8 * s + 6] = v1.z; fi[8 * s + 7] = v1.w;
        }
        // gather H_k (this batch tile) once into A-operand registers
        uint4 a[MT][KS];
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const bf16_t *row = xs + (m * 32 + ln) * S16;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                a[m][s].x = pack2(row[fi[8 * s + 0]], row[fi[8 * s + 1]]);
                a[m][s].y = pack2(row[fi[8 * s + 2]], row[fi[8 * s + 3]]);
                a[m][s].z = pack2(row[fi[8 * s + 4]], row[fi[8 * s + 5]]);
                a[m][s].w = pack2(row[fi[8 * s + 6]], row[fi[8 * s + 7]]);
            }
        }
        for (int nt = 0; nt < ntn; ++nt) {
            const int col = nt * 32 + ln;  // label within the group
            const bool valid = col < G;
            const int64_t lab = k * G + col;
            uint4 wv[KS];
            const bf16_t *wp = W + lab * F_IN + 8 * hh;
#pragma unroll
            for (int s = 0; s < KS; ++s)
                wv[s] = valid ? *reinterpret_cast<const uint4 *>(wp + 16 * s) : make_uint4(0, 0, 0, 0);
            f32x16_t acc[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                acc[m] = f32x16_t{0};
#pragma unroll
                for (int s = 0; s < KS; ++s) acc[m] = mfma32x32x16(as_bf16x8(a[m][s]), as_bf16x8(wv[s]), acc[m]);
            }
            if (valid) {
                const float bv = bias ? bias[lab] : 0.0f;
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            const int b = b0 + m * 32 + 8 * i + 4 * hh + j;
                            if (b < B) Y[(int64_t)b * L + lab] = f32_to_bf16(acc[m][4 * i + j] + bv);
                        }
            }
        }
    }
}

// --------------------------------------------------------------------------------------------
// Backward-weight.  One wave per (group, 32-label tile): A = dY^T column block (labels x batch,
// read as 2-byte loads down the batch), B = H_k gathered from X^T rows (16-byte loads, X^T is
// staged by k_transpose_x), K runs over the whole batch so dW is formed in one pass, on the
// support slots only.
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_transpose_x(const bf16_t *__restrict__ X, bf16_t *__restrict__ Xt,
                                                     int B, int Bp, int F_s) {
    __shared__ bf16_t tile[32][33];
    const int f0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    for (int r = ty; r < 32; r += 8) {
        const int b = b0 + r, f = f0 + tx;
        tile[r][tx] = (b < B && f < F_s) ? X[(int64_t)b * F_s + f] : (bf16_t)0;
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
        const int f = f0 + r, b = b0 + tx;
        if (f < F_s && b < Bp) Xt[(int64_t)f * Bp + b] = tile[tx][r];
    }
}

template <int F_IN>
__global__ __launch_bounds__(256) void k_bwd_w(const bf16_t *__restrict__ Xt, const int32_t *__restrict__ idx,
                                               const bf16_t *__restrict__ dY, float *__restrict__ dW,
                                               float *__restrict__ dbias, int beta, int B, int Bp, int64_t L,
                                               int G, int64_t K) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ln = lane & 31, hh = lane >> 5;
    const int mtiles = (G + 31) >> 5;
    const int64_t unit = (int64_t)blockIdx.x * 4 + wave;
    if (unit >= K * mtiles) return;
    const int64_t k = unit / mtiles;
    const int mt = (int)(unit - k * mtiles);
    const int r = mt * 32 + ln;       // A-operand row: label within the group
    const bool valid = r < G;
    const int64_t lab = k * G + (valid ? r : 0);
    constexpr int NT = F_IN / 32;     // N-tiles over the support slots

    const bf16_t *xrow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) xrow[nt] = Xt + (int64_t)idx[k * F_IN + nt * 32 + ln] * Bp + 8 * hh;

    f32x16_t acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x16_t{0};
    float dsum = 0.0f;
    const bf16_t *dyp = dY + lab;

#pragma unroll 2
    for (int b0 = 0; b0 < B; b0 += 16) {
        bf16_t v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int b = b0 + 8 * hh + i;
            v[i] = (valid && b < B) ? dyp[(int64_t)b * L] : (bf16_t)0;
        }
        uint4 av;
        av.x = pack2(v[0], v[1]);
        av.y = pack2(v[2], v[3]);
        av.z = pack2(v[4], v[5]);
        av.w = pack2(v[6], v[7]);
        if (dbias) {
#pragma unroll
            for (int i = 0; i < 8; ++i) dsum += bf16_to_f32(v[i]);
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const uint4 bx = *reinterpret_cast<const uint4 *>(xrow[nt] + b0);
            acc[nt] = mfma32x32x16(as_bf16x8(av), as_bf16x8(bx), acc[nt]);
        }
    }
    // D[m = 8i + 4hh + j][n = ln] -> dW[k*G + mt*32 + m][nt*32 + ln]
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int m = mt * 32 + 8 * i + 4 * hh + j;
                if (m < G) {
                    float *p = dW + (k * G + m) * F_IN + nt * 32 + ln;
                    const float v = acc[nt][4 * i + j];
                    *p = beta ? *p + v : v;
                }
            }
    if (dbias) {
        dsum += __shfl_xor(dsum, 32);
        if (hh == 0 && valid) dbias[lab] = beta ? dbias[lab] + dsum : dsum;
    }
}

// --------------------------------------------------------------------------------------------
// Backward-feature (split over label segments).  A workgroup owns a 32-row batch tile and one
// contiguous segment of groups; its partial dX^T[F_s][32] (fp32) lives in LDS.  Each wave takes
// one group at a time: W_k is staged transposed in a wave-private LDS tile (A operand: slots x
// labels), dY rows feed the B operand directly (labels are contiguous in dY), and the MFMA
// result dZ_k W_k (slots x batch) is scattered into the LDS accumulator rows idx[k, t].  The 32
// lanes holding one slot write 32 consecutive floats, so the scatter is bank-conflict free up to
// the two half-waves.  At the end the partial goes to ws[seg][F_s][Bp]; a fixed-order reduction
// over segments produces dX.
// --------------------------------------------------------------------------------------------
template <int F_IN, bool GVEC>
__global__ __launch_bounds__(512) void k_bwd_x(const int32_t *__restrict__ idx, const bf16_t *__restrict__ W,
                                               const bf16_t *__restrict__ dY, float *__restrict__ part, int B,
                                               int Bp, int F_s, int64_t L, int G, int64_t K, int nbt, int64_t gps,
                                               int WTS) {
    extern __shared__ __align__(16) char smem[];
    float *accs = reinterpret_cast<float *>(smem);                       // [F_s][32]
    bf16_t *wt_all = reinterpret_cast<bf16_t *>(smem + (size_t)F_s * 32 * 4);
    const int w = blockIdx.x;
    const int xcd = w % kXcds;
    const int jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x, nthr = blockDim.x;
    const int lane = tid & 63, wave = tid >> 6, nwaves = nthr >> 6;
    const int ln = lane & 31, hh = lane >> 5;

    for (int e = tid; e < F_s * 32; e += nthr) accs[e] = 0.0f;
    __syncthreads();

    bf16_t *wt = wt_all + (size_t)wave * F_IN * WTS;
    const int ksteps = (G + 15) >> 4;
    const int kpad = ksteps * 16;
    const int64_t g_begin = seg * gps;
    const int64_t g_end = g_begin + gps < K ? g_begin + gps : K;
    const int brow = b0 + ln;
    const bool brow_ok = brow < B;
    constexpr int MT = F_IN / 32;
    constexpr int CPR = F_IN / 8;  // 16-byte chunks per weight row

    for (int64_t k = g_begin + wave; k < g_end; k += nwaves) {
        // stage W_k^T: wt[t][l] = W[kG + l][t]
        const bf16_t *wk = W + k * G * F_IN;
        for (int c = lane; c < G * CPR; c += 64) {
            const int l = c / CPR, t0 = (c - l * CPR) * 8;
            const uint4 v = *reinterpret_cast<const uint4 *>(wk + (int64_t)l * F_IN + t0);
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                wt[(t0 + 2 * q) * WTS + l] = (bf16_t)(u[q] & 0xffffu);
                wt[(t0 + 2 * q + 1) * WTS + l] = (bf16_t)(u[q] >> 16);
            }
        }
        if (!GVEC) {
            const int padw = kpad - G;
            for (int c = lane; c < F_IN * padw; c += 64) {
                const int t = c / padw, l = G + (c - t * padw);
                wt[t * WTS + l] = 0;
            }
        }
        // B operand: dY[b0 + ln][kG + 16s + 8hh .. +7] (labels are contiguous in dY)
        const bf16_t *dp = dY + (int64_t)brow * L + k * G + 8 * hh;
        auto load_dy = [&](int s) -> uint4 {
            if (GVEC) return brow_ok ? *reinterpret_cast<const uint4 *>(dp + 16 * s) : make_uint4(0, 0, 0, 0);
            bf16_t e[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int l = 16 * s + 8 * hh + i;
                e[i] = (brow_ok && l < G) ? dp[16 * s + i] : (bf16_t)0;
            }
            return make_uint4(pack2(e[0], e[1]), pack2(e[2], e[3]), pack2(e[4], e[5]), pack2(e[6], e[7]));
        };
        uint4 dv[4];  // up to 4 K-steps (G <= 64) stay in registers; larger groups reload per step
#pragma unroll
        for (int s = 0; s < 4; ++s) dv[s] = (s < ksteps) ? load_dy(s) : make_uint4(0, 0, 0, 0);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            f32x16_t acc = f32x16_t{0};
            const bf16_t *arow = wt + (mt * 32 + ln) * WTS + 8 * hh;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                if (s < ksteps) {
                    const uint4 av = *reinterpret_cast<const uint4 *>(arow + 16 * s);
                    acc = mfma32x32x16(as_bf16x8(av), as_bf16x8(dv[s]), acc);
                }
            }
            for (int s = 4; s < ksteps; ++s) {
                const uint4 av = *reinterpret_cast<const uint4 *>(arow + 16 * s);
                acc = mfma32x32x16(as_bf16x8(av), as_bf16x8(load_dy(s)), acc);
            }
            // D[m = slot mt*32 + 8i + 4hh + j][n = batch ln] -> accs[idx[k, slot]][ln]
            const int32_t *ip = idx + k * F_IN + mt * 32 + 4 * hh;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int4 f4 = *reinterpret_cast<const int4 *>(ip + 8 * i);
                const int fv[4] = {f4.x, f4.y, f4.z, f4.w};
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    __hip_atomic_fetch_add(accs + fv[j] * 32 + ln, acc[4 * i + j], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
        // the next group's staging overwrites wt: every lane must be done reading it
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    __syncthreads();
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    for (int e = tid; e < F_s * 32; e += nthr) {
        const int f = e >> 5, b = e & 31;
        pp[(size_t)f * Bp + b] = accs[e];
    }
}

// ---------------------------------------------------------------------------------------------
// launch geometry
// ---------------------------------------------------------------------------------------------
int slab_s16(int F_s) {
    int dw = (F_s + 1) / 2;
    if ((dw & 1) == 0) dw += kSlabPadDw;
    return 2 * dw;
}

constexpr size_t kLdsBudget = 160 * 1024;

template <typename Kern>
hipError_t allow_lds(Kern k, size_t bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

struct BwdXGeom {
    int nbt, nwaves, WTS;
    int64_t nseg, gps;
    size_t lds;
};

BwdXGeom bwd_x_geom(const haste::TailArgs &a) {
    BwdXGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    const int ksteps = (int)haste::cdiv(a.G, 16);
    g.WTS = ksteps * 16 + 8;
    const size_t acc = (size_t)a.F_s * 32 * 4;
    const size_t per_wave = (size_t)a.F_in * g.WTS * 2;
    int nw = 8;
    while (nw > 1 && acc + nw * per_wave > kLdsBudget - 8 * 1024) --nw;
    g.nwaves = nw;
    g.lds = acc + nw * per_wave;
    const int64_t K = a.L / a.G;
    int64_t spx = kCusPerXcd / g.nbt;  // one workgroup per CU: the accumulator takes most of the LDS
    if (spx < 1) spx = 1;
    const int64_t max_spx = haste::cdiv(K, kXcds);
    if (spx > max_spx) spx = max_spx < 1 ? 1 : max_spx;
    g.nseg = spx * kXcds;
    g.gps = haste::cdiv(K, g.nseg);
    return g;
}

}  // namespace

namespace haste {

// ---- forward ----------------------------------------------------------------------------------
bool fwd_mfma_supported(const TailArgs &a) {
    return a.dtype == HASTE_DTYPE_BF16 && a.G >= 4 && (a.F_in == 32 || a.F_in == 64 || a.F_in == 128) &&
           (a.F_s % 2) == 0 && a.F_s <= kMaxFs;
}

template <int BT, int F_IN>
static hipError_t launch_fwd(const TailArgs &a, const void *X, const int32_t *idx, const void *W,
                             const float *bias, void *Y, hipStream_t s) {
    const int S16 = slab_s16((int)a.F_s);
    const size_t lds = (size_t)BT * S16 * 2;
    const int threads = BT == 64 ? 512 : 256;
    const int occ = (int)(kLdsBudget / lds) < 1 ? 1 : (int)(kLdsBudget / lds);
    const int occ_eff = BT == 64 ? 1 : (occ > 3 ? 3 : occ);
    const int nbt = (int)cdiv(a.B, BT);
    const int64_t K = a.L / a.G;
    int64_t spx = (int64_t)kCusPerXcd * occ_eff / nbt;
    if (spx < 1) spx = 1;
    const int64_t max_spx = cdiv(K, kXcds);
    if (spx > max_spx) spx = max_spx < 1 ? 1 : max_spx;
    const int64_t nstream = spx * kXcds;
    const int64_t gps = cdiv(K, nstream);
    const int64_t grid = nstream * nbt;
    auto kern = k_fwd<BT, F_IN>;
    hipError_t e = allow_lds(kern, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(threads), lds, s, (const bf16_t *)X, idx, (const bf16_t *)W,
                       bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, S16, a.L, (int)a.G, K, nbt, gps);
    return hipGetLastError();
}

hipError_t fwd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s) {
    // 64-row slabs halve the weight re-reads once the batch is large enough; at F_in = 128 the
    // gathered operand of 64 rows no longer fits the register file, so those stay at 32 rows
    const bool big = a.B > 32 && a.F_in <= 64;
    switch (a.F_in) {
        case 32: return big ? launch_fwd<64, 32>(a, X, idx, W, bias, Y, s) : launch_fwd<32, 32>(a, X, idx, W, bias, Y, s);
        case 64: return big ? launch_fwd<64, 64>(a, X, idx, W, bias, Y, s) : launch_fwd<32, 64>(a, X, idx, W, bias, Y, s);
        case 128: return big ? launch_fwd<64, 128>(a, X, idx, W, bias, Y, s) : launch_fwd<32, 128>(a, X, idx, W, bias, Y, s);
    }
    return hipErrorInvalidValue;
}

// ---- backward-weight ----------------------------------------------------------------------------
bool bwd_w_mfma_supported(const TailArgs &a) { return fwd_mfma_supported(a); }

size_t bwd_w_mfma_ws(const TailArgs &a) { return (size_t)a.F_s * (size_t)round_up(a.B, 16) * 2 + 256; }

hipError_t bwd_w_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 16);
    bf16_t *Xt = reinterpret_cast<bf16_t *>(ws);
    hipLaunchKernelGGL(k_transpose_x, dim3((unsigned)cdiv(a.F_s, 32), (unsigned)cdiv(Bp, 32)), dim3(256), 0, s,
                       (const bf16_t *)X, Xt, (int)a.B, Bp, (int)a.F_s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t K = a.L / a.G;
    const int64_t units = K * cdiv(a.G, 32);
    const dim3 grid((unsigned)cdiv(units, 4));
    switch (a.F_in) {
        case 32:
            hipLaunchKernelGGL(k_bwd_w<32>, grid, dim3(256), 0, s, Xt, idx, (const bf16_t *)dY, dW, dbias, beta,
                               (int)a.B, Bp, a.L, (int)a.G, K);
            break;
        case 64:
            hipLaunchKernelGGL(k_bwd_w<64>, grid, dim3(256), 0, s, Xt, idx, (const bf16_t *)dY, dW, dbias, beta,
                               (int)a.B, Bp, a.L, (int)a.G, K);
            break;
        case 128:
            hipLaunchKernelGGL(k_bwd_w<128>, grid, dim3(256), 0, s, Xt, idx, (const bf16_t *)dY, dW, dbias, beta,
                               (int)a.B, Bp, a.L, (int)a.G, K);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---- backward-feature ---------------------------------------------------------------------------
bool bwd_x_mfma_supported(const TailArgs &a) {
    if (!fwd_mfma_supported(a)) return false;
    BwdXGeom g = bwd_x_geom(a);
    return g.lds <= kLdsBudget;
}

size_t bwd_x_mfma_ws(const TailArgs &a) {
    BwdXGeom g = bwd_x_geom(a);
    return (size_t)g.nseg * (size_t)a.F_s * (size_t)(g.nbt * 32) * 4 + 256;
}

template <int F_IN, bool GVEC>
static hipError_t launch_bwd_x(const TailArgs &a, const BwdXGeom &g, const int32_t *idx, const void *W,
                               const void *dY, float *part, hipStream_t s) {
    auto kern = k_bwd_x<F_IN, GVEC>;
    hipError_t e = allow_lds(kern, g.lds);
    if (e != hipSuccess) return e;
    const int64_t K = a.L / a.G;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(g.nwaves * 64), g.lds, s, idx,
                       (const bf16_t *)W, (const bf16_t *)dY, part, (int)a.B, g.nbt * 32, (int)a.F_s, a.L, (int)a.G,
                       K, g.nbt, g.gps, g.WTS);
    return hipGetLastError();
}

hipError_t bwd_x_mfma(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s) {
    const BwdXGeom g = bwd_x_geom(a);
    float *part = reinterpret_cast<float *>(ws);
    const bool gvec = (a.G % 16) == 0;
    hipError_t e;
    switch (a.F_in) {
        case 32: e = gvec ? launch_bwd_x<32, true>(a, g, idx, W, dY, part, s) : launch_bwd_x<32, false>(a, g, idx, W, dY, part, s); break;
        case 64: e = gvec ? launch_bwd_x<64, true>(a, g, idx, W, dY, part, s) : launch_bwd_x<64, false>(a, g, idx, W, dY, part, s); break;
        case 128: e = gvec ? launch_bwd_x<128, true>(a, g, idx, W, dY, part, s) : launch_bwd_x<128, false>(a, g, idx, W, dY, part, s); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 32, a.B, a.F_s, dX, beta, s);
}

}  // namespace haste
