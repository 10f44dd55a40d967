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
// groups.  Each wave owns one (group, 32-label tile) unit at a time: it gathers the group's
// support columns straight from the slab into A-operand registers (gathered once per unit and
// batch tile, shared by the tile's 32 labels through the MFMA N dimension), takes the labels'
// weights as the B operand in their natural row layout, and writes bf16 logits.  The next
// unit's indices and weights are loaded while the current one computes.  The nbt workgroups of
// one stream (one per batch tile) carry the same blockIdx % 8, so they run on one XCD and W is
// fetched from HBM about once per stream.
// Orientation: Z = H_k W_k^T (M = batch rows, N = labels, K = support slots).
// --------------------------------------------------------------------------------------------
template <int F_IN, bool HAS_BIAS>
struct FwdUnit {
    int4 fi[F_IN / 8];     // support indices, this lane's half of every 16-slot K-step
    uint4 w[F_IN / 16];    // weights of this lane's label, same slots
    float bias;            // bias of this lane's label
};

template <int BT, int F_IN, bool HAS_BIAS>
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
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int nwaves = nthr >> 6;
    const int ln = lane & 31;
    const int hh = lane >> 5;
    const int ntn = (G + 31) >> 5;
    const int64_t u_begin = stream * gps * ntn;
    const int64_t g_end = (stream + 1) * gps < K ? (stream + 1) * gps : K;
    const int64_t u_end = g_end * ntn;
    constexpr int KS = F_IN / 16;   // MFMA K-steps over the support slots
    constexpr int NT = BT / 32;     // MFMA N-tiles over the batch rows

    auto issue = [&](int64_t u, FwdUnit<F_IN, HAS_BIAS> &f) {
        const int64_t k = u / ntn;
        const int tile = (int)(u - k * ntn);
        const int col = tile * 32 + ln;
        const int32_t *ip = idx + k * F_IN + 8 * hh;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            f.fi[2 * s] = *reinterpret_cast<const int4 *>(ip + 16 * s);
            f.fi[2 * s + 1] = *reinterpret_cast<const int4 *>(ip + 16 * s + 4);
        }
        // weights of the group (labels past G read as zero)
        const Buf wb(W + k * G * F_IN, (uint32_t)(G * F_IN * 2));
#pragma unroll
        for (int s = 0; s < KS; ++s) f.w[s] = wb.ld16((uint32_t)((col * F_IN + 8 * hh + 16 * s) * 2));
        if (HAS_BIAS) {
            const Buf bb(bias + k * G, (uint32_t)(G * 4));
            f.bias = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(bb.r, (int)(col * 4), 0, 0));
        }
    };

    // one unit: gather H_k for this tile from the slab, MFMA against the labels' weights, store.
    // Orientation Z = H_k W_k^T (M = batch rows, N = labels, K = slots): the result lane (label,
    // hh) holds rows 8i + 4hh + j, so one 2-byte store instruction writes 64 contiguous bytes in
    // each of just two rows.  (Memory instructions that span many rows of the [B, L] logits, which
    // are megabytes apart, are limited by address translation, not by HBM.)
    auto compute = [&](int64_t u, const FwdUnit<F_IN, HAS_BIAS> &cu) {
        const int64_t k = u / ntn;
        const int tile = (int)(u - k * ntn);
        f32x16_t acc[NT];
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[n] = f32x16_t{0};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            const int fa[8] = {cu.fi[2 * s].x, cu.fi[2 * s].y, cu.fi[2 * s].z, cu.fi[2 * s].w,
                               cu.fi[2 * s + 1].x, cu.fi[2 * s + 1].y, cu.fi[2 * s + 1].z, cu.fi[2 * s + 1].w};
#pragma unroll
            for (int n = 0; n < NT; ++n) {
                // gather: A[m = row][k = slot] = X[b0 + 32n + ln][idx[k, slot]]
                const bf16_t *row = xs + (n * 32 + ln) * S16;
                uint4 av;
                av.x = pack2(row[fa[0]], row[fa[1]]);
                av.y = pack2(row[fa[2]], row[fa[3]]);
                av.z = pack2(row[fa[4]], row[fa[5]]);
                av.w = pack2(row[fa[6]], row[fa[7]]);
                acc[n] = mfma32x32x16(as_bf16x8(av), as_bf16x8(cu.w[s]), acc[n]);
            }
        }
        // D[m = row 8i + 4hh + j][n = label ln]; rows past B fall outside the buffer, labels past G
        // are sent out of range
        const int64_t lab0 = k * G + tile * 32;
        const int rows = B - b0 < BT ? B - b0 : BT;
        const Buf yb(Y + (int64_t)b0 * L + lab0, (uint32_t)((int64_t)rows * L * 2));
        const bool ok = tile * 32 + ln < G;
        const float bv = HAS_BIAS ? cu.bias : 0.0f;
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = n * 32 + 8 * i + 4 * hh + j;
                    const uint32_t off = (uint32_t)(((int64_t)r * L + ln) * 2);
                    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(acc[n][4 * i + j] + bv), yb.r,
                                                          (int)(ok ? off : kOob), 0, 0);
                }
    };

    // Two units in flight per wave in ping-pong buffers (no register copies).  A wave takes two
    // consecutive 32-label tiles at a time, so both halves of each 128-byte line of a Y row are
    // written by the same wave back to back.  Prefetches are issued unconditionally (the index
    // is clamped to the last unit) so that every wait only covers the loads it needs.
    FwdUnit<F_IN, HAS_BIAS> ua, ub;
    const int64_t st = 2 * nwaves;
    const int64_t last = u_end - 1;
    auto cl = [&](int64_t v) { return v < last ? v : last; };
    int64_t u = u_begin + 2 * wave;
    if (u > last) return;
    issue(u, ua);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    issue(cl(u + 1), ub);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    for (; u <= last; u += st) {
        compute(u, ua);
        issue(cl(u + st), ua);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
        if (u + 1 <= last) compute(u + 1, ub);
        issue(cl(u + st + 1), ub);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    }
}

// --------------------------------------------------------------------------------------------
// Backward-weight.  One wave per (group, 32-label tile), contracting over the whole batch in
// blocks of 32 rows, so dW is formed in one pass on the support slots only.
// A = dY^T block (labels x rows): dY is read in its natural layout (16 bytes = 8 labels of one
// row per lane) and transposed through the matrix core (identity operand, exact).
// B = H_k (rows x slots): gathered from rows of X^T (staged by k_transpose_x), 8 bytes per load.
// The next block's loads are issued before the current block computes.
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

template <int NT>
struct BwdWBlock {
    uint2 dy[4];        // dY[row][label block], natural layout, as two 16-label halves
    uint2 x[NT][2][2];  // X^T gathers: [slot tile][K-step][half]
};


template <int F_IN>
__global__ __launch_bounds__(256) void k_bwd_w(const bf16_t *__restrict__ Xt, const int32_t *__restrict__ idx,
                                               const bf16_t *__restrict__ dY, float *__restrict__ dW,
                                               float *__restrict__ dbias, int beta, int B, int Bp, int64_t L,
                                               int G, int64_t K) {
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ln = lane & 31, hh = lane >> 5;
    const int mtiles = (G + 31) >> 5;
    const int64_t unit = (int64_t)blockIdx.x * 4 + wave;
    if (unit >= K * mtiles) return;
    const int64_t k = unit / mtiles;
    const int mt = (int)(unit - k * mtiles);
    const int c0 = mt * 32;                 // first label of the tile within the group
    const int64_t lab0 = k * G + c0;
    constexpr int NT = F_IN / 32;           // N-tiles over the support slots

    const bf16_t *xrow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) xrow[nt] = Xt + (int64_t)idx[k * F_IN + nt * 32 + ln] * Bp + 4 * hh;
    // natural dY load of this lane: row ln of the block, labels c0 + 8hh + 16s' + {0..3, 4..7}
    bool lab_ok[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) lab_ok[q] = c0 + 8 * hh + 16 * (q >> 1) + 4 * (q & 1) < G;

    auto issue = [&](int b0, BwdWBlock<NT> &blk) {
        // rows past B fall outside the buffer, labels past G are sent out of range; a block past
        // the end of the batch reads all zeros (its X^T reads stay inside the padded rows)
        const int rows = B - b0 < 32 ? (B - b0 > 0 ? B - b0 : 0) : 32;
        const Buf db(dY + (int64_t)b0 * L + lab0, (uint32_t)((int64_t)rows * L * 2));
        const uint32_t rowoff = (uint32_t)((int64_t)ln * L * 2) + 16 * hh;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            blk.dy[q] = db.ld8(lab_ok[q] ? rowoff + 32 * (q >> 1) + 8 * (q & 1) : kOob);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    blk.x[nt][s][h] = *reinterpret_cast<const uint2 *>(xrow[nt] + (b0 < Bp ? b0 : Bp - 32) + 16 * s + 8 * h);
    };

    const bf16x8_t e0 = eye_operand(ln, hh, 0), e16 = eye_operand(ln, hh, 16);
    f32x16_t acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x16_t{0};
    float dsum = 0.0f;

    auto compute = [&](const BwdWBlock<NT> &cb) {
        // transpose the 32x32 dY block: D[m = row][n = label], lane (label ln, hh) holds rows 8i+4hh+j
        f32x16_t d = f32x16_t{0};
        d = mfma32x32x16(as_bf16x8(make_uint4(cb.dy[0].x, cb.dy[0].y, cb.dy[1].x, cb.dy[1].y)), e0, d);
        d = mfma32x32x16(as_bf16x8(make_uint4(cb.dy[2].x, cb.dy[2].y, cb.dy[3].x, cb.dy[3].y)), e16, d);
        if (dbias) {
#pragma unroll
            for (int r = 0; r < 16; ++r) dsum += d[r];
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            // K-slot 8hh + q  <->  row b0 + 16s + 8(q/4) + 4hh + q%4  (registers 8s .. 8s+7)
            const bf16x8_t a = as_bf16x8(pack8(d, 8 * s));
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const uint4 bx = make_uint4(cb.x[nt][s][0].x, cb.x[nt][s][0].y, cb.x[nt][s][1].x, cb.x[nt][s][1].y);
                acc[nt] = mfma32x32x16(a, as_bf16x8(bx), acc[nt]);
            }
        }
    };

    // blocks in ping-pong buffers, two 32-row blocks in flight
    // Two 32-row blocks per iteration in ping-pong buffers; every load and every compute is
    // unconditional (blocks past the batch are all-zero), so each wait covers only its own loads.
    BwdWBlock<NT> ba, bb;
    issue(0, ba);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    issue(32, bb);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    for (int b0 = 0; b0 < B; b0 += 64) {
        compute(ba);
        issue(b0 + 64, ba);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
        compute(bb);
        issue(b0 + 96, bb);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    }
    // D[m = label 8i + 4hh + j][n = slot ln] -> dW[lab0 + m][nt*32 + ln]
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int m = 8 * i + 4 * hh + j;
                if (c0 + m < G) {
                    float *p = dW + (lab0 + m) * F_IN + nt * 32 + ln;
                    const float v = acc[nt][4 * i + j];
                    *p = beta ? *p + v : v;
                }
            }
    if (dbias) {
        // lanes (ln, 0) and (ln, 1) hold the two halves of label c0 + ln's row sum
        dsum += __shfl_xor(dsum, 32);
        if (hh == 0 && c0 + ln < G) dbias[lab0 + ln] = beta ? dbias[lab0 + ln] + dsum : dsum;
    }
}

// --------------------------------------------------------------------------------------------
// Backward-feature (split over label segments).  A workgroup owns a 32-row batch tile and one
// contiguous segment of groups; its partial dX^T[F_s][32] (fp32, rows padded to 36 floats)
// lives in LDS.  All waves of the workgroup work on the same group at the same time, each on a
// disjoint 16-slot x 16-row tile of dZ_k W_k.  The features of one group are distinct, so the
// tiles of one group update disjoint accumulator cells and plain (non-atomic) read-add-write is
// race free; one barrier per group orders consecutive groups.  This keeps every accumulation in
// fp32 in a fixed order (bit-reproducible) and avoids LDS float atomics, which run at a small
// fraction of the LDS rate on gfx950.
// Per tile (v_mfma_f32_16x16x32_bf16, M = rows, N = slots, K = labels):
//   B operand (labels x slots) = W_k rows in their natural layout, turned into slot-major
//     registers by two identity MFMAs (exact, see eye16_operand);
//   A operand (rows x labels) = dY rows, two 8-byte loads per 32-label chunk;
//   result lane (slot, q) holds rows 4q..4q+3 of one slot: one float4 read-add-write into the
//   accumulator row idx[k, slot].
// The tile products of the next group are computed before the barrier and the loads run two
// groups ahead (ping-pong buffers, unconditional prefetch with a clamped group index).
// --------------------------------------------------------------------------------------------
typedef float f32x4v_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4v_t mfma16x16x32(const bf16x8_t &a, const bf16x8_t &b, const f32x4v_t &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// identity slice for the 16x16x32 transpose: B[k][n] = (k == n), lane (n = l%16, q = l/16) holds k = 8q..8q+7
__device__ __forceinline__ bf16x8_t eye16_operand(int l16, int q) {
    uint32_t w[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const int k = 8 * q + 2 * p;
        w[p] = (l16 == k ? 0x3F80u : 0u) | (l16 == k + 1 ? 0x3F800000u : 0u);
    }
    return as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
}

template <int NLB>
struct BwdXTile {
    uint4 w[NLB][2];   // W[kG + 32c + 16h + l16][16st + 8q .. +7] (q < 2), natural layout
    uint2 dy[NLB][2];  // dY[row][kG + 32c + 16h + 4q .. +3]
    int f;             // accumulator row idx[k, 16st + l16]
};

template <int F_IN, int NLB>
__global__ __launch_bounds__(512) void k_bwd_x(const int32_t *__restrict__ idx, const bf16_t *__restrict__ W,
                                               const bf16_t *__restrict__ dY, float *__restrict__ part, int B,
                                               int Bp, int F_s, int64_t L, int G, int64_t K, int nbt,
                                               int64_t gps) {
    extern __shared__ __align__(16) float accs[];  // [F_s][AS]
    constexpr int AS = 36;
    constexpr int NT = (F_IN / 16) * 2;            // tiles per group: slot tiles x two 16-row halves
    constexpr int NWV = NT < 8 ? NT : 8;           // waves
    constexpr int TPW = NT / NWV;                  // tiles per wave
    const int w = blockIdx.x;
    const int xcd = w % kXcds;
    const int jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;

    for (int e = tid; e < F_s * AS; e += NWV * 64) accs[e] = 0.0f;
    __syncthreads();

    const int64_t g_begin = seg * gps;
    const int64_t g_end = g_begin + gps < K ? g_begin + gps : K;
    if (g_begin >= g_end) {
        // empty segment: the partial is zero
        float *pp = part + (size_t)seg * F_s * Bp + b0;
        for (int e = tid; e < F_s * 32; e += NWV * 64) pp[(size_t)(e >> 5) * Bp + (e & 31)] = 0.0f;
        return;
    }
    const int64_t lastk = g_end - 1;
    auto cl = [&](int64_t v) { return v < lastk ? v : lastk; };

    int st[TPW], bh[TPW];
    int64_t drows[TPW];   // valid rows of this tile's 16-row half
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int t = wave + NWV * i;
        st[i] = t >> 1;
        bh[i] = t & 1;
        const int r = B - (b0 + 16 * bh[i]);
        drows[i] = r < 0 ? 0 : (r > 16 ? 16 : r);
    }

    auto issue = [&](int64_t k, BwdXTile<NLB> (&tl)[TPW]) {
        // group k's weights: labels past G read as zero; lanes q >= 2 hold K-slots past the
        // tile's 16 slots and are sent out of range
        const Buf wb(W + k * G * F_IN, (uint32_t)(G * F_IN * 2));
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            // rows past B fall outside the buffer, labels past G are sent out of range
            const Buf db(dY + (int64_t)(b0 + 16 * bh[i]) * L + k * G, (uint32_t)(drows[i] * L * 2));
#pragma unroll
            for (int c = 0; c < NLB; ++c)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int lab = 32 * c + 16 * h + l16;
                    const uint32_t woff = (uint32_t)((lab * F_IN + 16 * st[i] + 8 * q) * 2);
                    tl[i].w[c][h] = wb.ld16(q < 2 ? woff : kOob);
                    const int c4 = 32 * c + 16 * h + 4 * q;   // 4 labels c4..c4+3 of the group
                    tl[i].dy[c][h] = db.ld8(c4 < G ? (uint32_t)((int64_t)l16 * L * 2) + 2 * c4 : kOob);
                }
            // a relaxed atomic load is not sunk towards its use (the scatter, two steps later), so it
            // stays in the prefetch batch
            tl[i].f = __hip_atomic_load(idx + k * F_IN + 16 * st[i] + l16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    };

    const bf16x8_t eye = eye16_operand(l16, q);
    auto compute = [&](const BwdXTile<NLB> (&tl)[TPW], f32x4v_t (&pr)[TPW], int (&ad)[TPW]) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            f32x4v_t acc = f32x4v_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < NLB; ++c) {
                // W chunk transposed: lane (slot l16, q) holds labels 32c + 4q + j and 32c + 16 + 4q + j
                const f32x4v_t d0 = mfma16x16x32(as_bf16x8(tl[i].w[c][0]), eye, f32x4v_t{0.f, 0.f, 0.f, 0.f});
                const f32x4v_t d1 = mfma16x16x32(as_bf16x8(tl[i].w[c][1]), eye, f32x4v_t{0.f, 0.f, 0.f, 0.f});
                const uint4 bo = make_uint4(pack_bf16(d0[0], d0[1]), pack_bf16(d0[2], d0[3]), pack_bf16(d1[0], d1[1]),
                                            pack_bf16(d1[2], d1[3]));
                // K-slot 8q + p  <->  label 32c + (p < 4 ? 4q + p : 16 + 4q + p - 4)
                const uint4 ao = make_uint4(tl[i].dy[c][0].x, tl[i].dy[c][0].y, tl[i].dy[c][1].x, tl[i].dy[c][1].y);
                acc = mfma16x16x32(as_bf16x8(ao), as_bf16x8(bo), acc);
            }
            pr[i] = acc;
            ad[i] = tl[i].f * AS + 16 * bh[i] + 4 * q;   // scatter address (floats)
        }
    };

    auto rmw = [&](const int (&ad)[TPW], const f32x4v_t (&pr)[TPW]) {
#pragma unroll
        for (int i = 0; i < TPW; ++i) {
            float4 *p = reinterpret_cast<float4 *>(accs + ad[i]);
            float4 v = *p;
            v.x += pr[i][0];
            v.y += pr[i][1];
            v.z += pr[i][2];
            v.w += pr[i][3];
            *p = v;
        }
    };

    // Two buffers in ping-pong (loop unrolled by two, as in the forward kernel): compute() turns a
    // buffer into registers (tile products and scatter addresses) and the buffer is refilled right
    // after, so loads get a full step to land and nothing loaded is carried across a refill.
    // Scatter order: group k - 1, then k, each behind one barrier.
    BwdXTile<NLB> ta[TPW], tb[TPW];
    f32x4v_t pa[TPW], pb[TPW];
    int aa[TPW], ab[TPW];
    issue(g_begin, ta);
    __builtin_amdgcn_sched_barrier(0);
    issue(cl(g_begin + 1), tb);
    __builtin_amdgcn_sched_barrier(0);
    for (int64_t k = g_begin; k <= lastk; k += 2) {
        compute(ta, pa, aa);                            // group k
        issue(cl(k + 2), ta);
        __builtin_amdgcn_sched_barrier(0);
        if (k > g_begin) {
            __syncthreads();
            rmw(ab, pb);                                // group k - 1
        }
        compute(tb, pb, ab);                            // group k + 1 (clamped past the end)
        issue(cl(k + 3), tb);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        rmw(aa, pa);                                    // group k
    }
    if (((g_end - g_begin) & 1) == 0) {
        __syncthreads();
        rmw(ab, pb);                                    // the last group
    }
    __syncthreads();
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    for (int e = tid; e < F_s * 32; e += NWV * 64) {
        const int f = e >> 5, b = e & 31;
        pp[(size_t)f * Bp + b] = accs[f * AS + b];
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
    int nbt, nwaves;
    int64_t nseg, gps;
    size_t lds;
};

BwdXGeom bwd_x_geom(const haste::TailArgs &a) {
    BwdXGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    const int nt = (int)(a.F_in / 16) * 2;
    g.nwaves = nt < 8 ? nt : 8;
    g.lds = (size_t)a.F_s * 36 * 4;
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
// The MFMA path needs bf16 storage, groups in multiples of 4 labels (8-byte label quads), a
// support of 32/64/128 slots and an even feature width that fits the LDS slab.
bool fwd_mfma_supported(const TailArgs &a) {
    return a.dtype == HASTE_DTYPE_BF16 && a.G >= 4 && (a.G % 4) == 0 &&
           (a.F_in == 32 || a.F_in == 64 || a.F_in == 128) && (a.F_s % 2) == 0 && a.F_s <= kMaxFs;
}

template <int BT, int F_IN, bool HAS_BIAS>
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
    auto kern = k_fwd<BT, F_IN, HAS_BIAS>;
    hipError_t e = allow_lds(kern, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(threads), lds, s, (const bf16_t *)X, idx, (const bf16_t *)W,
                       bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, S16, a.L, (int)a.G, K, nbt, gps);
    return hipGetLastError();
}

template <int BT, int F_IN>
static hipError_t launch_fwd_b(const TailArgs &a, const void *X, const int32_t *idx, const void *W,
                               const float *bias, void *Y, hipStream_t s) {
    return bias ? launch_fwd<BT, F_IN, true>(a, X, idx, W, bias, Y, s)
                : launch_fwd<BT, F_IN, false>(a, X, idx, W, bias, Y, s);
}

hipError_t fwd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s) {
    // 64-row slabs halve the weight re-reads once the batch is large enough
    const bool big = a.B > 32;
    switch (a.F_in) {
        case 32: return big ? launch_fwd_b<64, 32>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 32>(a, X, idx, W, bias, Y, s);
        case 64: return big ? launch_fwd_b<64, 64>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 64>(a, X, idx, W, bias, Y, s);
        case 128: return big ? launch_fwd_b<64, 128>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 128>(a, X, idx, W, bias, Y, s);
    }
    return hipErrorInvalidValue;
}

// ---- backward-weight ----------------------------------------------------------------------------
bool bwd_w_mfma_supported(const TailArgs &a) { return fwd_mfma_supported(a); }

// X^T staged with the batch padded to whole 32-row blocks
size_t bwd_w_mfma_ws(const TailArgs &a) { return (size_t)a.F_s * (size_t)round_up(a.B, 32) * 2 + 256; }

hipError_t bwd_w_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 32);
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
// Groups of up to 128 labels (four 32-label blocks held in registers per group).
bool bwd_x_mfma_supported(const TailArgs &a) {
    if (!fwd_mfma_supported(a) || a.G > 128) return false;
    return bwd_x_geom(a).lds <= kLdsBudget;
}

size_t bwd_x_mfma_ws(const TailArgs &a) {
    BwdXGeom g = bwd_x_geom(a);
    return (size_t)g.nseg * (size_t)a.F_s * (size_t)(g.nbt * 32) * 4 + 256;
}

template <int F_IN, int NLB>
static hipError_t launch_bwd_x(const TailArgs &a, const BwdXGeom &g, const int32_t *idx, const void *W,
                               const void *dY, float *part, hipStream_t s) {
    auto kern = k_bwd_x<F_IN, NLB>;
    hipError_t e = allow_lds(kern, g.lds);
    if (e != hipSuccess) return e;
    const int64_t K = a.L / a.G;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(g.nwaves * 64), g.lds, s, idx,
                       (const bf16_t *)W, (const bf16_t *)dY, part, (int)a.B, g.nbt * 32, (int)a.F_s, a.L, (int)a.G,
                       K, g.nbt, g.gps);
    return hipGetLastError();
}

template <int F_IN>
static hipError_t launch_bwd_x_g(const TailArgs &a, const BwdXGeom &g, const int32_t *idx, const void *W,
                                 const void *dY, float *part, hipStream_t s) {
    switch ((a.G + 31) / 32) {
        case 1: return launch_bwd_x<F_IN, 1>(a, g, idx, W, dY, part, s);
        case 2: return launch_bwd_x<F_IN, 2>(a, g, idx, W, dY, part, s);
        case 3: return launch_bwd_x<F_IN, 3>(a, g, idx, W, dY, part, s);
        case 4: return launch_bwd_x<F_IN, 4>(a, g, idx, W, dY, part, s);
    }
    return hipErrorInvalidValue;
}

hipError_t bwd_x_mfma(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s) {
    const BwdXGeom g = bwd_x_geom(a);
    float *part = reinterpret_cast<float *>(ws);
    hipError_t e;
    switch (a.F_in) {
        case 32: e = launch_bwd_x_g<32>(a, g, idx, W, dY, part, s); break;
        case 64: e = launch_bwd_x_g<64>(a, g, idx, W, dY, part, s); break;
        case 128: e = launch_bwd_x_g<128>(a, g, idx, W, dY, part, s); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 32, a.B, a.F_s, dX, beta, s);
}

}  // namespace haste
