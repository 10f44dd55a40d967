// Forward logits of the tail for small groups (G = 1, 2, 4, 8; bf16), on the matrix cores.
//
// Section 3.2's gather-once pays off in proportion to G: with a few labels per group, the work is
// the gather of X[:, I_k] for every group, and a 16- or 32-label matrix tile would sit mostly on
// one group's few labels.  Here one v_mfma_f32_16x16x32_bf16 tile covers 16 labels = 16 / G whole
// groups: its K = 32 positions are 2G slots of each of those groups, and the weight operand is
// block-diagonal (label n's weights sit only in the K positions of its own group; zeros
// elsewhere).  So each (group, slot, row) value is gathered exactly once, and the matrix core's
// extra zero products cost nothing that matters next to the gather.
//   M = 16 batch rows, N = 16 labels, K = 32 (group-slot pairs).
//   A (rows x K): gathered with ds_read_b64_tr_b16 from an X^T slab [F_s][32 rows] in LDS: source
//     lane 4j + a of each 16-lane group names K position 8q + j (and 8q + 4 + j) at rows 4a .. 4a+3,
//     so result lane (row l16, q) holds row l16 at K positions 8q .. 8q+7.
//   B (K x labels): lane (label n, q) holds K positions 8q .. 8q+7; the ones of n's group carry
//     W[n, slot], the others are zero.
//   D: lane (label n, q) holds rows 4q .. 4q+3 of label n.
// A workgroup of 8 waves keeps one 32-row slab of X^T for its whole segment of labels and sweeps it
// in passes of 128 labels (one 16-label tile per wave): the pass's supports and weights are staged
// in LDS (prefetched into registers during the previous pass), and its logits leave through LDS
// as 256-byte row runs.  The batch slabs of a segment run on one XCD, sharing W through its L2.

#include "common.hpp"

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kSgWaves = 8;
constexpr int kSgThreads = 64 * kSgWaves;
constexpr int kSgRows = 32;                     // batch rows per slab
constexpr int kSgXRow = 80;                     // bytes per staged X^T feature row (32 rows + pad)
constexpr int kSgPass = 16 * kSgWaves;          // labels per pass
constexpr int kSgOutRow = kSgPass * 2 + 16;     // bytes per staged output row (bf16 + pad)

__device__ __forceinline__ uint2 tr_read(const char *p) {
    return lds_read_tr(p);
}

template <int G, int F_IN>
struct SgGeom {
    static constexpr int PG = kSgPass / G;                      // groups per pass
    static constexpr int NS = F_IN / (2 * G);                   // K steps per tile
    static constexpr int IDX_BYTES = PG * F_IN * 4;             // staged supports per pass
    static constexpr int W_BYTES = kSgPass * F_IN * 2;          // staged weights per pass
    static constexpr int IC = IDX_BYTES / 16, WC = W_BYTES / 16;   // 16-byte chunks
    static constexpr int IL = (IC + kSgThreads - 1) / kSgThreads;  // prefetch loads per thread
    static constexpr int WL = (WC + kSgThreads - 1) / kSgThreads;
};

template <int G, int F_IN>
static size_t sg_lds(int F_s) {
    using S = SgGeom<G, F_IN>;
    return (size_t)F_s * kSgXRow + S::IDX_BYTES + S::W_BYTES + (size_t)kSgRows * kSgOutRow;
}

template <int G, int F_IN, bool HAS_BIAS>
__global__ __launch_bounds__(kSgThreads) void k_fwd_sg(const bf16_t *__restrict__ X, const int32_t *__restrict__ idx,
                                                       const bf16_t *__restrict__ W, const float *__restrict__ bias,
                                                       bf16_t *__restrict__ Y, int B, int F_s, int64_t L, int nbt,
                                                       int64_t pps, int64_t npass, const int32_t *__restrict__ spos,
                                                       int P) {
    using S = SgGeom<G, F_IN>;
    extern __shared__ __align__(16) char sgs[];
    char *xs = sgs;                                               // [F_s][kSgXRow]
    int32_t *sidx = reinterpret_cast<int32_t *>(sgs + (size_t)F_s * kSgXRow);   // [PG][F_IN]
    char *sw = reinterpret_cast<char *>(sidx) + S::IDX_BYTES;    // [128 labels][F_IN] bf16
    char *so = sw + S::W_BYTES;                                   // [32 rows][kSgOutRow]
    const int w = blockIdx.x, xcd = w % kXcds, jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int64_t p_begin = seg * pps, p_end = p_begin + pps < npass ? p_begin + pps : npass;
    if (p_begin >= p_end) return;   // workgroup-uniform
    const int b0 = bt * kSgRows;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;

    // the slab's X^T: 16-byte row pieces of X, scattered into feature rows (zero past B)
    {
        const int cpr = F_s / 8;   // 16-byte chunks per X row
        for (int c = tid; c < kSgRows * cpr; c += kSgThreads) {
            const int r = c / cpr, f8 = (c - r * cpr) * 8;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (b0 + r < B) v = *reinterpret_cast<const uint4 *>(X + (int64_t)(b0 + r) * F_s + f8);
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                *reinterpret_cast<bf16_t *>(xs + (f8 + e) * kSgXRow + r * 2) =
                    (bf16_t)((e & 1) ? (u[e >> 1] >> 16) : (u[e >> 1] & 0xffffu));
        }
    }

    // pass staging, prefetched into registers: supports of the pass's groups, weights of its labels
    uint4 pi[S::IL], pw[S::WL];
    auto fetch = [&](int64_t p) {
        const int64_t l0 = p * kSgPass;
        const int64_t g0 = l0 / G;
        const int64_t ng = (L - l0 < kSgPass ? L - l0 : kSgPass) / G;   // groups of the pass in the layer
        const Buf ib(idx + g0 * F_IN, (uint32_t)(ng * F_IN * 4));
        const Buf wb(W + l0 * F_IN, (uint32_t)(ng * G * F_IN * 2));
#pragma unroll
        for (int i = 0; i < S::IL; ++i) pi[i] = ib.ld16((uint32_t)(tid + kSgThreads * i) * 16);   // past: zero
#pragma unroll
        for (int i = 0; i < S::WL; ++i) pw[i] = wb.ld16((uint32_t)(tid + kSgThreads * i) * 16);
    };
    auto stage = [&]() {
#pragma unroll
        for (int i = 0; i < S::IL; ++i)
            if (tid + kSgThreads * i < S::IC)
                *reinterpret_cast<uint4 *>(reinterpret_cast<char *>(sidx) + (tid + kSgThreads * i) * 16) = pi[i];
#pragma unroll
        for (int i = 0; i < S::WL; ++i)
            if (tid + kSgThreads * i < S::WC) *reinterpret_cast<uint4 *>(sw + (tid + kSgThreads * i) * 16) = pw[i];
    };

    // this lane's roles: gather source (K position 8q + j, rows 4a ..) and weight operand window
    const int j = l16 >> 2, a = l16 & 3;
    const int klo = 8 * q + j, khi = klo + 4;
    const int n_grp = l16 / G;                       // this label's group within the tile
    // K positions of the label's group: [2G n_grp, 2G n_grp + 2G); this lane's octet [8q, 8q + 8)
    const int kg0 = 2 * G * n_grp;
    const bool wact = kg0 < 8 * q + 8 && kg0 + 2 * G > 8 * q;

    // the loss-gradient targets of this thread's output row, from the first window it stores
    PosCursor tgt;
    if (spos && b0 + (tid >> 4) < B) tgt.init(spos + (int64_t)(b0 + (tid >> 4)) * P, P, p_begin * kSgPass + 8 * (tid & 15));
    fetch(p_begin);
    for (int64_t p = p_begin; p < p_end; ++p) {
        __syncthreads();   // the previous pass's staging and output are no longer read
        stage();
        __syncthreads();
        if (p + 1 < p_end) fetch(p + 1);
        const int64_t l0 = p * kSgPass + 16 * wave;     // this wave's tile
        f32x4_t acc[2];
        {
            const float bv = HAS_BIAS && l0 + l16 < L ? bias[l0 + l16] : 0.0f;
            acc[0] = acc[1] = f32x4_t{bv, bv, bv, bv};
        }
        if (l0 < L) {   // wave-uniform
            const int32_t *ti = sidx + (16 * wave / G) * F_IN;    // the tile's groups' supports
            const char *tw = sw + (16 * wave + l16) * F_IN * 2;   // this lane's label's weights
#pragma unroll
            for (int s = 0; s < S::NS; ++s) {
                const int flo = ti[(klo / (2 * G)) * F_IN + s * 2 * G + klo % (2 * G)];
                const int fhi = ti[(khi / (2 * G)) * F_IN + s * 2 * G + khi % (2 * G)];
                uint4 bw = make_uint4(0u, 0u, 0u, 0u);
                if constexpr (G >= 4) {
                    // the whole octet is one group's: 8 consecutive slots
                    if (wact) bw = *reinterpret_cast<const uint4 *>(tw + (s * 2 * G + (8 * q) % (2 * G)) * 2);
                } else if constexpr (G == 2) {
                    // 4 slots of the label's group at octet position 0 or 4
                    if (wact) {
                        const uint2 v = *reinterpret_cast<const uint2 *>(tw + s * 4 * 2);
                        if (kg0 == 8 * q) bw = make_uint4(v.x, v.y, 0u, 0u);
                        else bw = make_uint4(0u, 0u, v.x, v.y);
                    }
                } else {
                    // 2 slots at octet position 0, 2, 4 or 6
                    if (wact) {
                        const uint32_t v = *reinterpret_cast<const uint32_t *>(tw + s * 2 * 2);
                        const int pos = (kg0 - 8 * q) >> 1;
                        bw = make_uint4(pos == 0 ? v : 0u, pos == 1 ? v : 0u, pos == 2 ? v : 0u, pos == 3 ? v : 0u);
                    }
                }
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    const uint2 lo = tr_read(xs + flo * kSgXRow + (16 * m + 4 * a) * 2);
                    const uint2 hi = tr_read(xs + fhi * kSgXRow + (16 * m + 4 * a) * 2);
                    acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)),
                                                                     as_bf16x8(bw), acc[m], 0, 0, 0);
                }
            }
        }
        // logits of rows 16m + 4q + r, label 16 wave + l16, into the pass's output block
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                *reinterpret_cast<bf16_t *>(so + (16 * m + 4 * q + r) * kSgOutRow + (16 * wave + l16) * 2) =
                    f32_to_bf16(acc[m][r]);
        __syncthreads();
        // 32 rows x 256 bytes: one 16-byte chunk per thread (16 chunks per row); with the positives,
        // the loss gradient of the rounded logits
        {
            const int r = tid >> 4, c = tid & 15;
            const int64_t lb = p * kSgPass + 8 * c;
            if (b0 + r < B && lb < L) {
                uint4 v = *reinterpret_cast<const uint4 *>(so + r * kSgOutRow + c * 16);
                if (spos) {   // kernel-uniform
                    const uint32_t t = tgt.bits(lb, 8);
                    v = make_uint4(bce_pair(v.x, t), bce_pair(v.y, t >> 2), bce_pair(v.z, t >> 4), bce_pair(v.w, t >> 6));
                }
                bf16_t *dst = Y + (int64_t)(b0 + r) * L + lb;
                if (lb + 8 <= L) {
                    __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v), reinterpret_cast<u32x4_t *>(dst));
                } else {
                    const uint32_t u[4] = {v.x, v.y, v.z, v.w};
                    for (int e = 0; lb + e < L; ++e) dst[e] = (bf16_t)((e & 1) ? (u[e >> 1] >> 16) : (u[e >> 1] & 0xffffu));
                }
            }
        }
    }
}

template <int G, int F_IN>
static hipError_t launch_fwd_sg(const haste::TailArgs &a, const void *X, const int32_t *idx, const void *W,
                                const float *bias, void *Y, hipStream_t s, const int32_t *spos, int P) {
    const size_t lds = sg_lds<G, F_IN>((int)a.F_s);
    const int nbt = (int)haste::cdiv(a.B, kSgRows);
    const int64_t npass = haste::cdiv(a.L, kSgPass);
    // one workgroup per CU (the slab and the pass staging take most of the LDS), each sweeping a
    // segment of passes; segments a multiple of the XCD count
    int64_t nseg = haste::round_up(haste::cdiv(kXcds * kCusPerXcd, nbt), kXcds);
    const int64_t max_seg = haste::round_up(npass, kXcds);
    if (nseg > max_seg) nseg = max_seg;
    const int64_t pps = haste::cdiv(npass, nseg);
    auto go = [&](auto kern) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, dim3((unsigned)(nseg * nbt)), dim3(kSgThreads), lds, s, (const bf16_t *)X, idx,
                           (const bf16_t *)W, bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, a.L, nbt, pps, npass, spos, P);
        return hipGetLastError();
    };
    return bias ? go(k_fwd_sg<G, F_IN, true>) : go(k_fwd_sg<G, F_IN, false>);
}

template <int G>
static hipError_t fwd_sg_g(const haste::TailArgs &a, const void *X, const int32_t *idx, const void *W,
                           const float *bias, void *Y, hipStream_t s, const int32_t *spos, int P) {
    switch (a.F_in) {
        case 32: return launch_fwd_sg<G, 32>(a, X, idx, W, bias, Y, s, spos, P);
        case 64: return launch_fwd_sg<G, 64>(a, X, idx, W, bias, Y, s, spos, P);
        case 128:
            if constexpr (G >= 2) return launch_fwd_sg<G, 128>(a, X, idx, W, bias, Y, s, spos, P);
            break;
    }
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------------------------
// Backward-weight for small groups (G = 1, 2, 4, 8), the same block-diagonal packing with K = rows:
// per tile of 16 labels (16 / G groups) and K step s, the M = 16 "slot lines" are slots
// s G .. s G + G - 1 of each of the tile's groups, and D[line][label] is kept where the line's
// group is the label's (the rest is the zero-weight side of the packing).
//   A (lines x rows) = X^T rows of the line's feature, rows 8q .. 8q+7: one 16-byte LDS read;
//   B (rows x labels) = dY, two ds_read_b64_tr_b16 per tile and slab (shared by every K step);
//   D: lane (label n, q) holds lines 4q .. 4q+3; for G >= 4 they are slots of n's group exactly
//     when 4q / G = n / G (4 consecutive slots), for G = 2 two of them are, for G = 1 one.
// A workgroup of 8 waves owns a span of 16 TPW * 8 labels (TPW tiles per wave, whose accumulators
// stay in registers for the whole batch; for G = 1 a pass covers 16 slots and the batch is swept
// once per pass) and sweeps the batch in 32-row slabs: per slab the X^T
// block (contiguous in the workspace copy) and the span's dY rows are staged in LDS, the next
// slab's arriving in registers meanwhile.  dbias is the same B operand against all-ones A.
// ---------------------------------------------------------------------------------------------
constexpr int kSwYPad = 32;                     // staged dY row padding (bytes)

// label tiles per wave, and K steps per pass over the batch: accumulators TPW * NSC * 4 <= 128
// registers (G = 1 sweeps the batch F_in / 16 times, 16 slots at a time)
__host__ __device__ constexpr int sw_tpw(int G, int F_in) {
    return G == 1 ? 2 : (32 * G / F_in < 4 ? 32 * G / F_in : 4);
}
__host__ __device__ constexpr int sw_nsc(int G, int F_in) {
    return F_in / G < 32 / sw_tpw(G, F_in) ? F_in / G : 32 / sw_tpw(G, F_in);
}
__host__ __device__ constexpr int sw_span(int G, int F_in) { return 16 * kSgWaves * sw_tpw(G, F_in); }

template <int G, int F_IN>
static size_t sw_lds(int F_s) {
    return (size_t)haste::round_up((int64_t)F_s * kSgXRow, 16) + (size_t)kSgRows * (sw_span(G, F_IN) * 2 + kSwYPad);
}

template <int G, int F_IN, bool WITH_DB>
__global__ __launch_bounds__(kSgThreads) void k_bwd_w_sg(const bf16_t *__restrict__ Xb, const int32_t *__restrict__ idx,
                                                         const bf16_t *__restrict__ dY, float *__restrict__ dW,
                                                         float *__restrict__ dbias, int beta, int B, int Bp, int F_s,
                                                         int64_t L) {
    constexpr int TPW = sw_tpw(G, F_IN);
    constexpr int SPAN = sw_span(G, F_IN);
    constexpr int NSW = sw_nsc(G, F_IN);           // K steps (slot-line tiles) per pass over the batch
    constexpr int NPASS = F_IN / G / NSW;          // passes (1 unless G = 1)
    constexpr int YR = SPAN * 2 + kSwYPad;         // staged dY row bytes
    constexpr int XL = kMaxFs * 4 / kSgThreads;    // 16-byte X^T loads per thread and slab (at most)
    constexpr int YC = SPAN / 8;                   // 16-byte dY chunks per row
    constexpr int YL = (kSgRows * YC + kSgThreads - 1) / kSgThreads;
    static_assert(TPW >= 1, "a wave needs a whole tile");
    extern __shared__ __align__(16) char sws[];
    char *xs = sws;
    char *ys = sws + ((F_s * kSgXRow + 15) & ~15);
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const int64_t K = L / G;
    const int64_t lab0 = (int64_t)blockIdx.x * SPAN;
    const int span = L - lab0 < SPAN ? (int)(L - lab0) : SPAN;

    int f[TPW][NSW];
    // this lane's slot-line features, per tile and K step of pass ps (groups past the layer: the last)
    auto features = [&](int ps) {
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const int64_t l0 = lab0 + 16 * (TPW * wave + t);
            int64_t g = l0 / G + l16 / G;
            g = g < K ? g : K - 1;
#pragma unroll
            for (int s = 0; s < NSW; ++s) f[t][s] = idx[g * F_IN + (ps * NSW + s) * G + l16 % G];
        }
    };

    const int nxc = 4 * F_s;
    uint4 xr[XL], yr[YL];
    auto load = [&](int blk) {
        const Buf xb(Xb + (int64_t)blk * F_s * 32, (uint32_t)(nxc * 16));
#pragma unroll
        for (int i = 0; i < XL; ++i) xr[i] = xb.ld16((uint32_t)(tid + kSgThreads * i) * 16);   // past the block: zero
        const int b0 = blk * kSgRows;
        const int rows = B - b0 < kSgRows ? B - b0 : kSgRows;
        const Buf db(dY + (int64_t)b0 * L + lab0, (uint32_t)(rows > 0 ? ((int64_t)(rows - 1) * L + span) * 2 : 0));
#pragma unroll
        for (int i = 0; i < YL; ++i) {
            const int c = tid + kSgThreads * i, row = c / YC, part = c % YC;
            const bool ok = c < kSgRows * YC && row < rows && 8 * part < span;
            yr[i] = db.ld16(ok ? (uint32_t)(((int64_t)row * L + 8 * part) * 2) : kOob);
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int i = 0; i < XL; ++i) {
            const int c = tid + kSgThreads * i;
            if (c < nxc) *reinterpret_cast<uint4 *>(xs + (c >> 2) * kSgXRow + (c & 3) * 16) = xr[i];
        }
#pragma unroll
        for (int i = 0; i < YL; ++i) {
            const int c = tid + kSgThreads * i;
            if (c < kSgRows * YC) *reinterpret_cast<uint4 *>(ys + (c / YC) * YR + (c % YC) * 16) = yr[i];
        }
    };

    f32x4_t acc[TPW][NSW], db[TPW];
    const bf16x8_t ones = as_bf16x8(make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    // B-operand source lanes: 16-lane group q names rows 8q + (l16 >> 2) (+ 4), labels 4 (l16 & 3) ..
    const char *ysrc = ys + (8 * q + (l16 >> 2)) * YR + (l16 & 3) * 8;
    const int nblk = Bp / kSgRows;

    for (int ps = 0; ps < NPASS; ++ps) {
    features(ps);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        db[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NSW; ++s) acc[t][s] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    if (ps > 0) __syncthreads();   // the previous pass's last slab is no longer read
    load(0);
    for (int blk = 0; blk < nblk; ++blk) {
        __syncthreads();   // the previous slab is no longer read
        store();
        __syncthreads();
        if (blk + 1 < nblk) load(blk + 1);
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const char *p = ysrc + 16 * (TPW * wave + t) * 2;
            const uint2 lo = lds_read_tr(p);
            const uint2 hi = lds_read_tr(p + 4 * YR);
            const bf16x8_t bv = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
            for (int s = 0; s < NSW; ++s) {
                const uint4 av = *reinterpret_cast<const uint4 *>(xs + f[t][s] * kSgXRow + 16 * q);
                acc[t][s] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(av), bv, acc[t][s], 0, 0, 0);
            }
            if constexpr (WITH_DB) {
                if (ps == 0) db[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, bv, db[t], 0, 0, 0);
            }
        }
    }
    // the kept lines: G >= 4: lines 4q .. 4q+3 are slots (4q mod G) .. +3 of the K step when 4q / G
    // is the label's group; G = 2: lines r0, r0 + 1 (r0 = 2 (n / 2) - 4q) when that lies in [0, 4)
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int64_t l = lab0 + 16 * (TPW * wave + t) + l16;
        if (l >= L) continue;
        float *wr = dW + l * F_IN;
        if constexpr (G >= 4) {
            if ((4 * q) / G == l16 / G) {
#pragma unroll
                for (int s = 0; s < NSW; ++s) {
                    float4 *p = reinterpret_cast<float4 *>(wr + s * G + (4 * q) % G);
                    float4 v = make_float4(acc[t][s][0], acc[t][s][1], acc[t][s][2], acc[t][s][3]);
                    if (beta) {
                        const float4 o = *p;
                        v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
                    }
                    *p = v;
                }
            }
        } else if constexpr (G == 2) {
            const int r0 = 2 * (l16 / 2) - 4 * q;
            if (r0 >= 0 && r0 < 4) {
#pragma unroll
                for (int s = 0; s < NSW; ++s) {
                    float2 *p = reinterpret_cast<float2 *>(wr + 2 * s);
                    float2 v = r0 == 0 ? make_float2(acc[t][s][0], acc[t][s][1]) : make_float2(acc[t][s][2], acc[t][s][3]);
                    if (beta) {
                        const float2 o = *p;
                        v.x += o.x; v.y += o.y;
                    }
                    *p = v;
                }
            }
        } else {
            // G = 1: line l16 is label l16's slot of the K step, held by lane (l16, l16 / 4) at l16 % 4
            if (q == l16 / 4) {
                const int r0 = l16 & 3;
#pragma unroll
                for (int s = 0; s < NSW; ++s) {
                    float *p = wr + ps * NSW + s;
                    const float v = r0 == 0 ? acc[t][s][0] : r0 == 1 ? acc[t][s][1] : r0 == 2 ? acc[t][s][2] : acc[t][s][3];
                    *p = beta ? *p + v : v;
                }
            }
        }
        if constexpr (WITH_DB) {
            if (ps == 0 && q == 0) dbias[l] = (beta ? dbias[l] : 0.0f) + db[t][0];
        }
    }
    }   // passes
}

template <int G, int F_IN>
static hipError_t launch_bwd_w_sg(const haste::TailArgs &a, const void *Xb, const int32_t *idx, const void *dY,
                                  float *dW, float *dbias, int beta, int Bp, hipStream_t s) {
    const size_t lds = sw_lds<G, F_IN>((int)a.F_s);
    const dim3 grid((unsigned)haste::cdiv(a.L, sw_span(G, F_IN)));
    auto go = [&](auto kern) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, grid, dim3(kSgThreads), lds, s, (const bf16_t *)Xb, idx, (const bf16_t *)dY, dW,
                           dbias, beta, (int)a.B, Bp, (int)a.F_s, a.L);
        return hipGetLastError();
    };
    return dbias ? go(k_bwd_w_sg<G, F_IN, true>) : go(k_bwd_w_sg<G, F_IN, false>);
}

template <int G>
static hipError_t bwd_w_sg_g(const haste::TailArgs &a, const void *Xb, const int32_t *idx, const void *dY, float *dW,
                             float *dbias, int beta, int Bp, hipStream_t s) {
    switch (a.F_in) {
        case 32: return launch_bwd_w_sg<G, 32>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
        case 64: return launch_bwd_w_sg<G, 64>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
        case 128:
            if constexpr (G == 1 || G >= 4) return launch_bwd_w_sg<G, 128>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
            break;
    }
    return hipErrorInvalidValue;
}


// ---------------------------------------------------------------------------------------------
// Backward-feature for small groups (G = 1, 2, 4, 8; bf16):
//   dX^T[f][rows] = sum over groups k and slots t with idx[k, t] = f of
//                   sum over the labels l of group k of W[l, t] dY[rows, l]   (Section 3.2),
// as the general kernel computes it (per-segment partial dX^T in LDS, fixed-order reduction), but
// with 32 consecutive labels (a "super-group" of 32 / G groups) per matrix-core K step.
//   M = 16 rows, N = 16 slots of one group, K = the super-group's 32 labels in natural order.
//   A (rows x labels): the staged dY block, one 16-byte LDS read per super-group, shared by the
//     tiles of all of its groups.
//   B (labels x slots): group gi's labels are K positions G gi .. G gi + G - 1, inside the 8-label
//     octet q = G gi / 8; lane (slot l16, octet q) holds W[G gi + u][slot] (u < G) there and zeros
//     elsewhere, and every other lane holds zeros.  The pre-pass lays W out per super-group so
//     that the non-zero values one lane contributes over all of its tiles are F_in contiguous
//     bytes: per super-group a consumer wave reads the 32-label block exactly once.
//   D: lane (slot, q) holds rows 4q .. 4q + 3 of the slot, added into accumulator row idx[k, slot].
// The slots of one group are distinct features, so the 16 accumulator rows of a tile are distinct;
// the groups of a super-group can share features, so each group's accumulator reads follow the
// previous group's writes in the wave's LDS program order.
// ---------------------------------------------------------------------------------------------
constexpr int kBsConsumers = 2;                  // consumer waves (one per 16-row half)
constexpr int kBsProducers = 2;                  // producer waves (staging dY)
constexpr int kBsThreads = 64 * (kBsConsumers + kBsProducers);
// groups' supports in flight per consumer lane (16, at most 64 registers), and the weight blocks
// of the next two super-groups: the loads come from HBM for the first batch tile of a segment
__host__ __device__ constexpr int bs_idx_depth(int f_in) { return f_in <= 64 ? 16 : 8; }

__host__ __device__ constexpr int bs_row_bytes(int ch) { return ch * 64 + 32; }   // staged dY row
__host__ __device__ constexpr int bs_stage_bytes(int ch) { return 2 * 32 * bs_row_bytes(ch); }

// Pre-pass: per group (one wave each), its supports in lane order as accumulator row offsets
// (idxl, as the general kernel's)
// and its weights into the super-group block WS: lane (l16, q) of super-group n owns the F_in bytes
// at ((n 4 + q) 16 + l16) F_in, holding for each group gi of octet q (local index j = gi mod 8/G)
// and slot tile st the G weights of position 16 st + l16 at byte (j F_in / 16 + st) 2G.  Groups
// from K to the end of the last super-group are written as zeros.
constexpr int kBtWaves = 8;

__global__ __launch_bounds__(kBtWaves * 64) void k_transpose_w_sg(const bf16_t *__restrict__ W,
                                                                  const int32_t *__restrict__ idx,
                                                                  bf16_t *__restrict__ WS, int32_t *__restrict__ idxl,
                                                                  int64_t K, int64_t Kp, int G, int F_in) {
    __shared__ int pslot[kBtWaves][128];          // slot at each position
    __shared__ uint32_t wrow[kBtWaves][8 * 128 / 2];   // the group's weights [G][F_in] bf16
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int nst = F_in / 16, sg = 32 / G;
    const uint16_t *wr16 = reinterpret_cast<const uint16_t *>(wrow[wv]);
    for (int64_t k = (int64_t)blockIdx.x * kBtWaves + wv; k < Kp; k += (int64_t)gridDim.x * kBtWaves) {
        if (k < K) {   // wave-uniform
            // the group's G weight rows (contiguous), whole dwords, into LDS
            const uint32_t *src = reinterpret_cast<const uint32_t *>(W + k * G * F_in);
            for (int e = lane; e < G * F_in / 2; e += 64) wrow[wv][e] = src[e];
            int f[2], ps[2];
            slot_positions(idx + k * F_in, F_in, lane, f, ps);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                if (ps[i] < 0) continue;
                pslot[wv][ps[i]] = lane + 64 * i;
                idxl[k * F_in + (ps[i] & 15) * nst + (ps[i] >> 4)] = (int32_t)acc_row(f[i]);
            }
        }
        __builtin_amdgcn_wave_barrier();
        const int64_t n = k / sg;
        const int gi = (int)(k - n * sg);
        const int q = G * gi / 8, j = gi % (8 / G);
        for (int p = lane; p < F_in; p += 64) {
            const int l16 = p & 15, st = p >> 4;
            char *dst = reinterpret_cast<char *>(WS) + ((n * 4 + q) * 16 + l16) * F_in + (j * nst + st) * 2 * G;
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (k < K) {
                const int t = pslot[wv][p];
                for (int u = 0; u < G; ++u) {
                    const uint32_t w = wr16[u * F_in + t];
                    v[u >> 1] |= (u & 1) ? w << 16 : w;
                }
            }
            if (G == 8) *reinterpret_cast<uint4 *>(dst) = make_uint4(v[0], v[1], v[2], v[3]);
            else if (G == 4) *reinterpret_cast<uint2 *>(dst) = make_uint2(v[0], v[1]);
            else if (G == 2) *reinterpret_cast<uint32_t *>(dst) = v[0];
            else *reinterpret_cast<bf16_t *>(dst) = (bf16_t)v[0];
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// The B operand of tile (group gi of the super-group, slot tile st) from the lane's F_in bytes wc.
template <int G, int NST, int GI, int ST>
__device__ __forceinline__ uint4 bs_operand(const uint32_t *wc, bool act) {
    constexpr int J = GI % (8 / G);
    uint32_t o[4] = {0u, 0u, 0u, 0u};
    if constexpr (G >= 2) {
        constexpr int DW = G / 2;                         // dwords per tile
        constexpr int D0 = (J * NST + ST) * DW;           // first source dword
        constexpr int P0 = ((G * GI) % 8) / 2;            // first destination dword
#pragma unroll
        for (int t = 0; t < DW; ++t) o[P0 + t] = act ? wc[D0 + t] : 0u;
    } else {
        constexpr int E = J * NST + ST;                   // source bf16
        const uint32_t x = (E & 1) ? (wc[E >> 1] >> 16) : (wc[E >> 1] & 0xffffu);
        o[(GI % 8) / 2] = act ? ((GI & 1) ? x << 16 : x) : 0u;
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

template <int G, int F_IN, int CH>
__global__ __launch_bounds__(kBsThreads) void k_bwd_x_sg(const int32_t *__restrict__ idxl, const bf16_t *__restrict__ WS,
                                                         const bf16_t *__restrict__ dY, float *__restrict__ part, int B,
                                                         int Bp, int F_s, int64_t L, int64_t K, int nbt, int64_t sps,
                                                         int64_t nsg) {
    constexpr int SG = 32 / G;                    // groups per super-group
    constexpr int NST = F_IN / 16;                // slot tiles per group
    constexpr int NWD = F_IN / 4;                 // dwords of W per lane and super-group
    constexpr int D = bs_idx_depth(F_IN);
    // weight blocks: a ring of NWR super-groups, loaded WD ahead
    constexpr int NWR = SG >= 16 ? 2 : 4;
    constexpr int WD = NWR - 1;
    // super-groups per unrolled period: every ring slot index is then a compile-time constant, so
    // no register is copied while its load is in flight (which would cost a wait for all loads)
    constexpr int P = (D > SG ? D / SG : 1) > NWR ? (D > SG ? D / SG : 1) : NWR;
    static_assert(P % NWR == 0 && (P * SG) % D == 0, "ring periods");
    constexpr int RS = bs_row_bytes(CH);
    constexpr int CB = 32 * RS;                   // bytes per chunk buffer
    static_assert((D > SG ? D % SG : SG % D) == 0, "the supports' ring must wrap at super-group boundaries");
    extern __shared__ __align__(16) float bsa[];  // [F_s][32] accumulator (acc_row), then [2][32][RS] staged dY
    char *ys = reinterpret_cast<char *>(bsa + (size_t)F_s * 32);
    const int w = blockIdx.x, xcd = w % kXcds, jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    const int64_t s_begin = seg * sps;
    const int64_t s_end = s_begin + sps < nsg ? s_begin + sps : nsg;
    if (s_begin >= s_end) {   // empty segment: the partial is zero (workgroup-uniform)
        for (int e = tid; e < F_s * 32; e += kBsThreads) pp[(size_t)(e >> 5) * Bp + (e & 31)] = 0.0f;
        return;
    }
    for (int e = tid; e < F_s * 32; e += kBsThreads) bsa[e] = 0.0f;
    __syncthreads();
    const int n = (int)(s_end - s_begin);         // super-groups of this segment
    const int nch = (n + CH - 1) / CH;            // staged chunks

    if (wave >= kBsConsumers) {
        // ---- producers: chunk c = super-groups c CH .. of the segment, 32 rows x CH 64 bytes ----
        // Lane i of instruction r of wave p: row 2 (p + kBsProducers r) + i / 32, 16-byte piece
        // i mod 32 (8 labels) of the chunk; labels past the layer (and rows past B) stage zeros.
        constexpr int PPR = 4 * CH;               // pieces per row
        constexpr int RPI = 64 / PPR;             // rows per instruction
        constexpr int NI = 32 / (RPI * kBsProducers);
        static_assert(NI * RPI * kBsProducers == 32, "producer rows");
        const int p = wave - kBsConsumers;
        const int rows = B - b0 < 32 ? B - b0 : 32;
        const int pr = lane / PPR, pc = lane % PPR;
        const Buf db(dY + (int64_t)b0 * L, (uint32_t)((int64_t)rows * L * 2));
        uint4 v[2][NI];
        auto load = [&](int c, uint4 (&vv)[NI]) {
            const int64_t lab = (s_begin + (int64_t)c * CH) * 32 + 8 * pc;
            const int nvalid = lab >= L ? 0 : (L - lab >= 8 ? 8 : (int)(L - lab));   // even (L even)
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                const int r = RPI * (p + kBsProducers * i) + pr;
                const uint32_t off = (nvalid > 0 && r < rows) ? (uint32_t)(((int64_t)r * L + lab) * 2) : kOob;
                if (nvalid == 8 || nvalid == 0) {
                    vv[i] = db.ld16(off);
                } else {
                    // the row's last piece when L is not a multiple of 8: dword by dword, so that
                    // nothing past the row (the next row, or past the end of dY) is read
                    vv[i] = make_uint4(db.ld4(off), db.ld4(nvalid > 2 ? off + 4 : kOob),
                                       db.ld4(nvalid > 4 ? off + 8 : kOob), db.ld4(nvalid > 6 ? off + 12 : kOob));
                }
            }
        };
        auto store = [&](int c, const uint4 (&vv)[NI]) {
            char *yb = ys + (c & 1) * CB + pc * 16;
#pragma unroll
            for (int i = 0; i < NI; ++i) *reinterpret_cast<uint4 *>(yb + (RPI * (p + kBsProducers * i) + pr) * RS) = vv[i];
        };
        load(0, v[0]);
        if (nch > 1) load(1, v[1]);
        // chunk c into buffer c % 2 (free: its previous chunk, c - 2, was consumed before barrier
        // c - 1), then barrier c hands it over; the registers then take chunk c + 2
        for (int c = 0; c < nch; c += 2) {
            store(c, v[0]);
            if (c + 2 < nch) load(c + 2, v[0]);
            __syncthreads();
            if (c + 1 < nch) {
                store(c + 1, v[1]);
                if (c + 3 < nch) load(c + 3, v[1]);
                __syncthreads();
            }
        }
    } else {
        // ---- consumers: rows 16 bh .. 16 bh + 15 of the tile ----
        const int bh = wave;
        const int64_t g_begin = s_begin * SG;
        const int64_t g_end = s_end * SG < K ? s_end * SG : K;
        // the segment's weight blocks and lane-ordered supports
        const Buf wseg(WS + s_begin * 32 * F_IN, (uint32_t)(n * 64 * F_IN));
        const Buf iseg(idxl + g_begin * F_IN, (uint32_t)((g_end - g_begin) * F_IN * 4));
        const uint32_t wlane = (uint32_t)((q * 16 + l16) * F_IN);
        auto load_w = [&](int s, uint32_t (&wv)[NWD]) __attribute__((always_inline)) {
            const int sc = s < n ? s : n - 1;
#pragma unroll
            for (int i = 0; i < NWD / 4; ++i) {
                const uint4 x = __builtin_bit_cast(
                    uint4, __builtin_amdgcn_raw_buffer_load_b128(wseg.r, (int)(wlane + 16 * i), sc * 64 * F_IN, 0));
                wv[4 * i] = x.x;
                wv[4 * i + 1] = x.y;
                wv[4 * i + 2] = x.z;
                wv[4 * i + 3] = x.w;
            }
        };
        const int ng = (int)(g_end - g_begin);   // at least 1
        // g: group index within the segment, clamped to its last (the padding groups of the last
        // super-group then repeat a real group's rows with zero weights, adding zeros)
        auto load_f = [&](int gu, int (&f)[NST]) __attribute__((always_inline)) {
            const int g = gu < ng ? gu : ng - 1;
            const uint32_t o = (uint32_t)(l16 * NST * 4);
            if constexpr (NST == 2) {
                const uint2 x = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(iseg.r, (int)o, g * F_IN * 4, 0));
                f[0] = (int)x.x;
                f[1] = (int)x.y;
            } else {
#pragma unroll
                for (int h = 0; h < NST / 4; ++h) {
                    const uint4 x = __builtin_bit_cast(
                        uint4, __builtin_amdgcn_raw_buffer_load_b128(iseg.r, (int)(o + 16 * h), g * F_IN * 4, 0));
                    f[4 * h] = (int)x.x;
                    f[4 * h + 1] = (int)x.y;
                    f[4 * h + 2] = (int)x.z;
                    f[4 * h + 3] = (int)x.w;
                }
            }
        };
        typedef __attribute__((address_space(3))) f32x4_t lds_f32x4_t;
        const uint32_t abase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float *)bsa;
        const uint32_t achunk = (uint32_t)((4 * bh + q) << 4);   // rows 16 bh + 4q .. +3
        const char *ylane = ys + (16 * bh + l16) * RS + 16 * q;

        uint32_t wr[NWR][NWD];                    // super-group s in slot s % NWR
        int fr[D][NST];                           // group g of the segment in slot g % D
#pragma unroll
        for (int i = 0; i < WD; ++i) load_w(i, wr[i]);
#pragma unroll
        for (int d = 0; d < D; ++d) load_f(d, fr[d]);
        // super-group s = s0 + UU (s0 a multiple of P)
        auto step = [&](int s, auto uc) __attribute__((always_inline)) {
            constexpr int UU = decltype(uc)::value;
            if (s > 0 && s % CH == 0) __syncthreads();   // chunk s / CH staged (workgroup-uniform)
            load_w(s + WD, wr[(UU + WD) % NWR]);          // the slot super-group s - 1 used
            __builtin_amdgcn_sched_barrier(0);
            const uint32_t *wc = wr[UU % NWR];
            const uint4 ay = *reinterpret_cast<const uint4 *>(ylane + ((s / CH) & 1) * CB + (s % CH) * 64);
            const bf16x8_t a = as_bf16x8(ay);
            // the SG groups of the super-group, in order
            static_for<SG>([&](auto gic) __attribute__((always_inline)) {
                constexpr int GI = decltype(gic)::value;
                constexpr int R = (UU * SG + GI) % D;     // ring slot of this group's supports
                const bool act = q == (G * GI) / 8;
                uint32_t ao[NST];
#pragma unroll
                for (int st = 0; st < NST; ++st) ao[st] = ((uint32_t)fr[R][st] ^ achunk) + abase;
                load_f(s * SG + GI + D, fr[R]);
                __builtin_amdgcn_sched_barrier(0);   // keep the prefetch where it is issued
                f32x4_t acc[NST];
#pragma unroll
                for (int st = 0; st < NST; ++st) acc[st] = *(lds_f32x4_t *)(uintptr_t)ao[st];
                // D = dY_s W_gi + old through the matrix core's accumulator input
                static_for<NST>([&](auto stc) __attribute__((always_inline)) {
                    constexpr int ST = decltype(stc)::value;
                    acc[ST] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        a, as_bf16x8(bs_operand<G, NST, GI, ST>(wc, act)), acc[ST], 0, 0, 0);
                });
#pragma unroll
                for (int st = 0; st < NST; ++st) *(lds_f32x4_t *)(uintptr_t)ao[st] = acc[st];
            });
        };
        __syncthreads();                          // chunk 0 staged
        // whole periods (no exit inside one, so the loads' waits keep their depth across the loop's
        // back edge), then the rest
        int s0 = 0;
        for (; s0 + P <= n; s0 += P)
            static_for<P>([&](auto uc) __attribute__((always_inline)) { step(s0 + decltype(uc)::value, uc); });
        static_for<P>([&](auto uc) __attribute__((always_inline)) {
            if (s0 + decltype(uc)::value < n) step(s0 + decltype(uc)::value, uc);
        });
    }
    __syncthreads();
    for (int e = tid; e < F_s * 32; e += kBsThreads) {
        const int f = e >> 5, b = e & 31;
        pp[(size_t)f * Bp + b] = bsa[acc_index(f, b)];
    }
}

struct BsGeom {
    int nbt, ch;
    int64_t nsg, nseg, sps;
    size_t lds;
};

static BsGeom bs_geom(const haste::TailArgs &a) {
    BsGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    g.nsg = haste::cdiv(a.L, 32);
    constexpr int64_t budget = 160 * 1024;
    // 8 super-groups per chunk where they fit beside the accumulator, else 2
    g.ch = (int64_t)a.F_s * 128 + bs_stage_bytes(8) <= budget ? 8 : 2;
    g.lds = (size_t)a.F_s * 128 + (size_t)bs_stage_bytes(g.ch);
    int64_t spx = kCusPerXcd / g.nbt;   // one workgroup per CU: the accumulator takes most of the LDS
    if (spx < 1) spx = 1;
    const int64_t max_spx = haste::cdiv(g.nsg, kXcds);
    if (spx > max_spx) spx = max_spx;
    g.nseg = spx * kXcds;
    g.sps = haste::cdiv(g.nsg, g.nseg);
    return g;
}

template <int G, int F_IN, int CH>
static hipError_t launch_bwd_x_sg(const haste::TailArgs &a, const BsGeom &g, const int32_t *idxl, const bf16_t *WS,
                                  const void *dY, float *part, hipStream_t s) {
    auto kern = k_bwd_x_sg<G, F_IN, CH>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)g.lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(kBsThreads), g.lds, s, idxl, WS,
                       (const bf16_t *)dY, part, (int)a.B, g.nbt * 32, (int)a.F_s, a.L, a.L / a.G, g.nbt, g.sps, g.nsg);
    return hipGetLastError();
}

template <int G, int F_IN>
static hipError_t bwd_x_sg_f(const haste::TailArgs &a, const BsGeom &g, const int32_t *idxl, const bf16_t *WS,
                             const void *dY, float *part, hipStream_t s) {
    return g.ch == 8 ? launch_bwd_x_sg<G, F_IN, 8>(a, g, idxl, WS, dY, part, s)
                     : launch_bwd_x_sg<G, F_IN, 2>(a, g, idxl, WS, dY, part, s);
}

template <int G>
static hipError_t bwd_x_sg_g(const haste::TailArgs &a, const BsGeom &g, const int32_t *idxl, const bf16_t *WS,
                             const void *dY, float *part, hipStream_t s) {
    switch (a.F_in) {
        case 32: return bwd_x_sg_f<G, 32>(a, g, idxl, WS, dY, part, s);
        case 64: return bwd_x_sg_f<G, 64>(a, g, idxl, WS, dY, part, s);
        case 128: return bwd_x_sg_f<G, 128>(a, g, idxl, WS, dY, part, s);
    }
    return hipErrorInvalidValue;
}

// workspace: the per-segment partials, the super-group weight blocks, the lane-ordered supports
static size_t bs_part_bytes(const haste::TailArgs &a, const BsGeom &g) {
    return (size_t)haste::round_up(g.nseg * a.F_s * (g.nbt * 32) * 4, 256);
}
static size_t bs_ws_bytes(const haste::TailArgs &a, const BsGeom &g) {
    return (size_t)haste::round_up(g.nsg * 32 * a.F_in * 2, 256);
}

}  // namespace

namespace haste {

// bf16, G in {1, 2, 4, 8}, F_in in {32, 64} (and 128 for G >= 2: the pass's staged supports and
// weights then still fit the LDS beside the slab), F_s a multiple of 8 up to kMaxFs, and the
// logits' row offsets within the 31-bit range of a row pointer.
bool fwd_sg_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2 || a.G == 4 || a.G == 8)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || (a.F_in == 128 && a.G >= 2))) return false;
    return a.F_s % 8 == 0 && a.F_s <= kMaxFs && a.L < ((int64_t)1 << 40);
}

// backward-weight: bf16, G in {2, 4, 8}, F_in in {32, 64} (and 128 for G >= 4), F_s a multiple of
// 8 up to kMaxFs; the X^T copy of the workspace (bwd_w_mfma_ws) is shared with the other kernels.
bool bwd_w_sg_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2 || a.G == 4 || a.G == 8)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || (a.F_in == 128 && (a.G == 1 || a.G >= 4)))) return false;
    // a slab's dY rows are addressed from its first row with 31-bit byte offsets, and read with
    // buffer loads that need dword-aligned rows (L even)
    return a.F_s % 8 == 0 && a.F_s <= kMaxFs && (a.L * 32 + 1024) * 2 < ((int64_t)1 << 31) && a.L % 2 == 0;
}

hipError_t bwd_w_sg(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW, float *dbias,
                    int beta, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 32);
    hipError_t e = transpose_x(a, X, ws, s);
    if (e != hipSuccess) return e;
    switch (a.G) {
        case 1: return bwd_w_sg_g<1>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
        case 2: return bwd_w_sg_g<2>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
        case 4: return bwd_w_sg_g<4>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
        case 8: return bwd_w_sg_g<8>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
    }
    return hipErrorInvalidValue;
}

// backward-feature: bf16, G in {1, 2, 4, 8}, F_in in {32, 64, 128}, even F_s up to kMaxFs; dY rows
// dword-aligned (L even) and 32 rows of them within the 31-bit range of a buffer offset.
bool bwd_x_sg_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2 || a.G == 4 || a.G == 8)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || a.F_in == 128)) return false;
    if (a.F_s % 2 != 0 || a.F_s > kMaxFs || a.L % 2 != 0 || a.L * 32 * 2 >= ((int64_t)1 << 31)) return false;
    const BsGeom g = bs_geom(a);
    return g.lds <= 160 * 1024 && g.sps * 64 * a.F_in < ((int64_t)1 << 31);
}

size_t bwd_x_sg_ws(const TailArgs &a) {
    const BsGeom g = bs_geom(a);
    return bs_part_bytes(a, g) + bs_ws_bytes(a, g) + (size_t)round_up((a.L / a.G) * a.F_in * 4, 256);
}

hipError_t bwd_x_sg(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta, void *ws,
                    hipStream_t s) {
    const BsGeom g = bs_geom(a);
    float *part = reinterpret_cast<float *>(ws);
    bf16_t *WS = reinterpret_cast<bf16_t *>(reinterpret_cast<char *>(ws) + bs_part_bytes(a, g));
    int32_t *idxl = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(WS) + bs_ws_bytes(a, g));
    const int64_t K = a.L / a.G, Kp = g.nsg * (32 / a.G);
    const int64_t tgrid = cdiv(Kp, kBtWaves) < 8192 ? cdiv(Kp, kBtWaves) : 8192;
    hipLaunchKernelGGL(k_transpose_w_sg, dim3((unsigned)tgrid), dim3(kBtWaves * 64), 0, s, (const bf16_t *)W, idx, WS,
                       idxl, K, Kp, (int)a.G, (int)a.F_in);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    switch (a.G) {
        case 1: e = bwd_x_sg_g<1>(a, g, idxl, WS, dY, part, s); break;
        case 2: e = bwd_x_sg_g<2>(a, g, idxl, WS, dY, part, s); break;
        case 4: e = bwd_x_sg_g<4>(a, g, idxl, WS, dY, part, s); break;
        case 8: e = bwd_x_sg_g<8>(a, g, idxl, WS, dY, part, s); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 32, a.B, a.F_s, dX, beta, s);
}

hipError_t fwd_sg(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias, void *Y,
                  hipStream_t s, const int32_t *spos, int P) {
    switch (a.G) {
        case 1: return fwd_sg_g<1>(a, X, idx, W, bias, Y, s, spos, P);
        case 2: return fwd_sg_g<2>(a, X, idx, W, bias, Y, s, spos, P);
        case 4: return fwd_sg_g<4>(a, X, idx, W, bias, Y, s, spos, P);
        case 8: return fwd_sg_g<8>(a, X, idx, W, bias, Y, s, spos, P);
    }
    return hipErrorInvalidValue;
}

}  // namespace haste
