// Group-shared fixed fan-in tail on bf16 MFMA (gfx950, v_mfma_f32_32x32x16_bf16).
//
// The three products of the paper's Section 3.2, each run per label group k (labels kG..kG+G-1,
// support idx[k, 0..F_in-1]):
//   forward          Z_k  = H_k W_k^T            H_k = X[:, idx[k, :]]   (M = batch, N = labels, K = slots)
//   backward-weight  dW_k = dZ_k^T H_k                                   (M = labels, N = slots, K = batch)
//   backward-feature dH_k = dZ_k W_k, scattered to X's columns idx[k,:] (M = slots,  N = batch,  K = labels)
// Every contraction is a small dense GEMM once the group's support columns are gathered, which is
// what makes the group-shared format MFMA-friendly (one gather serves all G labels).
#include <type_traits>

#include "common.hpp"

namespace {




// --------------------------------------------------------------------------------------------
// Forward.
// A workgroup keeps BT rows of X resident in LDS (the "slab") and sweeps a contiguous stream of
// groups.  Each wave owns two consecutive (group, 32-label tile) units at a time: it takes the
// labels' weights as the A operand in their natural row layout and gathers the group's support
// columns from the slab into B-operand registers (gathered once per unit and batch tile, shared by
// the tile's 32 labels through the MFMA M dimension).  The next pair's indices and weights are
// loaded while the current one computes.  The nbt workgroups of one stream (one per batch tile)
// carry the same blockIdx % 8, so they run on one XCD and W is fetched from HBM about once per
// stream.  Orientation: Z^T = W_k H_k^T (M = labels, N = batch rows, K = support slots); a result
// lane holds 4 consecutive labels of one row.
// Gather: the slab is stored transposed, one row of BT batch values per feature, so that a
// feature's values for 4 consecutive rows are one 8-byte word.  ds_read_b64_tr_b16 then hands
// each lane of a 16-lane group 4 support slots of its own row: source lane 4j + a names slot j of
// a 4-slot quad and rows 4a .. 4a+3, and result lane i receives element i % 4 of the words of
// lanes 4j + i / 4, i.e. row i of slots j = 0..3.  Two such reads fill one 8-slot B operand:
// 16 elements per lane per LDS instruction instead of one.
// Stores: the 32-row x 64-label output of a pair goes through a small per-wave LDS buffer and
// leaves as whole 128-byte row pieces, 8 rows per store instruction.  (Storing straight from the
// result layout takes 4x the instructions, or touches 32 rows of the [B, L] logits, megabytes
// apart, per instruction; both limit the kernel well below HBM bandwidth.)
// --------------------------------------------------------------------------------------------
template <int F_IN, bool HAS_BIAS>
struct FwdUnit {
    int fi[F_IN / 8];                 // support index of each of this lane's gather reads (2 per K-step)
    uint4 w[F_IN / 16];               // weights of this lane's label, 8 slots per K-step
    float4 bias[HAS_BIAS ? 4 : 1];    // bias of this lane's accumulator labels (8i + 4hh .. +3)
};

constexpr int kFwdStageRow = 144;     // bytes per staged row: 64 labels + 8 pad
constexpr int kFwdXtPad = 4;          // bf16 padding of a transposed slab row (BT + 4 values)

template <int BT, int F_IN, bool HAS_BIAS, bool WIDE>
__global__ __launch_bounds__(512) void k_fwd(const bf16_t *__restrict__ X, const int32_t *__restrict__ idx,
                                             const bf16_t *__restrict__ W, const float *__restrict__ bias,
                                             bf16_t *__restrict__ Y, int B, int F_s, int64_t L, int G,
                                             int64_t K, int nbt, int64_t gps) {
    extern __shared__ __align__(16) bf16_t xs[];
    constexpr int XR = BT + kFwdXtPad;   // values per transposed slab row (one feature)
    const int w = blockIdx.x;
    const int xcd = w % kXcds;
    const int jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t stream = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * BT;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;

    // transposed slab: xs[f * XR + r] = X[b0 + r, f], zero rows past B.  A thread takes two rows
    // and two features (F_s and BT are even): two 4-byte reads, two 4-byte writes.
    {
        const int half = F_s >> 1;
        const uint32_t *X32 = reinterpret_cast<const uint32_t *>(X);
        uint32_t *xs32 = reinterpret_cast<uint32_t *>(xs);
        for (int e = tid; e < (BT / 2) * half; e += nthr) {
            const int rp = e / half, c = e - rp * half;
            const int b = b0 + 2 * rp;
            const uint32_t v0 = b < B ? X32[(int64_t)b * half + c] : 0u;
            const uint32_t v1 = b + 1 < B ? X32[(int64_t)(b + 1) * half + c] : 0u;
            xs32[((2 * c) * XR >> 1) + rp] = (v0 & 0xffffu) | (v1 << 16);
            xs32[((2 * c + 1) * XR >> 1) + rp] = (v0 >> 16) | (v1 & 0xffff0000u);
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
    using Unit = FwdUnit<F_IN, HAS_BIAS>;
    const size_t xt_bytes = ((size_t)F_s * XR * 2 + 15) & ~(size_t)15;
    char *stg = reinterpret_cast<char *>(xs) + xt_bytes + wave * (32 * kFwdStageRow);

    // weight staging: WS slots per round, NR rounds; a load covers LPI labels x WS slots (CPL
    // 16-byte chunks per label, whole 128-byte lines), IPR loads per round; LDS rows of RW bytes
    constexpr int WS = F_IN < 64 ? F_IN : 64;
    constexpr int NR = F_IN / WS;
    constexpr int CPL = WS / 8;
    constexpr int LPI = 64 / CPL;
    constexpr int IPR = 32 / LPI;
    constexpr int RW = WS * 2 + 16;
    static_assert(32 * RW <= 32 * kFwdStageRow, "weight staging exceeds the wave's LDS buffer");
    const int wl = lane / CPL, wc = lane % CPL;

    // gather roles: 16-lane group lane / 16 covers rows 16 ((lane / 16) % 2) .. +15 of an n-tile
    // and K-half hh; as a source lane, i = lane % 16 = 4 jq + aq names slot jq of each 4-slot
    // quad and rows 4 aq .. 4 aq + 3
    const int jq = (lane & 15) >> 2;
    const char *gbase = reinterpret_cast<const char *>(xs) + (16 * ((lane >> 4) & 1) + 4 * (lane & 3)) * 2;

    // bias of this lane's accumulator labels in a unit: tile*32 + 8i + 4hh .. +3 of group k
    auto load_bias = [&](uint32_t k, int tile, float4 (&b)[4]) {
        const Buf bb(bias + (int64_t)k * G, (uint32_t)(G * 4));
#pragma unroll
        for (int i = 0; i < 4; ++i)
            b[i] = __builtin_bit_cast(float4, bb.ld16((uint32_t)((tile * 32 + 8 * i + 4 * hh) * 4)));
    };

    auto issue = [&](int64_t u, Unit &f) {
        const uint32_t uu = (uint32_t)u;   // unit indices fit in 32 bits (L * 128 < 2^31)
        const uint32_t k = ntn == 1 ? uu : uu / (uint32_t)ntn;
        const int tile = (int)(uu - k * (uint32_t)ntn);
        // read h of K-step s gathers slot 16 s + 8 hh + 4 h + jq
        const int32_t *ip = idx + (int64_t)k * F_IN + 8 * hh + jq;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            f.fi[2 * s] = ip[16 * s];
            f.fi[2 * s + 1] = ip[16 * s + 4];
        }
        // weights of the tile's labels, whole 128-byte lines per instruction (labels past G read
        // as zero): load s = r IPR + t holds slots r WS + 8 wc .. +7 of label LPI t + wl
        const Buf wb(W + (int64_t)k * G * F_IN, (uint32_t)(G * F_IN * 2));
        const uint32_t wo = (uint32_t)(((tile * 32 + wl) * F_IN + 8 * wc) * 2);
#pragma unroll
        for (int r = 0; r < NR; ++r)
#pragma unroll
            for (int t = 0; t < IPR; ++t)
                f.w[r * IPR + t] = wb.ld16(wo + (uint32_t)((LPI * t * F_IN + r * WS) * 2));
        if constexpr (HAS_BIAS) load_bias(k, tile, f.bias);
    };

    // one unit: gather H_k for this tile from the slab and MFMA with the labels' weights; the
    // accumulators start from the labels' biases (D[m = label 8i + 4hh + j][n = row]).  The
    // weights pass through the wave's LDS buffer, WS slots at a time, to reach the A-operand
    // layout (label ln, slots 16 s + 8 hh .. +7).  after_step(j) runs after the j-th product
    // (j = s * NT + n).
    auto compute = [&](const Unit &cu, f32x16_t (&acc)[NT], auto &&after_step) {
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            if constexpr (HAS_BIAS) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    acc[n][4 * i + 0] = cu.bias[i].x;
                    acc[n][4 * i + 1] = cu.bias[i].y;
                    acc[n][4 * i + 2] = cu.bias[i].z;
                    acc[n][4 * i + 3] = cu.bias[i].w;
                }
            } else {
                acc[n] = f32x16_t{0};
            }
        }
#pragma unroll
        for (int r = 0; r < NR; ++r) {
#pragma unroll
            for (int t = 0; t < IPR; ++t)
                *reinterpret_cast<uint4 *>(stg + (LPI * t + wl) * RW + wc * 16) = cu.w[r * IPR + t];
            uint4 wa[WS / 16];
#pragma unroll
            for (int sl = 0; sl < WS / 16; ++sl)
                wa[sl] = *reinterpret_cast<const uint4 *>(stg + ln * RW + (16 * sl + 8 * hh) * 2);
#pragma unroll
            for (int sl = 0; sl < WS / 16; ++sl) {
                const int s = r * (WS / 16) + sl;
                const char *p0 = gbase + cu.fi[2 * s] * (XR * 2);
                const char *p1 = gbase + cu.fi[2 * s + 1] * (XR * 2);
#pragma unroll
                for (int n = 0; n < NT; ++n) {
                    // B[k = 8 hh + e][n = row] = X[b0 + 32 n + row][idx[k, 16 s + 8 hh + e]]
                    const uint2 lo = lds_read_tr(p0 + 64 * n);
                    const uint2 hi = lds_read_tr(p1 + 64 * n);
                    acc[n] = mfma32x32x16(as_bf16x8(wa[sl]), as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), acc[n]);
                    after_step(s * NT + n);
                }
            }
        }
    };

    // D[m = label 8i + 4hh + j][n = row ln] of one n-tile -> stage[row ln][col0 + 8i + 4hh .. +3]
    auto stage = [&](const f32x16_t &acc, int col0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint2 v = make_uint2(pack_bf16(acc[4 * i + 0], acc[4 * i + 1]),
                                       pack_bf16(acc[4 * i + 2], acc[4 * i + 3]));
            *reinterpret_cast<uint2 *>(stg + ln * kFwdStageRow + (col0 + 8 * i + 4 * hh) * 2) = v;
        }
    };

    // Labels of a unit: [k G + 32 tile, + nlab).  Units u and u + 1 cover contiguous labels.
    auto unit_labels = [&](int64_t u, int64_t &lab0, int &nlab) {
        const uint32_t uu = (uint32_t)u;
        const uint32_t k = ntn == 1 ? uu : uu / (uint32_t)ntn;
        const int tile = (int)(uu - k * (uint32_t)ntn);
        lab0 = (int64_t)k * G + tile * 32;
        nlab = G - tile * 32 < 32 ? G - tile * 32 : 32;
    };

    // Stores of a unit pair's staged 32-row tiles (width labels from lab0).  WIDE: 16 bytes per
    // lane, 8 lanes per 128-byte row and 8 rows per instruction (needs G and L multiples of 8);
    // else 8 bytes per lane, 16 lanes per row and 4 rows per instruction.  Rows past B fall
    // outside the buffer; labels past the pair are sent out of range.
    constexpr int LPR = WIDE ? 8 : 16;          // lanes per staged row
    constexpr int RPS = 64 / LPR;               // rows per store instruction
    constexpr int SPT = 32 / RPS;               // store instructions per n-tile
    constexpr int NS = NT * SPT;                // store instructions per pair
    using SV = typename std::conditional<WIDE, uint4, uint2>::type;
    const int rows = B - b0 < BT ? B - b0 : BT;
    const int sr = lane / LPR, sc = lane % LPR;
    // row 32 n + RPS p + sr of store i = n SPT + p; offsets stay below 64 rows (L * 128 < 2^31)
    const uint32_t lane_off = (uint32_t)(((int64_t)sr * L + (int64_t)sc * (sizeof(SV) / 2)) * 2);
    const uint32_t row_step = (uint32_t)(L * 2 * RPS);
    auto unstage = [&](int n, SV (&sv)[NS]) {
#pragma unroll
        for (int p = 0; p < SPT; ++p)
            sv[n * SPT + p] = *reinterpret_cast<const SV *>(stg + (RPS * p + sr) * kFwdStageRow + sc * sizeof(SV));
    };
    Buf pyb(Y, 0);     // the pair whose tiles sv holds (none yet: every store out of range)
    bool pok = false;  // this lane's labels lie within that pair
    auto set_pair = [&](int64_t lab0, int width) {
        pyb = Buf(Y + (int64_t)b0 * L + lab0, (uint32_t)((int64_t)rows * L * 2));
        pok = sc * (int)(sizeof(SV) / 2) < width;
    };
    auto store_one = [&](int i, const SV (&sv)[NS]) {
        const uint32_t off = pok ? lane_off + (uint32_t)i * row_step : kOob;
        // the logits are written once and not read again by this kernel: streaming stores
        if constexpr (WIDE)
            pyb.st16<kStreaming>(sv[i], off);
        else
            pyb.st8<kStreaming>(sv[i], off);
    };

    // A wave takes two consecutive 32-label tiles (a pair) at a time and stores them together, so
    // each 128-byte line of a Y row is written whole.  A pair's output is held in registers and
    // its stores are spread over the next pair's products, so that loads and stores share the
    // memory pipeline evenly.  On gfx9 one in-order counter covers vector loads and stores, so a
    // wait for a pair's weights also waits for every store issued before them: the weights are
    // therefore prefetched two pairs ahead (two pairs of unit buffers, used alternately with no
    // register copies), which leaves the stores a whole pair's products to complete.  Prefetches
    // are issued unconditionally (the index is clamped to the last unit) so that every wait only
    // covers the loads it needs.  Where the registers do not hold four units (128-slot supports,
    // or a bias with 8-byte stores) the weights are prefetched one pair ahead.
    constexpr bool DEEP = F_IN <= 64 && (WIDE || !HAS_BIAS);
    Unit ua0, ub0, ua1, ub1;
    SV sv[NS];
    const int64_t st = 2 * nwaves;
    const int64_t last = u_end - 1;
    auto cl = [&](int64_t v) { return v < last ? v : last; };
    int64_t u = u_begin + 2 * wave;
    if (u > last) return;
    issue(u, ua0);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    issue(cl(u + 1), ub0);
    __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    if constexpr (DEEP) {
        issue(cl(u + st), ua1);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
        issue(cl(u + st + 1), ub1);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
    }
    // the pair starting at unit v from buffers (ua, ub), which then take the pair `ahead` units on
    auto step = [&](int64_t v, Unit &ua, Unit &ub, int64_t ahead) {
        int64_t lab0, lab1;
        int na, nb;
        unit_labels(v, lab0, na);
        unit_labels(cl(v + 1), lab1, nb);
        const int width = na + (v + 1 <= last ? nb : 0);
        f32x16_t acc_a[NT], acc_b[NT];
        compute(ua, acc_a, [&](int i) { if (i < NS) store_one(i, sv); });
        __builtin_amdgcn_sched_barrier(0);
        // past the last unit: a repeat, never stored
        compute(ub, acc_b, [&](int i) { if (KS * NT + i < NS) store_one(KS * NT + i, sv); });
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 2 * KS * NT; i < NS; ++i) store_one(i, sv);
        // both units' registers are free once their products are done
        issue(cl(v + ahead), ua);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
        issue(cl(v + ahead + 1), ub);
        __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            stage(acc_a[n], 0);
            stage(acc_b[n], na);   // a unit of fewer than 32 labels: its unused columns are overwritten
            unstage(n, sv);
        }
        set_pair(lab0, width);
    };
    if constexpr (DEEP) {
        // whole double steps (no exit between the halves), then a last single step
        for (; u + st <= last; u += 2 * st) {
            step(u, ua0, ub0, 2 * st);
            step(u + st, ua1, ub1, 2 * st);
        }
        if (u <= last) step(u, ua0, ub0, 2 * st);
    } else {
        for (; u <= last; u += st) step(u, ua0, ub0, st);
    }
#pragma unroll
    for (int i = 0; i < NS; ++i) store_one(i, sv);
}

// X [B][F_s] -> Xb [Bp/32][F_s][32]: X^T in 32-row batch blocks (rows past B zero).  Within a
// block, the 64-byte rows of nearby features are adjacent, so a gather over a tile's sorted
// support stays within a few pages.
__global__ __launch_bounds__(256) void k_transpose_x(const bf16_t *__restrict__ X, bf16_t *__restrict__ Xb,
                                                     int B, int F_s) {
    __shared__ bf16_t tile[32][33];
    const int f0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
    for (int r = ty; r < 32; r += 8) {
        const int b = b0 + r, f = f0 + tx;
        tile[r][tx] = (b < B && f < F_s) ? X[(int64_t)b * F_s + f] : (bf16_t)0;
    }
    __syncthreads();
    bf16_t *blk = Xb + (int64_t)blockIdx.y * F_s * 32;
    for (int r = ty; r < 32; r += 8) {
        const int f = f0 + r;
        if (f < F_s) blk[(int64_t)f * 32 + tx] = tile[tx][r];
    }
}

__device__ __forceinline__ f32x4_t mfma16x16x32(const bf16x8_t &a, const bf16x8_t &b, const f32x4_t &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// --------------------------------------------------------------------------------------------
// Backward-weight, slab-staged.  A workgroup of 8 waves takes 16 consecutive units (a contiguous
// span of at most 512 labels, two units per wave) and sweeps the batch in 32-row slabs.  Per slab
// it stages in LDS, cooperatively and with whole-line loads, the X^T block of all F_s features
// (contiguous in Xb, 64 bytes per feature) and the span's dY rows (up to 1 KB per row); each wave
// then gathers its units' support rows from the staged block, one 16-byte LDS read per slot tile,
// instead of from memory.  The next slab is loaded into registers while the current one is
// multiplied.
// Per unit and slab (v_mfma_f32_16x16x32_bf16, M = 16 slots, N = 16 labels, K = the 32 rows):
//   A operand (slots x rows) = X^T rows of the slot's feature, rows 8q .. 8q+7 of slot l16;
//   B operand (rows x labels) = dY, two ds_read_b64_tr_b16 (4 rows each) per 16-label tile;
//   result lane (label l16, q) holds slots 4q .. 4q+3 of one label: a 16-byte store into dW.
// dbias comes from the same B operands against an all-ones A operand.
// --------------------------------------------------------------------------------------------
constexpr int kBw2Waves = 8;
constexpr int kBw2Units = 2 * kBw2Waves;        // units per workgroup (two per wave)
constexpr int kBw2XRow = 80;                    // bytes per staged X^T feature row: 32 rows + 8 pad
constexpr int kBw2YRow = 1056;                  // bytes per staged dY row: 512 labels + 16 pad
constexpr int kBw2MaxXLoads = kMaxFs * 4 / (kBw2Waves * 64);   // 16-byte X^T loads per thread and slab

// the staged slabs, or at the end the per-wave dW staging ([32 labels][F_in + 4] fp32 per wave)
static size_t bw2_lds(int F_s, int F_in) {
    const size_t slabs = (size_t)haste::round_up((int64_t)F_s * kBw2XRow, 16) + 32 * kBw2YRow;
    const size_t out = (size_t)kBw2Waves * 32 * (F_in + 4) * 4;
    return slabs > out ? slabs : out;
}

template <int F_IN>
__global__ __launch_bounds__(512) void k_bwd_w2(const bf16_t *__restrict__ Xb, const int32_t *__restrict__ idx,
                                                const bf16_t *__restrict__ dY, float *__restrict__ dW,
                                                float *__restrict__ dbias, int beta, int B, int Bp, int F_s,
                                                int64_t L, int G, int64_t K) {
    extern __shared__ __align__(16) char bw2s[];
    constexpr int NST = F_IN / 16;              // 16-slot M-tiles
    char *xs = bw2s;
    char *ys = bw2s + ((F_s * kBw2XRow + 15) & ~15);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const int ntn = (G + 31) >> 5;
    const int64_t nunits = K * ntn;
    const int64_t u0 = (int64_t)blockIdx.x * kBw2Units;
    auto lab_of = [&](int64_t v) {
        const int64_t k = v / ntn;
        return k * G + 32 * (int)(v - k * ntn);
    };
    auto nlab_of = [&](int64_t v) {
        const int t = (int)(v % ntn);
        return G - 32 * t < 32 ? G - 32 * t : 32;
    };
    const int64_t ul = u0 + kBw2Units - 1 < nunits ? u0 + kBw2Units - 1 : nunits - 1;
    const int64_t lab0 = lab_of(u0);
    const int span = (int)(lab_of(ul) + nlab_of(ul) - lab0);   // at most 512 labels

    // this wave's units (a unit past the end repeats the last one and is never stored)
    int64_t vu[2];
    int off[2], nl[2];
    int f[2][NST];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t v = u0 + 2 * wave + j;
        vu[j] = v < nunits ? v : nunits - 1;
        off[j] = (int)(lab_of(vu[j]) - lab0);
        nl[j] = v < nunits ? nlab_of(vu[j]) : 0;
        const int64_t k = vu[j] / ntn;
#pragma unroll
        for (int st = 0; st < NST; ++st) f[j][st] = idx[k * F_IN + 16 * st + l16];
    }

    // cooperative slab loads: X^T block (4 F_s chunks of 16 bytes) and dY (32 rows x 64 chunks)
    const int nxc = 4 * F_s;
    uint4 xr[kBw2MaxXLoads], yr[4];
    auto load = [&](int blk) {
        const Buf xb(Xb + (int64_t)blk * F_s * 32, (uint32_t)(nxc * 16));
#pragma unroll
        for (int i = 0; i < kBw2MaxXLoads; ++i) xr[i] = xb.ld16((uint32_t)(tid + 512 * i) * 16);   // past the block: zero
        // rows past B and labels past the span read as zero
        const int b0 = blk * 32;
        const int rows = B - b0 < 32 ? B - b0 : 32;
        const Buf db(dY + (int64_t)b0 * L + lab0, (uint32_t)(rows > 0 ? ((int64_t)(rows - 1) * L + span) * 2 : 0));
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 512 * i, row = c >> 6, part = c & 63;
            const bool ok = row < rows && 8 * part < span;
            yr[i] = db.ld16(ok ? (uint32_t)(((int64_t)row * L + 8 * part) * 2) : kOob);
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int i = 0; i < kBw2MaxXLoads; ++i) {
            const int c = tid + 512 * i;
            if (c < nxc) *reinterpret_cast<uint4 *>(xs + (c >> 2) * kBw2XRow + (c & 3) * 16) = xr[i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 512 * i;
            *reinterpret_cast<uint4 *>(ys + (c >> 6) * kBw2YRow + (c & 63) * 16) = yr[i];
        }
    };

    f32x4_t acc[2][NST][2], db[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int lt = 0; lt < 2; ++lt) {
            db[j][lt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int st = 0; st < NST; ++st) acc[j][st][lt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
    }
    const bf16x8_t ones = as_bf16x8(make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    // B-operand source lanes: 16-lane group q reads rows 8q + 4h + (l16 >> 2), labels 4 (l16 & 3) ..
    const char *ysrc = ys + (8 * q + (l16 >> 2)) * kBw2YRow + (l16 & 3) * 8;

    const int nblk = Bp / 32;
    load(0);
    for (int blk = 0; blk < nblk; ++blk) {
        __syncthreads();   // the previous slab is no longer read
        store();
        __syncthreads();
        if (blk + 1 < nblk) load(blk + 1);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            uint4 yv[2];
#pragma unroll
            for (int lt = 0; lt < 2; ++lt) {
                const char *p = ysrc + (off[j] + 16 * lt) * 2;
                const uint2 lo = lds_read_tr(p);
                const uint2 hi = lds_read_tr(p + 4 * kBw2YRow);
                yv[lt] = make_uint4(lo.x, lo.y, hi.x, hi.y);
            }
#pragma unroll
            for (int st = 0; st < NST; ++st) {
                const uint4 xv = *reinterpret_cast<const uint4 *>(xs + f[j][st] * kBw2XRow + q * 16);
#pragma unroll
                for (int lt = 0; lt < 2; ++lt)
                    acc[j][st][lt] = mfma16x16x32(as_bf16x8(xv), as_bf16x8(yv[lt]), acc[j][st][lt]);
            }
            if (dbias) {
#pragma unroll
                for (int lt = 0; lt < 2; ++lt) db[j][lt] = mfma16x16x32(ones, as_bf16x8(yv[lt]), db[j][lt]);
            }
        }
    }

    // dW: a unit's block [32 labels][F_IN] fp32 is contiguous in dW, so each wave stages its
    // unit's products (lane (label 16 lt + l16, q) holds slots 16 st + 4q .. +3) in its own LDS
    // region and writes the block back as whole 1 KB runs (streaming stores; labels past the unit
    // are not written).  dbias from the q = 0 lanes.
    __syncthreads();   // every wave is done with the staged slabs
    constexpr int OS = F_IN + 4;                       // staged row stride (floats)
    float *ostg = reinterpret_cast<float *>(bw2s) + wave * 32 * OS;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t lb = lab_of(vu[j]);
#pragma unroll
        for (int lt = 0; lt < 2; ++lt)
#pragma unroll
            for (int st = 0; st < NST; ++st)
                *reinterpret_cast<float4 *>(ostg + (16 * lt + l16) * OS + 16 * st + 4 * q) =
                    make_float4(acc[j][st][lt][0], acc[j][st][lt][1], acc[j][st][lt][2], acc[j][st][lt][3]);
        const Buf ob(dW + lb * F_IN, (uint32_t)(nl[j] * F_IN * 4));   // this unit's labels only
#pragma unroll
        for (int i = 0; i < F_IN / 8; ++i) {
            const int e = 64 * i + lane;                   // float4 e of the block
            const int r = e / (F_IN / 4), c = (e % (F_IN / 4)) * 4;
            float4 v = *reinterpret_cast<const float4 *>(ostg + r * OS + c);
            if (beta) {
                const float4 o = __builtin_bit_cast(float4, ob.ld16((uint32_t)(e * 16)));
                v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
            }
            ob.st16<kStreaming>(__builtin_bit_cast(uint4, v), (uint32_t)(e * 16));
        }
        if (dbias && q == 0) {
#pragma unroll
            for (int lt = 0; lt < 2; ++lt) {
                const int t = 16 * lt + l16;
                if (t < nl[j]) dbias[lb + t] = (beta ? dbias[lb + t] : 0.0f) + db[j][lt][0];
            }
        }
    }
}

// --------------------------------------------------------------------------------------------
// Forward with the BCE-gradient epilogue, and the backward-weight product of that gradient in the
// same pass (Section 3.2 forward and backward-weight; Section 3.3 objective).  The logits are not
// stored: the output is dY = sigmoid(z) - T, and dW = dY^T H_k is formed from the dY registers.
// The workgroup layout follows the slab-staged backward-weight kernel: NW waves take one unit each
// (a contiguous span of at most 512 labels) and sweep the batch in 32-row slabs, with the X^T
// block of each slab staged in LDS.  A wave keeps its unit's weights in registers for the sweep,
// so W is read from memory once.  Per unit and slab, with v_mfma_f32_16x16x32_bf16:
//   forward, M = 16 rows, N = 16 labels, K = 32 slots:
//     A = the gathered support columns, two ds_read_b64_tr_b16 per 32-slot step.  Source lane
//         4j + a of 16-lane group q names slot 8q + 4h + j (read h) and rows 8a + 4m .. +3 of
//         M-tile m, so result lane i holds row 8(i / 4) + 4m + i % 4 of those slots;
//     B = W: 16 contiguous bytes of one label's row (slots 32s + 8q .. +7 of label l16) per lane.
//   Result lane (label l16, q) then holds rows 8q .. 8q+3 (M-tile 0) and 8q+4 .. 8q+7 (M-tile 1)
//   of its label.  After the epilogue these 8 values of dY are exactly the B operand of the
//   backward-weight product (K = rows 8q .. 8q+7, N = label), which thus never leaves the
//   registers; that product and its A operand are the backward-weight kernel's, in the same
//   order, so dW equals what haste_bwd_w computes from the stored dY, bit for bit.
// dY: adjacent lanes swap halves (DPP) so that each writes two labels of four rows as 4-byte
// words into the slab's [32 rows][512 labels] LDS block.  The block's 32-byte column blocks are
// XOR-permuted by row / 8 (the lanes of one write instruction then hit distinct banks), and the
// whole block leaves as 1 KB row runs, cooperatively, in the next slab's barrier window: one row
// per store instruction, the pattern the DRAM pages serve fastest.  (Double-buffering the block so
// that its stores run during the next slab's products measured the same time.)
// Rows past B (a last, partial slab) meet zero X^T rows in the backward-weight product and are
// never stored, so their dY is zeroed only where dbias sums it.
// Targets: the slab's positives that fall in the workgroup's span are set as bits of an LDS
// bitmap, one 32-bit word of rows per label.  Two bitmaps alternate by slab parity: in one
// barrier interval each thread clears its word of the previous slab's bitmap and sets the
// current slab's bits, and the bitmap is read only after the next barrier.  Rows of at most
// kFbMaxPos positives: every workgroup prefetches all of the slab's positives (two per thread)
// and keeps those in its span.  Longer rows: a pre-pass buckets the positives by (workgroup,
// slab) cell (counting sort), and a workgroup prefetches only its own cell's entries, one per
// thread (a cell of more than one entry per thread finishes with direct loads).
// --------------------------------------------------------------------------------------------
constexpr int kFbMaxSpan = 512;                 // labels per workgroup at most
constexpr int kFbMaxPos = 64;                   // positives per row the slab prefetch holds
constexpr int kFbYRow = 1056;                   // bytes per staged dY row: 512 labels + 32 pad

// waves per workgroup: one 32-label unit each; 128-slot supports need twice the registers
__host__ __device__ constexpr int fb_waves(int F_in) { return F_in == 128 ? 8 : 16; }

// a wave's LDS region for the transposed weights of its group (32 labels) and the slot positions
__host__ __device__ constexpr int fb_wt_region(int f_in) { return 32 * f_in * 2 + 128; }

// The X^T block (two with dbx: the next slab's is staged while the current one is in use), the
// target bitmaps (two, or three with dbx) and the staged dY block; or at the end the dW staging of
// every wave
static size_t fb_lds(int F_s, int F_in, bool dbx) {
    const size_t main = (size_t)(dbx ? 2 : 1) * haste::round_up((int64_t)F_s * kBw2XRow, 16) +
                        (size_t)(dbx ? 3 : 2) * kFbMaxSpan * 4 + (size_t)32 * kFbYRow;
    const size_t out = (size_t)fb_waves(F_in) * 32 * (F_in + 4) * 4;
    return main > out ? main : out;
}

__device__ __forceinline__ uint32_t dpp_swap_pairs(uint32_t v) {   // lane l receives lane l ^ 1's value
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);   // quad_perm [1, 0, 3, 2]
}

// byte offset of dword d of staged dY row r (32-byte column blocks permuted by r / 8)
__device__ __forceinline__ int fb_ystg_off(int r, int d) { return r * kFbYRow + 4 * (d ^ (8 * (r >> 3))); }

// widest input the kernel takes; its X^T prefetch registers cover the first kFbPrefetchFs features
// of a slab's block, and wider inputs load the rest while staging
constexpr int kFbMaxFs = 1024;
constexpr int kFbPrefetchFs = 768;

// what the kernel does with the backward-weight product: nothing, store dW, or apply the
// momentum step to W with it (dW never stored)
constexpr int kFbOutNone = 0, kFbOutDW = 1, kFbOutSGD = 2;

template <int F_IN, bool HAS_BIAS, int OUT, bool WITH_DB, bool BUCKETED, bool DBX>
__global__ __launch_bounds__(64 * fb_waves(F_IN)) void k_fwd_bce(
    const bf16_t *__restrict__ Xb, const int32_t *__restrict__ idx, const bf16_t *__restrict__ W,
    const float *__restrict__ bias, const int32_t *__restrict__ pos, int P, bf16_t *__restrict__ dY,
    float *__restrict__ dW, float *__restrict__ dbias, int beta, float lr, float momentum, float weight_decay,
    float *__restrict__ mom, bf16_t *__restrict__ W_next, int B, int Bp, int F_s, int64_t L, int G, int64_t K,
    bf16_t *__restrict__ WT, int32_t *__restrict__ idxl, const int32_t *__restrict__ cofs,
    const uint32_t *__restrict__ cent, int64_t n_ent) {
    constexpr bool WITH_DW = OUT != kFbOutNone;
    extern __shared__ __align__(16) char fbs[];
    constexpr int NW = fb_waves(F_IN);
    constexpr int NT = NW * 64;                 // threads
    constexpr int KS = F_IN / 32;               // forward K-steps (32 slots)
    constexpr int NST = F_IN / 16;              // backward-weight M-tiles (16 slots)
    constexpr int XL = kFbPrefetchFs * 4 / NT;  // prefetched 16-byte X^T loads per thread and slab
    constexpr int XW = (kFbMaxFs - kFbPrefetchFs) * 4 / NT;   // and the rest of the widest input
    constexpr int PL = 32 * kFbMaxPos / NT;     // positives per thread and slab
    constexpr int YL = 32 * 64 / NT;            // 16-byte dY stores per thread and slab
    constexpr int NBM = DBX ? 3 : 2;            // target bitmaps in rotation
    const int xsb = (F_s * kBw2XRow + 15) & ~15;   // bytes of one X^T block
    char *xs = fbs;
    uint32_t *bm = reinterpret_cast<uint32_t *>(fbs + (DBX ? 2 : 1) * xsb);
    char *ystg = reinterpret_cast<char *>(bm + NBM * kFbMaxSpan);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const int ntn = (G + 31) >> 5;
    const int64_t nunits = K * ntn;
    const int64_t u0 = (int64_t)blockIdx.x * NW;
    auto lab_of = [&](int64_t v) {
        const int64_t k = v / ntn;
        return k * G + 32 * (int)(v - k * ntn);
    };
    auto nlab_of = [&](int64_t v) {
        const int t = (int)(v % ntn);
        return G - 32 * t < 32 ? G - 32 * t : 32;
    };
    const int64_t ul = u0 + NW - 1 < nunits ? u0 + NW - 1 : nunits - 1;
    const int64_t lab0 = lab_of(u0);
    const int span = (int)(lab_of(ul) + nlab_of(ul) - lab0);

    // this wave's unit (past the end: a repeat of the last one, never stored), its supports in
    // both operand roles, weights and biases
    const int64_t v = u0 + wave;
    const int64_t vu = v < nunits ? v : nunits - 1;
    const int64_t lb = lab_of(vu);
    const int off = (int)(lb - lab0);
    const int nl = v < nunits ? nlab_of(vu) : 0;
    int fa[KS][2];     // forward gather: slot 32 s + 8 q + 4 h + l16 / 4
    int fw[NST];       // backward-weight A operand: slot 16 st + l16
    uint4 wop[2][KS];  // W[label 16 nt + l16][32 s + 8 q .. +7]
    float bl[2];
    const int aq = l16 & 3;
    {
        const int32_t *ik = idx + (vu / ntn) * F_IN;
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
            for (int h = 0; h < 2; ++h) fa[s][h] = ik[32 * s + 8 * q + 4 * h + (l16 >> 2)];
#pragma unroll
        for (int st = 0; st < NST; ++st) fw[st] = ik[16 * st + l16];
        const int nv = nlab_of(vu);
        const Buf wb(W + lb * F_IN, (uint32_t)(nv * F_IN * 2));
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
#pragma unroll
            for (int s = 0; s < KS; ++s)
                wop[nt][s] = wb.ld16((uint32_t)(((16 * nt + l16) * F_IN + 32 * s + 8 * q) * 2));
            const int t = 16 * nt + l16;
            bl[nt] = HAS_BIAS && t < nv ? bias[lb + t] : 0.0f;
        }
    }

    // cooperative slab loads: the X^T block (4 F_s chunks of 16 bytes) and the slab's positives
    // (all of them, or this workgroup's bucket: entries (row in slab) << 16 | (label - lab0))
    const int nxc = 4 * F_s;
    const int nslab = Bp / 32;
    constexpr bool bucketed = BUCKETED;   // positives bucketed by cell (rows of more than kFbMaxPos)
    const Buf eb(cent, (uint32_t)(bucketed ? n_ent * 4 : 0));
    uint4 xr[XL];
    uint32_t pr[PL];
    int pc0 = 0, pc1 = 0;   // the current bucket's entries (bucketed)
    auto load = [&](int blk) {
        const Buf xb(Xb + (int64_t)blk * F_s * 32, (uint32_t)(nxc * 16));
#pragma unroll
        for (int i = 0; i < XL; ++i) xr[i] = xb.ld16((uint32_t)(tid + NT * i) * 16);   // past the block: zero
        if constexpr (bucketed) {
            const int64_t cell = (int64_t)blockIdx.x * nslab + blk;
            pc0 = __builtin_amdgcn_readfirstlane(cofs[cell]);   // workgroup-uniform: scalar registers
            pc1 = __builtin_amdgcn_readfirstlane(cofs[cell + 1]);
            pr[0] = eb.ld4(tid < pc1 - pc0 ? (uint32_t)(pc0 + tid) * 4 : kOob);
        } else {
            const int b0 = blk * 32;
            const int rows = B - b0 < 32 ? B - b0 : 32;
            const Buf pb(pos + (int64_t)b0 * P, (uint32_t)(rows > 0 ? rows * P * 4 : 0));
#pragma unroll
            for (int i = 0; i < PL; ++i) pr[i] = pb.ld4((uint32_t)(tid + NT * i) * 4);   // validity checked at use
        }
    };
    auto stage_slab = [&](int blk) {
        char *xd = xs + (DBX ? (blk & 1) * xsb : 0);
#pragma unroll
        for (int i = 0; i < XL; ++i) {
            const int c = tid + NT * i;
            if (c < nxc) *reinterpret_cast<uint4 *>(xd + (c >> 2) * kBw2XRow + (c & 3) * 16) = xr[i];
        }
        // clear this thread's word of the bitmap that comes next in the rotation (the slab that
        // used it is done), set this slab's targets
        uint32_t *cur = bm + (blk % NBM) * kFbMaxSpan;
        if (tid < kFbMaxSpan) bm[((blk + 1) % NBM) * kFbMaxSpan + tid] = 0u;
        if constexpr (bucketed) {
            // entries lie in this workgroup's span by construction; the masks only keep a corrupt
            // entry inside the bitmap
            if (tid < pc1 - pc0) atomicOr(cur + (pr[0] & (kFbMaxSpan - 1)), 1u << ((pr[0] >> 16) & 31));
            for (int e = pc0 + NT + tid; e < pc1; e += NT) {
                const uint32_t v = eb.ld4((uint32_t)e * 4);
                atomicOr(cur + (v & (kFbMaxSpan - 1)), 1u << ((v >> 16) & 31));
            }
        } else {
            const int rows = B - blk * 32 < 32 ? B - blk * 32 : 32;
#pragma unroll
            for (int i = 0; i < PL; ++i) {
                const int e = tid + NT * i;
                if (e < rows * P) {
                    const int64_t o = (int64_t)(int32_t)pr[i] - lab0;
                    if (o >= 0 && o < span) atomicOr(cur + o, 1u << (e / P));
                }
            }
        }
        if (nxc > XL * NT) {   // an input wider than the prefetch: the rest of the block, loaded here
            const Buf xb(Xb + (int64_t)blk * F_s * 32, (uint32_t)(nxc * 16));
#pragma unroll
            for (int i = 0; i < XW; ++i) {
                const int c = XL * NT + tid + NT * i;
                if (c < nxc) *reinterpret_cast<uint4 *>(xd + (c >> 2) * kBw2XRow + (c & 3) * 16) = xb.ld16((uint32_t)c * 16);
            }
        }
    };
    // the staged dY block of slab blk leaves as 1 KB row runs: 64 chunks of 16 bytes per row
    auto read_ystg = [&](uint4 (&yv)[YL]) {
#pragma unroll
        for (int i = 0; i < YL; ++i) {
            const int c = tid + NT * i;
            yv[i] = *reinterpret_cast<const uint4 *>(ystg + fb_ystg_off(c >> 6, 4 * (c & 63)));
        }
    };
    auto store_y = [&](int blk, const uint4 (&yv)[YL]) {
        const int b0 = blk * 32;
        const int rows = B - b0 < 32 ? B - b0 : 32;
        const Buf yo(dY + (int64_t)b0 * L + lab0, (uint32_t)(rows * L * 2));
#pragma unroll
        for (int i = 0; i < YL; ++i) {
            const int c = tid + NT * i, r = c >> 6, ch = c & 63;
            const uint32_t o = r < rows && 8 * ch < span ? (uint32_t)(((int64_t)r * L + 8 * ch) * 2) : kOob;
            yo.st16<kStreaming>(yv[i], o);
        }
    };
    auto store_slab = [&](int blk) {
        uint4 yv[YL];
        read_ystg(yv);
        store_y(blk, yv);
    };

    f32x4_t acc[NST][2], db[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        db[nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < NST; ++st) acc[st][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    const bf16x8_t ones = as_bf16x8(make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    const bool odd = (l16 & 1) != 0;

    // For the backward-feature pass of the same step (groups of 32 labels, so a wave's unit is one
    // group): the group's weights transposed and its supports in lane order, in that pass's layout
    // (W^T label-octet major [4][F_IN positions][8 labels]; positions dealt by residue mod 8, as its
    // accumulator banks need).  Staged through this wave's LDS region before the slabs use the LDS.
    if constexpr (WITH_DW) {
        if (WT) {
            constexpr int RB = 32 * F_IN * 2;                         // bytes of a group's W^T
            char *tw = fbs + wave * fb_wt_region(F_IN);
            uint8_t *sp = reinterpret_cast<uint8_t *>(tw + RB);        // position of each slot
            int f[2], ps[2];
            slot_positions(idx + vu * F_IN, F_IN, lane, f, ps);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                if (ps[i] < 0) continue;
                sp[lane + 64 * i] = (uint8_t)ps[i];
                if (v < nunits) idxl[vu * F_IN + (ps[i] & 15) * NST + (ps[i] >> 4)] = (int32_t)acc_row(f[i]);
            }
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const uint2 pp = *reinterpret_cast<const uint2 *>(sp + 32 * s + 8 * q);   // positions of 8 slots
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    const int lam = 16 * nt + l16;
                    const uint32_t u[4] = {wop[nt][s].x, wop[nt][s].y, wop[nt][s].z, wop[nt][s].w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int ps = (int)(((e < 4 ? pp.x : pp.y) >> (8 * (e & 3))) & 0xffu);
                        *reinterpret_cast<bf16_t *>(tw + (((lam >> 3) * F_IN + ps) * 8 + (lam & 7)) * 2) =
                            (bf16_t)((e & 1) ? (u[e >> 1] >> 16) : (u[e >> 1] & 0xffffu));
                    }
                }
            }
            __builtin_amdgcn_wave_barrier();
            if (v < nunits) {
                char *dst = reinterpret_cast<char *>(WT) + vu * RB;
#pragma unroll
                for (int i = 0; i < RB / 1024; ++i)
                    *reinterpret_cast<uint4 *>(dst + (i * 64 + lane) * 16) =
                        *reinterpret_cast<const uint4 *>(tw + (i * 64 + lane) * 16);
            }
            __syncthreads();   // every wave's region is read out before the bitmaps and slabs use the LDS
        }
    }
    for (int i = tid; i < NBM * kFbMaxSpan; i += NT) bm[i] = 0u;
    const int nblk = Bp / 32;
    load(0);
    if constexpr (DBX) {
        __syncthreads();   // bitmaps cleared
        stage_slab(0);
        if (nblk > 1) load(1);
    }
    for (int blk = 0; blk < nblk; ++blk) {
        if constexpr (DBX) {
            // Two X^T blocks: slab blk + 1 is staged while slab blk is in use, and the barrier pair
            // brackets only the reads of the staged dY block.
            __syncthreads();   // slab blk is staged; the previous slab is done and its dY block staged
            uint4 yv[YL];
            if (blk > 0) read_ystg(yv);
            __syncthreads();   // the dY block has been read out
            if (blk > 0) store_y(blk - 1, yv);
            if (blk + 1 < nblk) stage_slab(blk + 1);
            if (blk + 2 < nblk) load(blk + 2);
        } else {
            __syncthreads();   // the previous slab is no longer read, and its dY block is staged
            if (blk > 0) store_slab(blk - 1);
            stage_slab(blk);
            __syncthreads();
            if (blk + 1 < nblk) load(blk + 1);
        }
        const char *xsc = xs + (DBX ? (blk & 1) * xsb : 0);   // this slab's X^T block
        const uint32_t *cur = bm + (blk % NBM) * kFbMaxSpan;
        const int rows = B - blk * 32 < 32 ? B - blk * 32 : 32;
        // forward: z^T tile [32 rows][32 labels] of the unit
        f32x4_t z[2][2];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) z[m][nt] = f32x4_t{bl[nt], bl[nt], bl[nt], bl[nt]};
#pragma unroll
        for (int s = 0; s < KS; ++s) {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const uint2 lo = lds_read_tr(xsc + fa[s][0] * kBw2XRow + 16 * aq + 8 * m);
                const uint2 hi = lds_read_tr(xsc + fa[s][1] * kBw2XRow + 16 * aq + 8 * m);
                const bf16x8_t av = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) z[m][nt] = mfma16x16x32(av, as_bf16x8(wop[nt][s]), z[m][nt]);
            }
        }
        // epilogue: dY = sigmoid(z) - T for rows 8q .. 8q+7 of label 16 nt + l16, zero on rows past B.
        // Branch-free per element (so that the exp / rcp chains of the 16 values interleave); the
        // row mask is needed only in a last, partial slab and the targets only where a positive
        // falls in the tile, both wave-uniform tests.  The bitmap word of a label past the unit
        // lies inside the 512-word bitmap and is never used.
        uint4 yb[2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            const uint32_t tw = cur[off + 16 * nt + l16] >> (8 * q);
            float d[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) d[r] = sigmoid_f32(z[r >> 2][nt][r & 3]);
            if (WITH_DB && rows < 32) {
#pragma unroll
                for (int r = 0; r < 8; ++r) d[r] = 8 * q + r < rows ? d[r] : 0.0f;
            }
            if (__builtin_amdgcn_ballot_w64((tw & 0xffu) != 0u) != 0) {
#pragma unroll
                for (int r = 0; r < 8; ++r) d[r] -= (float)((tw >> r) & 1u);
            }
            yb[nt] = make_uint4(pack_bf16(d[0], d[1]), pack_bf16(d[2], d[3]), pack_bf16(d[4], d[5]),
                                pack_bf16(d[6], d[7]));
        }
        // stage: even lanes write rows 8q .. 8q+3 of labels (t, t+1), odd lanes rows 8q+4 .. +7 of (t-1, t)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            if (16 * nt >= nl) continue;   // wave-uniform: groups are whole 16-label tiles
            const uint4 y = yb[nt];
            const uint32_t r0 = dpp_swap_pairs(odd ? y.x : y.z);
            const uint32_t r1 = dpp_swap_pairs(odd ? y.y : y.w);
            const uint32_t L0 = odd ? r0 : y.x, H0 = odd ? y.z : r0;
            const uint32_t L1 = odd ? r1 : y.y, H1 = odd ? y.w : r1;
            const int row = 8 * q + (odd ? 4 : 0);
            const int dw = (off + 16 * nt + (l16 & ~1)) >> 1;
            char *p = ystg + fb_ystg_off(row, dw);   // rows row .. row+3 share the column permutation
            // low halves of (L, H), then high halves: one byte permute each
            *reinterpret_cast<uint32_t *>(p) = __builtin_amdgcn_perm(H0, L0, 0x05040100u);
            *reinterpret_cast<uint32_t *>(p + kFbYRow) = __builtin_amdgcn_perm(H0, L0, 0x07060302u);
            *reinterpret_cast<uint32_t *>(p + 2 * kFbYRow) = __builtin_amdgcn_perm(H1, L1, 0x05040100u);
            *reinterpret_cast<uint32_t *>(p + 3 * kFbYRow) = __builtin_amdgcn_perm(H1, L1, 0x07060302u);
        }
        if constexpr (WITH_DW) {
#pragma unroll
            for (int st = 0; st < NST; ++st) {
                const uint4 xv = *reinterpret_cast<const uint4 *>(xsc + fw[st] * kBw2XRow + q * 16);
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) acc[st][nt] = mfma16x16x32(as_bf16x8(xv), as_bf16x8(yb[nt]), acc[st][nt]);
            }
            if constexpr (WITH_DB) {
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) db[nt] = mfma16x16x32(ones, as_bf16x8(yb[nt]), db[nt]);
            }
        }
    }
    __syncthreads();   // the last slab's dY block is staged
    store_slab(nblk - 1);

    if constexpr (WITH_DW) {
        // dW: as in the backward-weight kernel, a wave stages its unit's [32 labels][F_IN] fp32 block
        // in its own LDS region (every wave at once: each reads back only its own block) and writes
        // it as whole contiguous runs.  With the momentum step, the same runs read the unit's W and
        // velocity and write the velocity and the next weights instead.  dbias from the q = 0 lanes.
        constexpr int OS = F_IN + 4;
        float *ostg = reinterpret_cast<float *>(fbs) + wave * 32 * OS;
        const Buf ob(OUT == kFbOutSGD ? (void *)(mom + lb * F_IN) : (void *)(dW + lb * F_IN),
                     (uint32_t)(nl * F_IN * 4));   // this unit's labels only
        const Buf wb(W + lb * F_IN, (uint32_t)(nl * F_IN * 2));
        const Buf nb(W_next + lb * F_IN, (uint32_t)(OUT == kFbOutSGD ? nl * F_IN * 2 : 0));
        __syncthreads();   // every wave is done with the staged slabs
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int st = 0; st < NST; ++st)
                *reinterpret_cast<float4 *>(ostg + (16 * nt + l16) * OS + 16 * st + 4 * q) =
                    make_float4(acc[st][nt][0], acc[st][nt][1], acc[st][nt][2], acc[st][nt][3]);
#pragma unroll
        for (int i = 0; i < F_IN / 8; ++i) {
            const int e = 64 * i + lane;
            const int r = e / (F_IN / 4), c = (e % (F_IN / 4)) * 4;
            float4 val = *reinterpret_cast<const float4 *>(ostg + r * OS + c);
            if constexpr (OUT == kFbOutSGD) {
                // slots 4e .. 4e+3 of the unit's block: W (4 bf16) and velocity (4 fp32)
                const uint2 wv = wb.ld8((uint32_t)(e * 8));
                float4 mv = __builtin_bit_cast(float4, ob.ld16((uint32_t)(e * 16)));
                float n0, n1, n2, n3;
                sgd_step(bf16_to_f32((bf16_t)(wv.x & 0xffffu)), val.x, mv.x, n0, lr, momentum, weight_decay);
                sgd_step(bf16_to_f32((bf16_t)(wv.x >> 16)), val.y, mv.y, n1, lr, momentum, weight_decay);
                sgd_step(bf16_to_f32((bf16_t)(wv.y & 0xffffu)), val.z, mv.z, n2, lr, momentum, weight_decay);
                sgd_step(bf16_to_f32((bf16_t)(wv.y >> 16)), val.w, mv.w, n3, lr, momentum, weight_decay);
                ob.st16<kStreaming>(__builtin_bit_cast(uint4, mv), (uint32_t)(e * 16));
                nb.st8<kStreaming>(make_uint2(pack_bf16(n0, n1), pack_bf16(n2, n3)), (uint32_t)(e * 8));
            } else {
                if (beta) {
                    const float4 o = __builtin_bit_cast(float4, ob.ld16((uint32_t)(e * 16)));
                    val.x += o.x; val.y += o.y; val.z += o.z; val.w += o.w;
                }
                ob.st16<kStreaming>(__builtin_bit_cast(uint4, val), (uint32_t)(e * 16));
            }
        }
        if constexpr (WITH_DB) {
            if (q == 0) {
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    const int t = 16 * nt + l16;
                    if (t < nl) dbias[lb + t] = (beta ? dbias[lb + t] : 0.0f) + db[nt][0];
                }
            }
        }
    }
}

// --------------------------------------------------------------------------------------------
// Backward-feature (split over label segments).
//
// The contraction runs over the labels of a group, which are strided in W's natural layout
// (one row of F_in slots per label), so k_transpose_w first writes every group's block
// transposed, in the order the matrix-core operand loads read it, into the workspace: one pass
// over W instead of one transpose per group and batch tile.
//
// A workgroup owns a 32-row batch tile and one contiguous segment of groups; its partial
// dX^T[F_s][32] (fp32, rows swizzled as acc_row states) lives in LDS.  Two consumer waves each own one
// 16-row half of the tile for every group and every support slot, so no two waves ever touch
// the same accumulator cell: each wave adds its products with plain read-add-write in its own
// program order (LDS operations of one wave are executed in order), with no barrier between
// groups.  Every accumulation is fp32 in a fixed order, so dX is bit-reproducible, and no LDS
// float atomics are used (they run at a small fraction of the LDS rate on gfx950).
//
// Producer waves stage dY through LDS in chunks of CH consecutive groups (at most 256 labels):
// one load instruction reads 512 contiguous bytes of a single row.  Reading dY straight into the
// MFMA operand layout instead would touch 16 rows (16 pages megabytes apart) per instruction,
// and such loads are limited by address translation rather than by HBM.  One barrier per chunk
// hands a staged chunk to the consumers and the previous buffer back to the producers, which
// keep the next chunks in flight meanwhile.
//
// Per group and 16-slot tile (v_mfma_f32_16x16x32_bf16, M = rows, N = slots, K = labels):
//   A operand (rows x labels) = staged dY, labels 32c + 8q .. +7 of row l16 (one 16-byte LDS
//     read per 32-label block, shared by all slot tiles);
//   B operand (labels x slots) = the same 8 labels of slot l16 (one 16-byte load);
//   result lane (slot, q) holds rows 4q..4q+3 of one slot: one float4 read-add-write into the
//     accumulator row idx[k, slot].
// --------------------------------------------------------------------------------------------

// W [K][G][F_in] -> WT [K][Gp / 8][F_in][8] and idx [K][F_in] -> idxl [K][F_in] (the accumulator
// row offsets acc_row(idx[k, slot]) of the slots), both in lane
// order: position p = 16 st + l16 is the slot that lane l16 of 16-slot tile st handles.  WT holds
// label octet o of position p at (o F_in + p) 8 (labels G .. Gp - 1 zero, Gp = G rounded up to
// 8), so a consumer's operand load (16 positions x one octet per 16 lanes) reads contiguous
// 256-byte runs; idxl keeps the supports of lanes l16, 16 + l16, ... side by side (one vector load
// per lane).
//
// Slot order: slot_positions (the residues of the rows mod 8 dealt round-robin, for the banks).
// One group per wave step (the four waves of a workgroup work independently, each in its own LDS
// region: the positions and the transposed block).
constexpr int kTwWaves = 4;

__host__ __device__ constexpr int tw_wave_bytes(int f_in, int gp) {
    return ((f_in * 4 + f_in * (gp + 4) * 2) + 15) / 16 * 16;
}

__global__ __launch_bounds__(kTwWaves * 64) void k_transpose_w(const bf16_t *__restrict__ W, const int32_t *__restrict__ idx,
                                                              bf16_t *__restrict__ WT, int32_t *__restrict__ idxl, int64_t K,
                                                              int G, int Gp, int F_in) {
    extern __shared__ __align__(16) char twsh[];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    char *mine = twsh + wv * tw_wave_bytes(F_in, Gp);
    int *spos = reinterpret_cast<int *>(mine);                // [F_in] lane-order position of each slot
    bf16_t *tw = reinterpret_cast<bf16_t *>(spos + F_in);     // [F_in][Gp + 4], rows by position
    const int TS = Gp + 4;
    const int nq = F_in / 4;                      // slot quads per label
    const int nst = F_in / 16;
    for (int64_t k = (int64_t)blockIdx.x * kTwWaves + wv; k < K; k += (int64_t)gridDim.x * kTwWaves) {
        // slots t = lane and t = lane + 64 (F_in = 128)
        int f[2], ps[2];
        slot_positions(idx + k * F_in, F_in, lane, f, ps);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            if (ps[i] < 0) continue;
            spos[lane + 64 * i] = ps[i];
            idxl[k * F_in + (ps[i] & 15) * nst + (ps[i] >> 4)] = (int32_t)acc_row(f[i]);
        }
        __builtin_amdgcn_wave_barrier();
        const uint2 *src = reinterpret_cast<const uint2 *>(W + k * G * F_in);
        for (int e = lane; e < G * nq; e += 64) {
            const int g = e / nq, s4 = (e - g * nq) * 4;
            const uint2 v = src[e];
            tw[spos[s4 + 0] * TS + g] = (bf16_t)(v.x & 0xFFFFu);
            tw[spos[s4 + 1] * TS + g] = (bf16_t)(v.x >> 16);
            tw[spos[s4 + 2] * TS + g] = (bf16_t)(v.y & 0xFFFFu);
            tw[spos[s4 + 3] * TS + g] = (bf16_t)(v.y >> 16);
        }
        __builtin_amdgcn_wave_barrier();
        // label-octet major: element (position p, label 8o + j) at (o F_in + p) 8 + j, so that the
        // consumers' operand loads (16 positions x 8 labels per 16 lanes) read contiguous runs
        uint4 *dst = reinterpret_cast<uint4 *>(WT + k * F_in * Gp);
        for (int e = lane; e < F_in * (Gp / 8); e += 64) {
            const int o = e / F_in, sl = e - o * F_in, g8 = 8 * o;
            const bf16_t *t = tw + sl * TS + g8;
            uint32_t w[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                w[j] = (g8 + 2 * j < G ? t[2 * j] : 0u) | ((uint32_t)(g8 + 2 * j + 1 < G ? t[2 * j + 1] : 0u) << 16);
            dst[e] = make_uint4(w[0], w[1], w[2], w[3]);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

template <int F_IN, int NLB>
struct BwdXGroup {
    uint4 w[NLB][F_IN / 16];  // W_k^T[16st + l16][32c + 8q .. +7]
    int f[F_IN / 16];         // accumulator row offsets acc_row(idx[k, 16st + l16])
};

constexpr int kBxConsumers = 2;    // consumer waves (one per 16-row half)
constexpr int kBxProducers = 4;    // producer waves
constexpr int kBxProdDepth = 4;    // staged dY chunks in flight per producer wave
constexpr int kBxChunkBytes = 20480;   // staged dY per chunk buffer, at most

// groups of weights in flight per consumer wave: registers, and at most 63 outstanding loads
__host__ __device__ constexpr int bx_depth_for(int f_in, int nlb) {
    const int per = nlb * (f_in / 16) * 4 + f_in / 16;   // registers per group
    return per <= 20 ? 8 : (per <= 40 ? 4 : 2);          // a power of two: the chunk size is a multiple
}

// Staged dY layout, per chunk buffer: [32 rows][CH groups x 32 NLB labels, then 16 spare labels]
// bf16, row stride RS = 64 NLB CH + 32 bytes.  A producer store (one row, 64 lanes x 8 bytes) is
// then one contiguous run, and a consumer's operand for one group is one 16-byte read per
// 32-label block at a lane-constant offset plus a per-group constant; with RS = 32 (mod 256)
// bytes the 8 rows one read pass serves fall in distinct banks.  Labels G .. 32 NLB - 1 of
// every group stay zero (written once, never staged), and the producers stage zeros for groups
// past the segment, so the consumers need no masking: the steps they pad their loop with (up to a
// multiple of the prefetch depth, which divides CH) read staged zeros and add nothing.
__host__ __device__ constexpr int bx_stage_row_bytes(int nlb, int ch) { return 64 * nlb * ch + 32; }

template <int F_IN, int NLB>
__global__ __launch_bounds__((kBxConsumers + kBxProducers) * 64) void k_bwd_x(
    const int32_t *__restrict__ idx, const bf16_t *__restrict__ WT, const bf16_t *__restrict__ dY, float *__restrict__ part, int B, int Bp, int F_s, int64_t L, int G, int Gp,
    int64_t K, int nbt, int64_t gps, int CH) {
    extern __shared__ __align__(16) float accs[];  // [F_s][32] (swizzled, acc_row), then the staged dY
    constexpr int NST = F_IN / 16;                 // 16-slot tiles
    constexpr int NP = kBxProducers;
    constexpr int NJ = 32 / NP;                    // rows per producer wave and chunk
    constexpr int NB = bx_depth_for(F_IN, NLB);
    constexpr int GB = 64 * NLB;                   // staged bytes per group and row
    const int RS = bx_stage_row_bytes(NLB, CH);    // staged row stride
    char *ys = reinterpret_cast<char *>(accs + F_s * 32);   // [2][32][RS]
    const int cbytes = 32 * RS;
    const int w = blockIdx.x;
    const int xcd = w % kXcds;
    const int jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x;
    const int nthr = (kBxConsumers + NP) * 64;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    float *pp = part + (size_t)seg * F_s * Bp + b0;

    const int64_t g_begin = seg * gps;
    const int64_t g_end = g_begin + gps < K ? g_begin + gps : K;
    if (g_begin >= g_end) {
        // empty segment: the partial is zero
        for (int e = tid; e < F_s * 32; e += nthr) pp[(size_t)(e >> 5) * Bp + (e & 31)] = 0.0f;
        return;
    }
    // accumulator and the whole staging area (its zero label padding is never written again)
    {
        uint32_t *z = reinterpret_cast<uint32_t *>(accs);
        const int nz = F_s * 32 + (2 * cbytes) / 4;
        for (int e = tid; e < nz; e += nthr) z[e] = 0u;
    }
    __syncthreads();
    const int n = (int)(g_end - g_begin);          // groups of this segment
    const int nch = (n + CH - 1) / CH;             // dY chunks

    if (wave >= kBxConsumers) {
        // ---- producers: dY chunk c (groups cCH .. of the segment) -> staging buffer c % 2 ----
        // Lane i loads WB bytes of one row per instruction: labels (i mod LPR) WB/2 .. of the
        // chunk, which belong to one group (WB = 16 needs groups of a multiple of 8 labels, else
        // WB = 8), and row half i / LPR of the instruction's RPI rows.  Labels past the segment read
        // as zero.  Each wave keeps PD chunks in flight in registers, so a load has PD chunk
        // periods to arrive.
        auto produce = [&](auto wb) {
            constexpr int WB = decltype(wb)::value;
            constexpr int LPR = 512 / WB;            // lanes per row (a chunk row is at most 512 bytes)
            constexpr int RPI = 64 / LPR;            // rows per instruction
            constexpr int NI = NJ / RPI;             // instructions per chunk and wave
            typedef typename std::conditional<WB == 16, uint4, uint2>::type V;
            constexpr int PD = kBxProdDepth;
            const int p = wave - kBxConsumers;
            const int rows = B - b0 < 32 ? B - b0 : 32;
            const int half = lane / LPR;
            const int lab = (lane % LPR) * (WB / 2);
            const int gi = lab / G, wl = lab - gi * G;
            // Byte offset within the chunk buffer.  Lanes past the chunk write into the spare
            // bytes at the end of the row, which no consumer reads, so every store is unconditional.
            const bool lane_st = lab < CH * G;
            const uint32_t soff = (lane_st ? (uint32_t)(gi * GB + wl * 2) : (uint32_t)(CH * GB)) + half * NP * RS;
            V v[PD][NI];
            // chunk c (past the last one: all zeros)
            auto load = [&](int c, V (&vv)[NI]) {
                const int64_t lab0 = (g_begin + (int64_t)c * CH) * G;
                const int nlab = (n - c * CH < CH ? n - c * CH : CH) * G;   // this chunk's labels
                const Buf db(dY + (int64_t)b0 * L + lab0, (uint32_t)(((int64_t)rows * L - lab0) * 2));
                // a select, not a branch around the loads (which would cost the waits their depth)
                uint32_t lo = lab < nlab ? (uint32_t)(2 * lab) + (uint32_t)((int64_t)half * NP * L * 2) : kOob;
                asm volatile("" : "+v"(lo));
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    const uint32_t ro = (uint32_t)((int64_t)(p + NP * RPI * i) * L * 2);
                    if constexpr (WB == 16) vv[i] = db.ld16(ro + lo);
                    else vv[i] = db.ld8(ro + lo);
                }
            };
            auto store = [&](int c, const V (&vv)[NI]) {
                char *yb = ys + (c & 1) * cbytes + soff;
#pragma unroll
                for (int i = 0; i < NI; ++i) *reinterpret_cast<V *>(yb + (p + NP * RPI * i) * RS) = vv[i];
            };
#pragma unroll
            for (int j = 0; j < PD; ++j) load(j, v[j]);
            store(0, v[0]);
            load(PD, v[0]);
            // after the barrier of chunk c: chunk c + 1 into the buffer chunk c - 1 used (past the
            // last chunk: unused zeros), then the registers it came from take chunk c + 1 + PD.
            // Whole passes of PD chunks first (no exit inside a pass, so the load waits keep their
            // depth across the loop's back edge), then the remaining chunks.
            int c0 = 0;
            for (; c0 + PD <= nch; c0 += PD) {
#pragma unroll
                for (int j = 0; j < PD; ++j) {
                    __syncthreads();  // chunk c0 + j staged, chunk c0 + j - 1 consumed
                    store(c0 + j + 1, v[(j + 1) % PD]);
                    load(c0 + j + 1 + PD, v[(j + 1) % PD]);
                }
            }
#pragma unroll
            for (int j = 0; j < PD - 1; ++j) {
                if (c0 + j < nch) {
                    __syncthreads();
                    store(c0 + j + 1, v[(j + 1) % PD]);
                }
            }
        };
        if (G % 8 == 0) produce(std::integral_constant<int, 16>{});
        else produce(std::integral_constant<int, 8>{});
    } else {
        // ---- consumers: rows 16bh .. 16bh + 15 of the tile ----
        // (their per-group chain sets the pace: they issue ahead of the producers on a shared SIMD)
        const int bh = wave;
        __builtin_amdgcn_s_setprio(2);
        const int last = n - 1;
        auto cl = [&](int v) { return v < last ? v : last; };

        // This segment's transposed weights and support, addressed by a per-lane offset within
        // a group plus a wave-uniform group offset (the segment spans less than 2 GB).
        const uint32_t gbytes = (uint32_t)(F_IN * Gp * 2);
        const Buf wseg(WT + g_begin * F_IN * Gp, (uint32_t)n * gbytes);
        const Buf iseg(idx + g_begin * F_IN, (uint32_t)(n * F_IN * 4));  // lane-ordered supports
        uint32_t wvo[NLB][NST];
#pragma unroll
        for (int c = 0; c < NLB; ++c)
#pragma unroll
            for (int st = 0; st < NST; ++st) {
                const int o = 4 * c + q;          // label octet; octets past Gp read as zero
                wvo[c][st] = 8 * o < Gp ? (uint32_t)((o * F_IN + 16 * st + l16) * 16) : kOob;
            }
        auto issue = [&](int sg, BwdXGroup<F_IN, NLB> &t) {
#pragma unroll
            for (int c = 0; c < NLB; ++c)
#pragma unroll
                for (int st = 0; st < NST; ++st)
                    t.w[c][st] = __builtin_bit_cast(
                        uint4, __builtin_amdgcn_raw_buffer_load_b128(wseg.r, (int)wvo[c][st], (int)(sg * gbytes), 0));
            // the NST supports of this lane's slots, side by side
            if constexpr (NST == 2) {
                const uint2 v = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(iseg.r, l16 * 8, sg * F_IN * 4, 0));
                t.f[0] = (int)v.x;
                t.f[1] = (int)v.y;
            } else {
#pragma unroll
                for (int h = 0; h < NST / 4; ++h) {
                    const uint4 v = __builtin_bit_cast(
                        uint4, __builtin_amdgcn_raw_buffer_load_b128(iseg.r, (l16 * NST + 4 * h) * 4, sg * F_IN * 4, 0));
                    t.f[4 * h + 0] = (int)v.x;
                    t.f[4 * h + 1] = (int)v.y;
                    t.f[4 * h + 2] = (int)v.z;
                    t.f[4 * h + 3] = (int)v.w;
                }
            }
        };

        // this lane's dY operand: row 16 bh + l16 of a group, labels 32c + 8q .. +7
        const char *ylane = ys + (16 * bh + l16) * RS + 16 * q;
        // this lane's accumulator chunk: rows 16 bh + 4q .. +3 of an accumulator row
        typedef __attribute__((address_space(3))) f32x4_t lds_f32x4_t;
        const uint32_t abase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float *)accs;
        const uint32_t achunk = (uint32_t)((4 * bh + q) << 4);
        auto read_dy = [&](uint4 (&ay)[NLB], const char *yp) {
#pragma unroll
            for (int c = 0; c < NLB; ++c) ay[c] = *reinterpret_cast<const uint4 *>(yp + 64 * c);
        };

        auto acc_addr = [&](int f) {   // f: acc_row of the accumulator row
            uint32_t ao = ((uint32_t)f ^ achunk) + abase;
            asm volatile("" : "+v"(ao));   // computed once, kept for the write
            return ao;
        };
        auto acc_read = [&](uint32_t ao) { return *(lds_f32x4_t *)(uintptr_t)ao; };
        auto acc_write = [&](uint32_t ao, const f32x4_t &v) { *(lds_f32x4_t *)(uintptr_t)ao = v; };

        // Group g's weights live in buffer g % NB, loaded NB - 1 groups ahead (clamped index past
        // the end, so every wait covers only its own loads); its dY operand is read one step ahead,
        // in buffer g % 2.  One unrolled pass covers NB groups, and a chunk holds CH = m NB groups,
        // so a chunk ends after the last step of every m-th pass: there the consumers wait for the
        // next chunk (if the segment has one) and switch buffers.
        BwdXGroup<F_IN, NLB> tl[NB];
        uint4 ay[2][NLB];
#pragma unroll
        for (int b = 0; b < NB - 1; ++b) {
            issue(cl(b), tl[b]);
            __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
        }
        const int m = CH / NB;                           // passes per chunk
        const int n_pad = (n + NB - 1) / NB * NB;        // at most nch CH, as NB divides CH
        const int nst = nch * CH;                        // groups staged, zeros past n included
        int ic = 0;            // pass within the chunk
        int ybuf = 0;          // byte offset of the chunk buffer in use
        // dY operand of group s0 + b + 1, read during step b of the pass starting at s0
        auto next_dy = [&](int b, int s0, const char *yit, uint4 (&ay)[NLB]) {
            if (b < NB - 1) {
                read_dy(ay, yit + (b + 1) * GB);
            } else {
                if (++ic == m) {
                    ic = 0;
                    ybuf = cbytes - ybuf;
                    if (s0 + NB < nst) __syncthreads();   // the next chunk is staged
                }
                read_dy(ay, ylane + ybuf + ic * (NB * GB));
            }
        };

        __syncthreads();                                 // chunk 0 staged
        read_dy(ay[0], ylane);
        int s0 = 0;
        // Step s: read the accumulator rows of group s; refill the buffer group s - 1 has finished
        // with (the load issue overlaps the LDS reads); read the dY operand of group s + 1; then
        // D = dZ_s W_s + old through the matrix core (its accumulator input) and write D back.
        for (; s0 < n_pad; s0 += NB) {
            const char *yit = ylane + ybuf + ic * (NB * GB);   // group s0 of this pass
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int sg = s0 + b;
                f32x4_t acc[NST];
                uint32_t ao[NST];
#pragma unroll
                for (int st = 0; st < NST; ++st) {
                    ao[st] = acc_addr(tl[b].f[st]);
                    acc[st] = acc_read(ao[st]);
                }
                __builtin_amdgcn_sched_barrier(0);  // accumulator reads first
                issue(cl(sg + NB - 1), tl[(b + NB - 1) % NB]);
                __builtin_amdgcn_sched_barrier(0);  // keep prefetch order
                next_dy(b, s0, yit, ay[(b + 1) & 1]);
#pragma unroll
                for (int st = 0; st < NST; ++st) {
#pragma unroll
                    for (int c = 0; c < NLB; ++c)
                        acc[st] = mfma16x16x32(as_bf16x8(ay[b & 1][c]), as_bf16x8(tl[b].w[c][st]), acc[st]);
                    acc_write(ao[st], acc[st]);
                }
            }
        }
    }
    __syncthreads();
    for (int e = tid; e < F_s * 32; e += nthr) {
        const int f = e >> 5, b = e & 31;
        pp[(size_t)f * Bp + b] = accs[acc_index(f, b)];
    }
}

// ---------------------------------------------------------------------------------------------
// launch geometry
// ---------------------------------------------------------------------------------------------

constexpr size_t kLdsBudget = 160 * 1024;

template <typename Kern>
hipError_t allow_lds(Kern k, size_t bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void *>(k), hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)bytes);
}

struct BwdXGeom {
    int nbt, nwaves, ch;
    int64_t nseg, gps;
    size_t lds;
};

BwdXGeom bwd_x_geom(const haste::TailArgs &a) {
    BwdXGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    g.nwaves = kBxConsumers + kBxProducers;
    // groups per staged dY chunk: at most 256 labels (one 512-byte load per row), kBxChunkBytes and
    // what the LDS holds beside the accumulator, rounded down to a multiple of the prefetch depth
    const int nlb = (int)((a.G + 31) / 32), gb = 32 * 64 * nlb;   // staged bytes per group
    int ch = (int)(256 / a.G) < kBxChunkBytes / gb ? (int)(256 / a.G) : kBxChunkBytes / gb;
    const int nb = bx_depth_for(a.F_in, nlb);
    auto stage = [&](int c) { return (int64_t)2 * 32 * bx_stage_row_bytes(nlb, c); };   // both buffers
    while (ch > 0 && (int64_t)a.F_s * 128 + stage(ch) > (int64_t)kLdsBudget) --ch;
    g.ch = ch / nb * nb;
    g.lds = (size_t)a.F_s * 128 + (size_t)stage(g.ch);
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
// Byte offsets within 64 rows of the [B, L] logits must fit the 31-bit buffer range.
bool fwd_mfma_supported(const TailArgs &a) {
    return a.dtype == HASTE_DTYPE_BF16 && a.G >= 4 && (a.G % 4) == 0 &&
           (a.F_in == 32 || a.F_in == 64 || a.F_in == 128) && (a.F_s % 2) == 0 && a.F_s <= kMaxFs &&
           a.L * 128 < ((int64_t)1 << 31);
}

static size_t fwd_lds(int BT, int F_s) {
    const size_t xt = ((size_t)F_s * (BT + kFwdXtPad) * 2 + 15) & ~(size_t)15;
    return xt + (size_t)(BT == 64 ? 8 : 4) * 32 * kFwdStageRow;
}

template <int BT, int F_IN, bool HAS_BIAS, bool WIDE>
static hipError_t launch_fwd(const TailArgs &a, const void *X, const int32_t *idx, const void *W,
                             const float *bias, void *Y, hipStream_t s) {
    const int threads = BT == 64 ? 512 : 256;
    const size_t lds = fwd_lds(BT, (int)a.F_s);
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
    auto kern = k_fwd<BT, F_IN, HAS_BIAS, WIDE>;
    hipError_t e = allow_lds(kern, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(threads), lds, s, (const bf16_t *)X, idx, (const bf16_t *)W,
                       bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, a.L, (int)a.G, K, nbt, gps);
    return hipGetLastError();
}

template <int BT, int F_IN>
static hipError_t launch_fwd_b(const TailArgs &a, const void *X, const int32_t *idx, const void *W,
                               const float *bias, void *Y, hipStream_t s) {
    // 16-byte stores need whole 8-label chunks: groups of a multiple of 8 labels, aligned logits
    const bool wide = (a.G % 8) == 0 && (reinterpret_cast<uintptr_t>(Y) & 15) == 0;
    if (wide)
        return bias ? launch_fwd<BT, F_IN, true, true>(a, X, idx, W, bias, Y, s)
                    : launch_fwd<BT, F_IN, false, true>(a, X, idx, W, bias, Y, s);
    return bias ? launch_fwd<BT, F_IN, true, false>(a, X, idx, W, bias, Y, s)
                : launch_fwd<BT, F_IN, false, false>(a, X, idx, W, bias, Y, s);
}

hipError_t fwd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s) {
    // 64-row slabs halve the weight re-reads once the batch is large enough (and the slab fits)
    const bool big = a.B > 32 && fwd_lds(64, (int)a.F_s) <= kLdsBudget;
    switch (a.F_in) {
        case 32: return big ? launch_fwd_b<64, 32>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 32>(a, X, idx, W, bias, Y, s);
        case 64: return big ? launch_fwd_b<64, 64>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 64>(a, X, idx, W, bias, Y, s);
        case 128: return big ? launch_fwd_b<64, 128>(a, X, idx, W, bias, Y, s) : launch_fwd_b<32, 128>(a, X, idx, W, bias, Y, s);
    }
    return hipErrorInvalidValue;
}

// ---- backward-weight ----------------------------------------------------------------------------
bool bwd_w_mfma_supported(const TailArgs &a) { return fwd_mfma_supported(a); }

// X^T staged in 32-row batch blocks (the batch padded to whole blocks)
size_t bwd_w_mfma_ws(const TailArgs &a) { return (size_t)a.F_s * (size_t)round_up(a.B, 32) * 2 + 256; }

// X^T in 32-row batch blocks, [B/32][F_s][32] (rows past B zero), into the workspace
hipError_t transpose_x(const TailArgs &a, const void *X, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 32);
    hipLaunchKernelGGL(k_transpose_x, dim3((unsigned)cdiv(a.F_s, 32), (unsigned)cdiv(Bp, 32)), dim3(256), 0, s,
                       (const bf16_t *)X, reinterpret_cast<bf16_t *>(ws), (int)a.B, (int)a.F_s);
    return hipGetLastError();
}

hipError_t bwd_w_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 32);
    bf16_t *Xb = reinterpret_cast<bf16_t *>(ws);
    hipLaunchKernelGGL(k_transpose_x, dim3((unsigned)cdiv(a.F_s, 32), (unsigned)cdiv(Bp, 32)), dim3(256), 0, s,
                       (const bf16_t *)X, Xb, (int)a.B, (int)a.F_s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t K = a.L / a.G;
    const int64_t units = K * cdiv(a.G, 32);
    {
        const size_t lds = bw2_lds((int)a.F_s, (int)a.F_in);
        const dim3 grid2((unsigned)cdiv(units, kBw2Units));
        auto launch2 = [&](auto kern) {
            hipError_t e2 = allow_lds(kern, lds);
            if (e2 != hipSuccess) return e2;
            hipLaunchKernelGGL(kern, grid2, dim3(kBw2Waves * 64), lds, s, Xb, idx, (const bf16_t *)dY, dW, dbias, beta,
                               (int)a.B, Bp, (int)a.F_s, a.L, (int)a.G, K);
            return hipGetLastError();
        };
        switch (a.F_in) {
            case 32: return launch2(k_bwd_w2<32>);
            case 64: return launch2(k_bwd_w2<64>);
            case 128: return launch2(k_bwd_w2<128>);
            default: break;
        }
    }
    return hipErrorInvalidValue;
}

// ---- forward with the BCE-gradient epilogue, fused with backward-weight -------------------------
// Groups of whole 16-label tiles (the staged dY columns of a wave's units stay contiguous) and
// inputs of at most kFbMaxFs features; any number of positives per row (more than kFbMaxPos are
// bucketed by a pre-pass, in the workspace).
bool fwd_bce_mfma_supported(const TailArgs &a, int P) {
    return bwd_w_mfma_supported(a) && (a.G % 16) == 0 && a.F_s <= kFbMaxFs && P >= 0 &&
           a.B * (int64_t)P < ((int64_t)1 << 29) && fb_lds((int)a.F_s, (int)a.F_in, false) <= kLdsBudget;
}

// the fused kernel's (workgroup, slab) cells: workgroups of fb_waves units, slabs of 32 rows
struct FbCells {
    int ntn, nw, nslab;
    int64_t nwg, ncell;
};

static FbCells fb_cells(const TailArgs &a) {
    FbCells c;
    c.ntn = (int)cdiv(a.G, 32);
    c.nw = fb_waves((int)a.F_in);
    c.nslab = (int)(round_up(a.B, 32) / 32);
    c.nwg = cdiv((a.L / a.G) * c.ntn, c.nw);
    c.ncell = c.nwg * c.nslab;
    return c;
}

// workspace of the bucketed positives (rows of more than kFbMaxPos): per-cell counts, offsets and
// the entries
static size_t fb_pos_ws(const TailArgs &a, int P) {
    if (P <= kFbMaxPos) return 0;
    const FbCells c = fb_cells(a);
    return (size_t)(round_up(c.ncell * 4, 256) + round_up((c.ncell + 1) * 4, 256) + round_up(a.B * (int64_t)P * 4, 256));
}

size_t fwd_bce_mfma_ws(const TailArgs &a, int P) { return bwd_w_mfma_ws(a) + fb_pos_ws(a, P); }

// cell of the positive (row b, label col), and the first label of a workgroup's span
__device__ __forceinline__ int64_t fb_cell_of(int64_t col, int b, int G, int ntn, int nw, int nslab) {
    const int64_t k = col / G;
    const int64_t unit = k * ntn + (col - k * G) / 32;
    return (unit / nw) * nslab + (b >> 5);
}

__device__ __forceinline__ int64_t fb_span_start(int64_t w, int G, int ntn, int nw) {
    const int64_t v = w * nw, k = v / ntn;
    return k * G + 32 * (v - k * ntn);
}

__global__ void k_fb_pos_count(const int32_t *__restrict__ pos, int B, int P, int64_t L, int G, int ntn, int nw,
                               int nslab, int32_t *__restrict__ cnt) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * P) return;
    const int64_t col = pos[i];
    if (col < 0 || col >= L) return;   // outside the layer: ignored
    atomicAdd(&cnt[fb_cell_of(col, (int)(i / P), G, ntn, nw, nslab)], 1);
}

// cofs = exclusive prefix sums of cnt (cofs[ncell] = total), and cnt cleared for use as cursors
// (one workgroup of 1024 threads, each over a contiguous run of cells)
__global__ __launch_bounds__(1024) void k_fb_pos_scan(int32_t *__restrict__ cnt, int64_t ncell,
                                                      int32_t *__restrict__ cofs) {
    __shared__ int32_t s[1024];
    const int64_t per = (ncell + 1023) / 1024;
    const int64_t c0 = threadIdx.x * per, c1 = c0 + per < ncell ? c0 + per : ncell;
    int32_t tot = 0;
    for (int64_t c = c0; c < c1; ++c) tot += cnt[c];
    s[threadIdx.x] = tot;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
        const int32_t v = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
        __syncthreads();
        s[threadIdx.x] += v;
        __syncthreads();
    }
    int32_t run = s[threadIdx.x] - tot;
    for (int64_t c = c0; c < c1; ++c) {
        const int32_t n = cnt[c];
        cofs[c] = run;
        cnt[c] = 0;
        run += n;
    }
    if (threadIdx.x == 1023) cofs[ncell] = s[1023];
}

// entries (row in slab) << 16 | (label - span start), in cell order (order within a cell is free:
// the kernel only ORs them into a bitmap)
__global__ void k_fb_pos_fill(const int32_t *__restrict__ pos, int B, int P, int64_t L, int G, int ntn, int nw,
                              int nslab, const int32_t *__restrict__ cofs, int32_t *__restrict__ cur,
                              uint32_t *__restrict__ cent) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * P) return;
    const int64_t col = pos[i];
    if (col < 0 || col >= L) return;
    const int b = (int)(i / P);
    const int64_t cell = fb_cell_of(col, b, G, ntn, nw, nslab);
    const int slot = atomicAdd(&cur[cell], 1);
    const int64_t o = col - fb_span_start(cell / nslab, G, ntn, nw);
    cent[cofs[cell] + slot] = ((uint32_t)(b & 31) << 16) | (uint32_t)o;
}

struct FbArgs {
    const bf16_t *Xb;
    const int32_t *idx;
    const void *W;
    const float *bias;
    const int32_t *pos;
    int P;
    void *dY;
    float *dW, *dbias;
    int beta;
    haste_sgd_t opt;
    float *m;
    void *W_next;
    int Bp;
    bf16_t *WT;       // transposed weights and lane-ordered supports for backward-feature, or null
    int32_t *idxl;
    const int32_t *cofs = nullptr;   // bucketed positives (rows of more than kFbMaxPos), or null
    const uint32_t *cent = nullptr;
    int64_t n_ent = 0;
};

template <int F_IN, int OUT, bool BK, bool DBX, class Go>
static hipError_t launch_fwd_bce_k(const FbArgs &f, Go &go) {
    if constexpr (OUT == kFbOutNone)
        return f.bias ? go(k_fwd_bce<F_IN, true, OUT, false, BK, DBX>) : go(k_fwd_bce<F_IN, false, OUT, false, BK, DBX>);
    if (f.dbias)
        return f.bias ? go(k_fwd_bce<F_IN, true, OUT, true, BK, DBX>) : go(k_fwd_bce<F_IN, false, OUT, true, BK, DBX>);
    return f.bias ? go(k_fwd_bce<F_IN, true, OUT, false, BK, DBX>) : go(k_fwd_bce<F_IN, false, OUT, false, BK, DBX>);
}

template <int F_IN, int OUT>
static hipError_t launch_fwd_bce(const TailArgs &a, const FbArgs &f, hipStream_t s) {
    const int64_t K = a.L / a.G;
    const int64_t units = K * cdiv(a.G, 32);
    // a second X^T block where the LDS holds it (inputs of up to 768 features)
    const bool dbx = fb_lds((int)a.F_s, F_IN, true) <= kLdsBudget;
    size_t lds = fb_lds((int)a.F_s, F_IN, dbx);
    if (f.WT && lds < (size_t)fb_waves(F_IN) * fb_wt_region(F_IN)) lds = (size_t)fb_waves(F_IN) * fb_wt_region(F_IN);
    const dim3 grid((unsigned)cdiv(units, fb_waves(F_IN)));
    auto go = [&](auto kern) {
        hipError_t e = allow_lds(kern, lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, grid, dim3(fb_waves(F_IN) * 64), lds, s, f.Xb, f.idx, (const bf16_t *)f.W, f.bias,
                           f.pos, f.P, (bf16_t *)f.dY, f.dW, f.dbias, f.beta, f.opt.lr, f.opt.momentum,
                           f.opt.weight_decay, f.m, (bf16_t *)f.W_next, (int)a.B, f.Bp, (int)a.F_s, a.L, (int)a.G, K,
                           f.WT, f.idxl, f.cofs, f.cent, f.n_ent);
        return hipGetLastError();
    };
    if (dbx) return f.cofs ? launch_fwd_bce_k<F_IN, OUT, true, true>(f, go) : launch_fwd_bce_k<F_IN, OUT, false, true>(f, go);
    return f.cofs ? launch_fwd_bce_k<F_IN, OUT, true, false>(f, go) : launch_fwd_bce_k<F_IN, OUT, false, false>(f, go);
}

template <int OUT>
static hipError_t fwd_bce_dispatch(const TailArgs &a, const void *X, FbArgs &f, void *ws, hipStream_t s) {
    f.Bp = (int)round_up(a.B, 32);
    bf16_t *Xb = reinterpret_cast<bf16_t *>(ws);
    f.Xb = Xb;
    hipLaunchKernelGGL(k_transpose_x, dim3((unsigned)cdiv(a.F_s, 32), (unsigned)cdiv(f.Bp, 32)), dim3(256), 0, s,
                       (const bf16_t *)X, Xb, (int)a.B, (int)a.F_s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (f.P > kFbMaxPos) {   // bucket the positives by (workgroup, slab) cell
        const FbCells c = fb_cells(a);
        char *pw = reinterpret_cast<char *>(ws) + bwd_w_mfma_ws(a);
        int32_t *cnt = reinterpret_cast<int32_t *>(pw);
        int32_t *cofs = reinterpret_cast<int32_t *>(pw + round_up(c.ncell * 4, 256));
        uint32_t *cent = reinterpret_cast<uint32_t *>(pw + round_up(c.ncell * 4, 256) + round_up((c.ncell + 1) * 4, 256));
        const int64_t n = a.B * (int64_t)f.P;
        e = fill_f32(reinterpret_cast<float *>(cnt), c.ncell, 0.0f, s);   // all-zero bits: integer zeros
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_fb_pos_count, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, f.pos, (int)a.B, f.P, a.L,
                           (int)a.G, c.ntn, c.nw, c.nslab, cnt);
        hipLaunchKernelGGL(k_fb_pos_scan, dim3(1), dim3(1024), 0, s, cnt, c.ncell, cofs);
        hipLaunchKernelGGL(k_fb_pos_fill, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, f.pos, (int)a.B, f.P, a.L,
                           (int)a.G, c.ntn, c.nw, c.nslab, cofs, cnt, cent);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        f.cofs = cofs;
        f.cent = cent;
        f.n_ent = n;
    }
    switch (a.F_in) {
        case 32: return launch_fwd_bce<32, OUT>(a, f, s);
        case 64: return launch_fwd_bce<64, OUT>(a, f, s);
        case 128: return launch_fwd_bce<128, OUT>(a, f, s);
    }
    return hipErrorInvalidValue;
}

hipError_t fwd_bce_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                        const int32_t *pos, int P, void *dY, float *dW, float *dbias, int beta, void *ws,
                        hipStream_t s) {
    FbArgs f{nullptr, idx, W, bias, pos, P, dY, dW, dbias, beta, haste_sgd_t{0.f, 0.f, 0.f, 0}, nullptr, nullptr, 0,
             nullptr, nullptr};
    return dW ? fwd_bce_dispatch<kFbOutDW>(a, X, f, ws, s) : fwd_bce_dispatch<kFbOutNone>(a, X, f, ws, s);
}

hipError_t fwd_bce_sgd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                            const int32_t *pos, int P, void *dY, float *dbias, const haste_sgd_t &opt, float *m,
                            void *W_next, void *ws, hipStream_t s) {
    FbArgs f{nullptr, idx, W, bias, pos, P, dY, nullptr, dbias, 0, opt, m, W_next, 0, nullptr, nullptr};
    return fwd_bce_dispatch<kFbOutSGD>(a, X, f, ws, s);
}

// ---- backward-feature ---------------------------------------------------------------------------
// Groups of up to 128 labels (four 32-label blocks held in registers per group), at least two
// groups per staged dY chunk, and the accumulator plus the staging buffers within the LDS.
bool bwd_x_mfma_supported(const TailArgs &a) {
    if (!fwd_mfma_supported(a) || a.G > 128) return false;
    const BwdXGeom g = bwd_x_geom(a);
    return g.ch > 0 && g.lds <= kLdsBudget;
}

// workspace: the per-segment partials, then W^T (group blocks [Gp / 8][F_in][8]), then the supports
// in lane order
static size_t bwd_x_part_bytes(const TailArgs &a, const BwdXGeom &g) {
    return round_up((int64_t)g.nseg * a.F_s * (g.nbt * 32) * 4, 256);
}

static size_t bwd_x_wt_bytes(const TailArgs &a) {
    return (size_t)round_up((a.L / a.G) * a.F_in * round_up(a.G, 8) * 2, 256);
}

size_t bwd_x_mfma_ws(const TailArgs &a) {
    const BwdXGeom g = bwd_x_geom(a);
    const int64_t K = a.L / a.G;
    return bwd_x_part_bytes(a, g) + bwd_x_wt_bytes(a) + (size_t)round_up(K * a.F_in * 4, 256) + 256;
}

template <int F_IN, int NLB>
static hipError_t launch_bwd_x(const TailArgs &a, const BwdXGeom &g, const int32_t *idx, const bf16_t *WT,
                               const void *dY, float *part, hipStream_t s) {
    auto kern = k_bwd_x<F_IN, NLB>;
    hipError_t e = allow_lds(kern, g.lds);
    if (e != hipSuccess) return e;
    const int64_t K = a.L / a.G;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(g.nwaves * 64), g.lds, s, idx, WT,
                       (const bf16_t *)dY, part, (int)a.B, g.nbt * 32, (int)a.F_s, a.L, (int)a.G,
                       (int)round_up(a.G, 8), K, g.nbt, g.gps, g.ch);
    return hipGetLastError();
}

template <int F_IN>
static hipError_t launch_bwd_x_g(const TailArgs &a, const BwdXGeom &g, const int32_t *idx, const bf16_t *WT,
                                 const void *dY, float *part, hipStream_t s) {
    switch ((a.G + 31) / 32) {
        case 1: return launch_bwd_x<F_IN, 1>(a, g, idx, WT, dY, part, s);
        case 2: return launch_bwd_x<F_IN, 2>(a, g, idx, WT, dY, part, s);
        case 3: return launch_bwd_x<F_IN, 3>(a, g, idx, WT, dY, part, s);
        case 4: return launch_bwd_x<F_IN, 4>(a, g, idx, WT, dY, part, s);
    }
    return hipErrorInvalidValue;
}

static hipError_t bwd_x_main(const TailArgs &a, const BwdXGeom &g, const int32_t *idxl, const bf16_t *WT,
                             const void *dY, float *part, float *dX, int beta, hipStream_t s);

hipError_t bwd_x_mfma(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s) {
    const BwdXGeom g = bwd_x_geom(a);
    float *part = reinterpret_cast<float *>(ws);
    bf16_t *WT = reinterpret_cast<bf16_t *>(reinterpret_cast<char *>(ws) + bwd_x_part_bytes(a, g));
    int32_t *idxl = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(WT) + bwd_x_wt_bytes(a));
    const int64_t K = a.L / a.G;
    const int Gp = (int)round_up(a.G, 8);
    const int64_t tgrid = cdiv(K, kTwWaves) < 4096 ? cdiv(K, kTwWaves) : 4096;
    const size_t tlds = (size_t)kTwWaves * tw_wave_bytes((int)a.F_in, Gp);
    hipError_t e = allow_lds(k_transpose_w, tlds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_transpose_w, dim3((unsigned)tgrid), dim3(kTwWaves * 64), tlds, s, (const bf16_t *)W, idx,
                       WT, idxl, K, (int)a.G, Gp, (int)a.F_in);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return bwd_x_main(a, g, idxl, WT, dY, part, dX, beta, s);
}

// the main kernel and the reduction, on transposed weights and lane-ordered supports already built
static hipError_t bwd_x_main(const TailArgs &a, const BwdXGeom &g, const int32_t *idxl, const bf16_t *WT,
                             const void *dY, float *part, float *dX, int beta, hipStream_t s) {
    hipError_t e = hipSuccess;
    switch (a.F_in) {
        case 32: e = launch_bwd_x_g<32>(a, g, idxl, WT, dY, part, s); break;
        case 64: e = launch_bwd_x_g<64>(a, g, idxl, WT, dY, part, s); break;
        case 128: e = launch_bwd_x_g<128>(a, g, idxl, WT, dY, part, s); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 32, a.B, a.F_s, dX, beta, s);
}

// ---- the tail's training pass: fused forward + loss gradient + dW, then backward-feature ----------
// Groups of 32 labels, where a fused-kernel wave's unit is one group: that kernel also writes the
// transposed weights and lane-ordered supports backward-feature reads (the pre-pass is skipped).
bool tail_step_fused(const TailArgs &a, int P) {
    return a.G == 32 && fwd_bce_mfma_supported(a, P) && bwd_x_mfma_supported(a);
}

size_t tail_step_ws(const TailArgs &a, int P) { return round_up(bwd_x_mfma_ws(a), 256) + fwd_bce_mfma_ws(a, P); }

hipError_t tail_step_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                          const int32_t *pos, int P, void *dY, float *dW, float *dbias, int beta, float *dX,
                          int beta_dx, void *ws, hipStream_t s) {
    const BwdXGeom g = bwd_x_geom(a);
    char *wb = reinterpret_cast<char *>(ws);
    float *part = reinterpret_cast<float *>(wb);
    bf16_t *WT = reinterpret_cast<bf16_t *>(wb + bwd_x_part_bytes(a, g));
    int32_t *idxl = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(WT) + bwd_x_wt_bytes(a));
    FbArgs f{nullptr, idx, W, bias, pos, P, dY, dW, dbias, beta, haste_sgd_t{0.f, 0.f, 0.f, 0}, nullptr, nullptr, 0,
             WT, idxl};
    hipError_t e = fwd_bce_dispatch<kFbOutDW>(a, X, f, wb + round_up(bwd_x_mfma_ws(a), 256), s);
    if (e != hipSuccess) return e;
    return bwd_x_main(a, g, idxl, WT, dY, part, dX, beta_dx, s);
}

// the same pass with the momentum step in the fused kernel (dW never stored); the transposed
// weights it hands over are those of the step's W, read before the update
hipError_t tail_step_sgd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                              const int32_t *pos, int P, void *dY, float *dbias, const haste_sgd_t &opt, float *m,
                              void *W_next, float *dX, int beta_dx, void *ws, size_t fb_ws_bytes, hipStream_t s) {
    (void)fb_ws_bytes;
    const BwdXGeom g = bwd_x_geom(a);
    char *wb = reinterpret_cast<char *>(ws);
    float *part = reinterpret_cast<float *>(wb);
    bf16_t *WT = reinterpret_cast<bf16_t *>(wb + bwd_x_part_bytes(a, g));
    int32_t *idxl = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(WT) + bwd_x_wt_bytes(a));
    FbArgs f{nullptr, idx, W, bias, pos, P, dY, nullptr, dbias, 0, opt, m, W_next, 0, WT, idxl};
    hipError_t e = fwd_bce_dispatch<kFbOutSGD>(a, X, f, wb + round_up(bwd_x_mfma_ws(a), 256), s);
    if (e != hipSuccess) return e;
    return bwd_x_main(a, g, idxl, WT, dY, part, dX, beta_dx, s);
}

}  // namespace haste
