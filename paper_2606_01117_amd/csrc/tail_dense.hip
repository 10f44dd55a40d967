// Backward-feature for small groups as a dense matrix-core product over scattered weight tiles
// (bf16, G in {1, 2, 4, 8}).
//
//   dX[rows, f] = sum over labels l of dY[rows, l] W'[l, f],   W'[l, f] = W[l, t] where
//   idx[g(l), t] = f, and 0 where f is not in the support of l's group   (Section 3.2, the
//   backward-feature product; W' is the weight grid of Fig. 2 (d) with its empty cells as zeros).
//
// With G <= 8 a group's tile of the segmented-accumulator kernels is mostly padding, and their
// LDS traffic per (label, slot, row) is a 4-byte read and a 4-byte write of the accumulator.  Here
// the accumulator never leaves the registers: a workgroup owns 32 batch rows and all F_s features
// (dX^T [F_s][32] fp32 spread over its 8 waves' matrix-core accumulators) for a segment of
// labels.  Per step of 32 labels:
//   - the step's weights are scattered into a zeroed [F_s][32] bf16 tile in LDS (one 2-byte write
//     per (label, slot): W'[l, idx[g(l), t]] = W[l, t]), and cleared with the same writes after use;
//   - D += A B with A = dY[32 rows][32 labels] (staged in LDS) and B = the tile, F_s / 16 tiles
//     of v_mfma_f32_16x16x32_bf16 per row half: K = the step's labels, in natural order.
// Three tiles rotate: step t + 1 is scattered and step t - 1 cleared while step t is multiplied,
// with one barrier per step.  Each 32-label half of a 64-label round is scattered by one half of
// the waves (a lane: one label, F_in / 8 consecutive slots), which also clears what it wrote two
// steps earlier, so a clear and a later write of the same cell are ordered by that barrier.
// Segments of labels are summed by the fixed-order reduction over segment partials; the result is
// bit-reproducible and uses no atomics.
#include "common.hpp"

namespace {

constexpr int kDnWaves = 8;
constexpr int kDnThreads = 64 * kDnWaves;
constexpr int kDnStageRow = 160;                 // bytes per staged dY row: 64 labels + pad
constexpr int kDnStage = 32 * kDnStageRow;       // one round's staged dY block [32 rows][64 labels]

// the [FR][32] bf16 weight tile: row f is 64 bytes, and its 16-byte chunk c (labels 8c .. 8c+7)
// sits at chunk position c ^ ((f >> 2) mod 4), which spreads a step's scattered writes over all
// 64 banks (the matrix-core operand reads, 16 whole rows at a time, stay conflict-free)
__host__ __device__ constexpr int dn_tile_bytes(int fr) { return fr * 64; }
__host__ __device__ constexpr int dn_lds(int fr) { return 3 * dn_tile_bytes(fr) + 2 * kDnStage + 64; }

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint16_t lds_u16_t;
typedef __attribute__((address_space(3))) u32x2_t lds_u32x2_t;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;
typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;

// NFT: 16-feature tiles per wave (wave w owns tiles w, w + 8, ...), so F_s <= 128 NFT.
// TAIL2: L = 2 mod 4 (the last dY piece of a row holds two labels).
template <int F_IN, int NFT, bool TAIL2>
__global__ __launch_bounds__(kDnThreads) void k_bwd_x_dn(const int32_t *__restrict__ idx, const bf16_t *__restrict__ W,
                                                         const bf16_t *__restrict__ dY, float *__restrict__ part, int B,
                                                         int Bp, int F_s, int FR, int64_t L, int gshift, int nbt,
                                                         int64_t lps) {
    constexpr int E = F_IN / 8;                   // slots per lane and round
    constexpr int NW = E / 2;                     // dwords of weights per lane and round
    static_assert(E % 4 == 0, "whole 16-byte support loads");
    extern __shared__ __align__(16) char dn[];    // 3 tiles, then [2] staged rounds, then a dummy cell
    const int w = blockIdx.x, xcd = w % kXcds, jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const int NT = FR / 16;                       // feature tiles
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    const int64_t l_begin = seg * lps;
    const int64_t l_end = l_begin + lps < L ? l_begin + lps : L;
    if (l_begin >= l_end) {   // empty segment: the partial is zero (workgroup-uniform)
        for (int e = tid; e < F_s * 32; e += kDnThreads) pp[(size_t)(e >> 5) * Bp + (e & 31)] = 0.0f;
        return;
    }
    const int nr = (int)((l_end - l_begin + 63) / 64);   // rounds of 64 labels; 2 nr steps
    const int TB = dn_tile_bytes(FR);
    const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)dn;
    const uint32_t sbase = lbase + 3 * TB;        // staged dY
    const uint32_t dummy = sbase + 2 * kDnStage;  // written by the first clear, never read

    for (int e = tid; e < 3 * TB / 16; e += kDnThreads)
        *(lds_u32x4_t *)(uintptr_t)(lbase + 16 * e) = u32x4_t{0u, 0u, 0u, 0u};

    // ---- per-lane roles ----
    // scatter: half h of the waves takes the round's labels 32 h .. 32 h + 31, i.e. step 2R + h;
    // lane -> label 8 (wave mod 4) + lane / 8 of the step, slots E (lane mod 8) .. + E - 1
    const int h = wave >> 2;
    const int ls = 8 * (wave & 3) + (lane >> 3);  // label within its step
    const int o = lane & 7;
    const uint32_t lpos = (uint32_t)(((ls >> 3) << 4) | ((ls & 7) << 1));   // chunk and label bits
    const Buf wseg(W + l_begin * F_IN, (uint32_t)((l_end - l_begin) * F_IN * 2));
    const int64_t g_begin = l_begin >> gshift;
    const Buf iseg(idx + g_begin * F_IN, (uint32_t)(((l_end >> gshift) - g_begin) * F_IN * 4));
    // dY: lane -> row tid / 16, labels 4 (tid mod 16) .. + 3 of the round (8 bytes)
    const int rows = B - b0 < 32 ? B - b0 : 32;
    const int dr = tid >> 4, dp = tid & 15;
    const Buf dseg(dY + (int64_t)b0 * L, (uint32_t)((int64_t)rows * L * 2));

    struct Round {
        uint32_t wv[NW];   // W[l, E o .. E o + E - 1] (bf16 pairs)
        int32_t f[E];      // the same slots' features
        uint2 y;           // dY piece
    };
    Round rg[3];           // round R in slot R mod 3
    auto load_round = [&](int R, Round &r) __attribute__((always_inline)) {
        const int64_t lr = (int64_t)R * 64 + 32 * h + ls;     // label offset within the segment
        const uint32_t wo = (uint32_t)(lr * F_IN * 2 + E * 2 * o);
#pragma unroll
        for (int i = 0; i < NW / 4; ++i) {
            const uint4 x = wseg.ld16(wo + 16 * i);
            r.wv[4 * i] = x.x;
            r.wv[4 * i + 1] = x.y;
            r.wv[4 * i + 2] = x.z;
            r.wv[4 * i + 3] = x.w;
        }
        if constexpr (NW == 2) {
            const uint2 x = wseg.ld8(wo);
            r.wv[0] = x.x;
            r.wv[1] = x.y;
        }
        const int64_t gl = ((l_begin + lr) >> gshift) - g_begin;
        const uint32_t io = (uint32_t)(gl * F_IN * 4 + E * 4 * o);
#pragma unroll
        for (int i = 0; i < E / 4; ++i) {
            const uint4 x = iseg.ld16(io + 16 * i);
            r.f[4 * i] = (int32_t)x.x;
            r.f[4 * i + 1] = (int32_t)x.y;
            r.f[4 * i + 2] = (int32_t)x.z;
            r.f[4 * i + 3] = (int32_t)x.w;
        }
        // dY piece: 4 labels of row dr.  Segments start and end at multiples of 64 labels, except
        // the layer's end, so with L even a piece is whole, past the end, or (L = 2 mod 4) the
        // layer's last two labels, read as one dword so that nothing past the row is read
        const int64_t lab = l_begin + (int64_t)R * 64 + 4 * dp;
        const int64_t nv = l_end - lab;
        const uint32_t yo = dr < rows && nv > 0 ? (uint32_t)(((int64_t)dr * L + lab) * 2) : kOob;
        r.y = dseg.ld8(nv >= 4 ? yo : kOob);
        if constexpr (TAIL2) r.y.x |= dseg.ld4(nv == 2 ? yo : kOob);
    };
    // scatter of a step's lane entries into tile buffer tb; the addresses are kept for the clear
    uint32_t ca[E];
#pragma unroll
    for (int j = 0; j < E; ++j) ca[j] = dummy;
    auto scatter = [&](const Round &r, int tb) __attribute__((always_inline)) {
        const uint32_t base = lbase + (uint32_t)(tb * TB);
#pragma unroll
        for (int j = 0; j < E; ++j) {
            const uint32_t f = (uint32_t)r.f[j];
            ca[j] = base + (f << 6) + (lpos ^ ((f << 2) & 0x30u));
            const uint32_t v = r.wv[j >> 1];
            *(lds_u16_t *)(uintptr_t)ca[j] = (uint16_t)((j & 1) ? (v >> 16) : v);
        }
    };
    auto clear = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < E; ++j) *(lds_u16_t *)(uintptr_t)ca[j] = (uint16_t)0;
    };
    auto store_y = [&](const Round &r, int sb) __attribute__((always_inline)) {
        *(lds_u32x2_t *)(uintptr_t)(sbase + (uint32_t)(sb * kDnStage + dr * kDnStageRow + 8 * dp)) = u32x2_t{r.y.x, r.y.y};
    };

    f32x4_t acc[2][NFT];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
        for (int i = 0; i < NFT; ++i) acc[hh][i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    // operand addresses: A rows 16 hh + l16, labels 8q .. of the step; B rows 16 ft + l16, chunk q
    const uint32_t aoff = sbase + (uint32_t)(l16 * kDnStageRow + 16 * q);
    uint32_t boff[NFT];
#pragma unroll
    for (int i = 0; i < NFT; ++i) {
        const int ft = wave + 8 * i < NT ? wave + 8 * i : NT - 1;   // past the last tile: a repeat, not stored
        boff[i] = lbase + (uint32_t)(ft * 1024 + l16 * 64 + ((q ^ ((l16 >> 2) & 3)) << 4));
    }

    load_round(0, rg[0]);
    load_round(1, rg[1]);
    __syncthreads();                              // tiles zeroed
    if (h == 0) scatter(rg[0], 0);                // step 0
    store_y(rg[0], 0);
    __syncthreads();

    // step t = t0 + U of the unrolled period (U = t mod 6): round t / 2 in ring slot U / 2, tile t mod 3
    auto step = [&](int t, auto uc) __attribute__((always_inline)) {
        constexpr int U = decltype(uc)::value;
        constexpr int PAR = U % 2, RS = U / 2, TBI = U % 3;
        const int R = t >> 1;
        if constexpr (PAR == 0) load_round(R + 2, rg[(RS + 2) % 3]);
        __builtin_amdgcn_sched_barrier(0);
        // step t's operands, all issued before anything else touches the LDS
        const uint32_t ab = aoff + (uint32_t)((R & 1) * kDnStage + PAR * 64);
        const bf16x8_t a0 = *(lds_bf16x8_t *)(uintptr_t)ab;
        const bf16x8_t a1 = *(lds_bf16x8_t *)(uintptr_t)(ab + 16 * kDnStageRow);
        bf16x8_t b[NFT];
#pragma unroll
        for (int i = 0; i < NFT; ++i) b[i] = *(lds_bf16x8_t *)(uintptr_t)(boff[i] + TBI * TB);
        __builtin_amdgcn_sched_barrier(0);
        // scatter step t + 1 (its half), after clearing that half's step t - 1
        if (h != PAR) {
            clear();
            scatter(rg[PAR == 0 ? RS : (RS + 1) % 3], (TBI + 1) % 3);
        }
        if constexpr (PAR == 1) store_y(rg[(RS + 1) % 3], (R + 1) & 1);
        // products of step t
#pragma unroll
        for (int i = 0; i < NFT; ++i) {
            acc[0][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, b[i], acc[0][i], 0, 0, 0);
            acc[1][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, b[i], acc[1][i], 0, 0, 0);
        }
        __syncthreads();
    };
    const int n = 2 * nr;
    int t0 = 0;
    for (; t0 + 6 <= n; t0 += 6)
        static_for<6>([&](auto uc) __attribute__((always_inline)) { step(t0 + decltype(uc)::value, uc); });
    static_for<6>([&](auto uc) __attribute__((always_inline)) {
        if (t0 + decltype(uc)::value < n) step(t0 + decltype(uc)::value, uc);
    });

    // partial dX^T of the segment: lane (l16, q) of tile ft holds feature 16 ft + l16, rows
    // 16 hh + 4q .. + 3
#pragma unroll
    for (int i = 0; i < NFT; ++i) {
        const int f = 16 * (wave + 8 * i) + l16;
        if (wave + 8 * i < NT && f < F_s) {
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                *reinterpret_cast<float4 *>(pp + (size_t)f * Bp + 16 * hh + 4 * q) =
                    make_float4(acc[hh][i][0], acc[hh][i][1], acc[hh][i][2], acc[hh][i][3]);
        }
    }
}

struct DnGeom {
    int nbt, FR, nft;
    int64_t nseg, lps;
    size_t lds;
};

static DnGeom dn_geom(const haste::TailArgs &a) {
    DnGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    g.FR = (int)haste::round_up(a.F_s, 16);
    const int per_wave = (int)haste::cdiv(g.FR / 16, kDnWaves);
    g.nft = per_wave <= 2 ? 2 : per_wave <= 4 ? 4 : per_wave <= 6 ? 6 : per_wave <= 7 ? 7 : 0;
    // one workgroup per CU (the tiles take most of the LDS): segments x batch tiles ~ 256
    int64_t nseg = haste::round_up(haste::cdiv(kXcds * kCusPerXcd, g.nbt), kXcds);
    const int64_t max_seg = haste::round_up(haste::cdiv(a.L, 64), kXcds);
    g.nseg = nseg < max_seg ? nseg : max_seg;
    g.lps = haste::round_up(haste::cdiv(a.L, g.nseg), 64);
    g.lds = (size_t)dn_lds(g.FR);
    return g;
}

template <int F_IN, int NFT>
static hipError_t launch_dn(const haste::TailArgs &a, const DnGeom &g, const int32_t *idx, const void *W,
                            const void *dY, float *part, hipStream_t s) {
    auto kern = a.L % 4 == 2 ? k_bwd_x_dn<F_IN, NFT, true> : k_bwd_x_dn<F_IN, NFT, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)g.lds);
    if (e != hipSuccess) return e;
    const int gshift = a.G == 1 ? 0 : a.G == 2 ? 1 : a.G == 4 ? 2 : 3;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(kDnThreads), g.lds, s, idx, (const bf16_t *)W,
                       (const bf16_t *)dY, part, (int)a.B, g.nbt * 32, (int)a.F_s, g.FR, a.L, gshift, g.nbt, g.lps);
    return hipGetLastError();
}

template <int F_IN>
static hipError_t dn_f(const haste::TailArgs &a, const DnGeom &g, const int32_t *idx, const void *W, const void *dY,
                       float *part, hipStream_t s) {
    switch (g.nft) {
        case 2: return launch_dn<F_IN, 2>(a, g, idx, W, dY, part, s);
        case 4: return launch_dn<F_IN, 4>(a, g, idx, W, dY, part, s);
        case 6: return launch_dn<F_IN, 6>(a, g, idx, W, dY, part, s);
        case 7: return launch_dn<F_IN, 7>(a, g, idx, W, dY, part, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

namespace haste {

// bf16, G in {1, 2, 4, 8}, F_in in {32, 64, 128}; F_s up to the three [F_s][32] tiles the LDS holds
// (800); dY rows dword-aligned (L even) and 32 of them within the 31-bit range of a buffer offset;
// a segment's weight and support offsets within that range too.
bool bwd_x_dn_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2 || a.G == 4 || a.G == 8)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || a.F_in == 128)) return false;
    if (a.F_s <= 0 || a.L % 2 != 0 || a.L * 32 * 2 >= ((int64_t)1 << 31)) return false;
    const DnGeom g = dn_geom(a);
    return g.nft != 0 && g.lds <= 160 * 1024 && (g.lps + 256) * a.F_in * 4 < ((int64_t)1 << 31);
}

size_t bwd_x_dn_ws(const TailArgs &a) {
    const DnGeom g = dn_geom(a);
    return (size_t)round_up(g.nseg * a.F_s * (g.nbt * 32) * 4, 256);
}

hipError_t bwd_x_dn(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta, void *ws,
                    hipStream_t s) {
    const DnGeom g = dn_geom(a);
    float *part = reinterpret_cast<float *>(ws);
    hipError_t e;
    switch (a.F_in) {
        case 32: e = dn_f<32>(a, g, idx, W, dY, part, s); break;
        case 64: e = dn_f<64>(a, g, idx, W, dY, part, s); break;
        case 128: e = dn_f<128>(a, g, idx, W, dY, part, s); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 32, a.B, a.F_s, dX, beta, s);
}

}  // namespace haste
