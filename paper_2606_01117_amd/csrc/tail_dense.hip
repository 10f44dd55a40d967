// Backward-feature for small groups as a dense matrix-core product over scattered weight tiles
// (bf16, G in {1, 2, 4, 8}).
//
//   dX[rows, f] = sum over labels l of dY[rows, l] W'[l, f],   W'[l, f] = W[l, t] where
//   idx[g(l), t] = f, and 0 where f is not in the support of l's group   (Section 3.2, the
//   backward-feature product; W' is the weight grid of Fig. 2 (d) with its empty cells as zeros).
//
// With G <= 8 a group's tile of the segmented-accumulator kernels is mostly padding, and their
// LDS traffic per (label, slot, row) is a 4-byte read and a 4-byte write of the accumulator.  Here
// the accumulator never leaves the registers: a workgroup owns 16 MT batch rows and all F_s
// features (dX^T [F_s][16 MT] fp32 spread over its 8 waves' matrix-core accumulators) for a
// segment of labels.  Per step of 32 labels:
//   - the step's weights are scattered into a zeroed [F_s][32] bf16 tile in LDS (one 2-byte write
//     per (label, slot): W'[l, idx[g(l), t]] = W[l, t]), and cleared with the same writes after use;
//   - D += A B with A = dY[16 MT rows][32 labels] (staged in LDS) and B = the tile, F_s / 16 tiles
//     of v_mfma_f32_16x16x32_bf16 per 16 rows: K = the step's labels, in natural order.
// The scatter costs the same for every row of the workgroup, so more rows per workgroup (MT = 4)
// halve it per row.  Three tiles rotate: step t + 1 is scattered and step t - 1 cleared while
// step t is multiplied, with one barrier per step.  Each 32-label half of a 64-label round is
// scattered by one half of the waves (a lane: one label, F_in / 8 consecutive slots), which also
// clears what it wrote two steps earlier, so a clear and a later write of the same cell are
// ordered by that barrier.  Segments of labels are summed by the fixed-order reduction over
// segment partials; the result is bit-reproducible and uses no atomics.
#include "common.hpp"

namespace {

constexpr int kDnStageRow = 80;                  // bytes per staged dY row: 32 labels + pad

// the [FR][32] bf16 weight tile: row f is 64 bytes, and its 16-byte chunk c (labels 8c .. 8c+7)
// sits at chunk position c ^ ((f >> 2) mod 4), which spreads a step's scattered writes over all
// 64 banks (the matrix-core operand reads, 16 whole rows at a time, stay conflict-free)
__host__ __device__ constexpr int dn_tile_bytes(int fr) { return fr * 64; }
__host__ __device__ constexpr int dn_stage_bytes(int mt) { return 16 * mt * kDnStageRow; }   // one step's dY
__host__ __device__ constexpr int dn_lds(int fr, int mt) { return 3 * dn_tile_bytes(fr) + 2 * dn_stage_bytes(mt) + 64; }

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint16_t lds_u16_t;
typedef __attribute__((address_space(3))) u32x2_t lds_u32x2_t;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;
typedef __attribute__((address_space(3))) bf16x8_t lds_bf16x8_t;

// NWV: waves (8: two per SIMD; 4: one per SIMD, whose 512 registers then hold the accumulators of
// 64 rows).  MT: 16-row tiles per workgroup.  NFT: 16-feature tiles per wave (wave w owns tiles
// w, w + NWV, ...); the tiles have FR = 16 NWV NFT >= F_s rows.  TAILP: L is not a multiple of the
// PL labels of a staged dY piece (the last piece of a row is then read dword by dword).
template <int NWV, int MT, int F_IN, int NFT, bool TAILP>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * NWV, 64 * NWV), amdgpu_waves_per_eu(NWV / 4, NWV / 4)))
void k_bwd_x_dn(const int32_t *__restrict__ idx, const bf16_t *__restrict__ W, const bf16_t *__restrict__ dY,
                float *__restrict__ part, int B, int Bp, int F_s, int FR, int64_t L, int gshift, int nbt,
                int64_t lps) {
    constexpr int T = 64 * NWV;                   // threads
    constexpr int RW = 16 * MT;                   // batch rows of the workgroup
    constexpr int LPL = T / 32;                   // lanes per label of a step
    constexpr int E = F_IN / LPL;                 // slots per lane and step
    constexpr int NW = E / 2;                     // dwords of weights per lane and step
    constexpr int PL = 16 * MT * 32 / T;          // labels per staged dY piece (2 or 8)
    constexpr int PPR = 32 / PL;                  // pieces per row and step
    constexpr int SB = dn_stage_bytes(MT);
    constexpr int RSL = 4;                        // steps whose loads are in flight (ring slots)
    constexpr int PER = 12;                       // unrolled period: multiple of RSL, 3 tiles, 2 parities
    constexpr int NMF = MT * NFT;                 // products per wave and step
    static_assert(E == 2 || E % 4 == 0, "support loads of 8 or 16 bytes");
    static_assert(RW * PPR == T, "one dY piece per thread and step");
    static_assert(PER % RSL == 0 && PER % 6 == 0, "ring period");
    extern __shared__ __align__(16) char dn[];    // 3 tiles, then [2] staged steps, then a dummy cell
    const int w = blockIdx.x, xcd = w % kXcds, jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * RW;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    float *pp = part + (size_t)seg * F_s * Bp + b0;
    const int64_t l_begin = seg * lps;
    const int64_t l_end = l_begin + lps < L ? l_begin + lps : L;
    if (l_begin >= l_end) {   // empty segment: the partial is zero (workgroup-uniform)
        for (int e = tid; e < F_s * RW; e += T) pp[(size_t)(e / RW) * Bp + (e % RW)] = 0.0f;
        return;
    }
    const int n = (int)((l_end - l_begin + 31) / 32);   // steps of 32 labels
    const int TB = dn_tile_bytes(FR);
    const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)dn;
    const uint32_t sbase = lbase + 3 * TB;        // staged dY
    const uint32_t dummy = sbase + 2 * SB;        // written by the first clears, never read

    for (int e = tid; e < 3 * TB / 16; e += T) *(lds_u32x4_t *)(uintptr_t)(lbase + 16 * e) = u32x4_t{0u, 0u, 0u, 0u};

    // ---- per-lane roles ----
    // scatter: lane -> label ls of the step, slots E (tid mod LPL) .. + E - 1.  The labels of one
    // wave should cover the four 4-byte label pairs of a chunk, which with random features spreads
    // an instruction's 2-byte writes over all 64 banks: 8 lanes per label, 8 consecutive labels a
    // wave; 16 lanes per label, labels 2k + j of the chunk (k = 0 .. 3) per wave
    const int gl0 = tid / LPL;
    const int ls = LPL == 8 ? gl0 : 8 * (gl0 >> 3) + 2 * (gl0 & 3) + ((gl0 >> 2) & 1);
    const int o = tid % LPL;
    const uint32_t lpos = (uint32_t)(((ls >> 3) << 4) | ((ls & 7) << 1));   // chunk and label bits
    const Buf wseg(W + l_begin * F_IN, (uint32_t)((l_end - l_begin) * F_IN * 2));
    const int64_t g_begin = l_begin >> gshift;
    const Buf iseg(idx + g_begin * F_IN, (uint32_t)(((l_end >> gshift) - g_begin) * F_IN * 4));
    // dY: lane -> row tid / PPR, labels PL (tid mod PPR) .. + PL - 1 of the step
    const int rows = B - b0 < RW ? B - b0 : RW;
    const int dr = tid / PPR, dp = tid % PPR;
    const Buf dseg(dY + (int64_t)b0 * L, (uint32_t)((int64_t)rows * L * 2));

    struct Slot {
        uint32_t wv[NW];   // W[l, E o .. E o + E - 1] (bf16 pairs)
        int32_t f[E];      // the same slots' features
        uint32_t y[PL / 2];
    };
    Slot rg[RSL];          // step s in slot s mod RSL
    auto load_step = [&](int st, Slot &r) __attribute__((always_inline)) {
        const int64_t lr = (int64_t)st * 32 + ls;             // label offset within the segment
        const uint32_t wo = (uint32_t)(lr * F_IN * 2 + E * 2 * o);
        if constexpr (NW == 1) {
            r.wv[0] = wseg.ld4(wo);
        } else if constexpr (NW == 2) {
            const uint2 x = wseg.ld8(wo);
            r.wv[0] = x.x;
            r.wv[1] = x.y;
        } else {
#pragma unroll
            for (int i = 0; i < NW / 4; ++i) {
                const uint4 x = wseg.ld16(wo + 16 * i);
                r.wv[4 * i] = x.x;
                r.wv[4 * i + 1] = x.y;
                r.wv[4 * i + 2] = x.z;
                r.wv[4 * i + 3] = x.w;
            }
        }
        const int64_t gl = ((l_begin + lr) >> gshift) - g_begin;
        const uint32_t io = (uint32_t)(gl * F_IN * 4 + E * 4 * o);
        if constexpr (E == 2) {
            const uint2 x = iseg.ld8(io);
            r.f[0] = (int32_t)x.x;
            r.f[1] = (int32_t)x.y;
        } else {
#pragma unroll
            for (int i = 0; i < E / 4; ++i) {
                const uint4 x = iseg.ld16(io + 16 * i);
                r.f[4 * i] = (int32_t)x.x;
                r.f[4 * i + 1] = (int32_t)x.y;
                r.f[4 * i + 2] = (int32_t)x.z;
                r.f[4 * i + 3] = (int32_t)x.w;
            }
        }
        // dY piece: PL labels of row dr.  Segments start and end at multiples of 64 labels, except
        // the layer's end, so a piece is whole or past the end unless L is not a multiple of PL;
        // then the layer's last piece of a row is read dword by dword (L is even), so that
        // nothing past the row is read
        const int64_t lab = l_begin + (int64_t)st * 32 + PL * dp;
        const int64_t nv = l_end - lab;
        const uint32_t yo = dr < rows && nv > 0 ? (uint32_t)(((int64_t)dr * L + lab) * 2) : kOob;
        if constexpr (PL == 2) {
            r.y[0] = dseg.ld4(yo);
        } else if constexpr (!TAILP) {
            const uint4 v = dseg.ld16(yo);
            r.y[0] = v.x;
            r.y[1] = v.y;
            r.y[2] = v.z;
            r.y[3] = v.w;
        } else {
#pragma unroll
            for (int k = 0; k < PL / 2; ++k) r.y[k] = dseg.ld4(nv > 2 * k ? yo + 4 * k : kOob);
        }
    };
    // a step's lane entries are written into tile buffer tb, and their addresses kept in ca[] so
    // that the same lanes clear them two steps later
    uint32_t ca[2][E];
#pragma unroll
    for (int j = 0; j < E; ++j) ca[0][j] = ca[1][j] = dummy;
    auto scatter = [&](const Slot &r, int tb, uint32_t (&c)[E]) __attribute__((always_inline)) {
        const uint32_t base = lbase + (uint32_t)(tb * TB);
#pragma unroll
        for (int j = 0; j < E; ++j) {
            const uint32_t f = (uint32_t)r.f[j];
            c[j] = base + (f << 6) + (lpos ^ ((f << 2) & 0x30u));
            const uint32_t v = r.wv[j >> 1];
            *(lds_u16_t *)(uintptr_t)c[j] = (uint16_t)((j & 1) ? (v >> 16) : v);
        }
    };
    auto clear = [&](const uint32_t (&c)[E]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < E; ++j) *(lds_u16_t *)(uintptr_t)c[j] = (uint16_t)0;
    };
    const uint32_t yst = sbase + (uint32_t)(dr * kDnStageRow + PL * 2 * dp);
    auto store_y = [&](const Slot &r, int sb) __attribute__((always_inline)) {
        if constexpr (PL == 2) *(__attribute__((address_space(3))) uint32_t *)(uintptr_t)(yst + sb * SB) = r.y[0];
        else *(lds_u32x4_t *)(uintptr_t)(yst + sb * SB) = u32x4_t{r.y[0], r.y[1], r.y[2], r.y[3]};
    };

    f32x4_t acc[MT][NFT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int i = 0; i < NFT; ++i) acc[m][i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    // operand addresses: A rows 16 m + l16, labels 8q .. 8q + 7 of the step; B rows 16 ft + l16,
    // chunk q
    const uint32_t aoff = sbase + (uint32_t)(l16 * kDnStageRow + 16 * q);
    const uint32_t boff = lbase + (uint32_t)(wave * 1024 + l16 * 64 + ((q ^ ((l16 >> 2) & 3)) << 4));

#pragma unroll
    for (int i = 0; i < RSL; ++i) load_step(i, rg[i]);
    __syncthreads();                              // tiles zeroed
    scatter(rg[0], 0, ca[0]);                     // step 0
    store_y(rg[0], 0);
    __syncthreads();

    // step t = t0 + U of the unrolled period: its loads in slot U mod RSL, tile t mod 3, staged dY
    // and clear addresses t mod 2
    // Step t's operands are read into register set t mod 2 right after the barrier that completes
    // its tile, and its products are split in two halves: the first runs beside the scatter of
    // step t + 1, the second at the start of step t + 1, where it covers the latency of that step's
    // operand reads (the matrix cores would otherwise wait at every barrier).
    bf16x8_t oa[2][MT], ob[2][NFT];
#pragma unroll
    for (int m = 0; m < MT; ++m) oa[1][m] = bf16x8_t{};
#pragma unroll
    for (int i = 0; i < NFT; ++i) ob[1][i] = bf16x8_t{};   // "step -1": zero products
    constexpr int H1 = NFT / 2;                   // feature tiles of the first half
    static_assert(NFT % 2 == 0, "two halves");
    auto step = [&](int t, auto uc) __attribute__((always_inline)) {
        constexpr int U = decltype(uc)::value;
        constexpr int TBI = U % 3, PAR = U % 2;
        constexpr int SN = (U + 1) % RSL;         // slot of step t + 1
        const uint32_t ab = aoff + (uint32_t)(PAR * SB);
#pragma unroll
        for (int m = 0; m < MT; ++m) oa[PAR][m] = *(lds_bf16x8_t *)(uintptr_t)(ab + 16 * m * kDnStageRow);
#pragma unroll
        for (int i = 0; i < NFT; ++i) ob[PAR][i] = *(lds_bf16x8_t *)(uintptr_t)(boff + TBI * TB + NWV * 1024 * i);
        __builtin_amdgcn_sched_barrier(0);
        // second half of step t - 1
#pragma unroll
        for (int i = H1; i < NFT; ++i)
#pragma unroll
            for (int m = 0; m < MT; ++m)
                acc[m][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(oa[1 - PAR][m], ob[1 - PAR][i], acc[m][i], 0, 0, 0);
        // step t + 1: clear step t - 1's cells (tile (t + 2) mod 3, read before the last barrier),
        // write step t + 1's weights into tile (t + 1) mod 3 (cleared before the last barrier) and
        // stage its dY
        clear(ca[1 - PAR]);
        scatter(rg[SN], (TBI + 1) % 3, ca[1 - PAR]);
        store_y(rg[SN], 1 - PAR);
        // first half of step t
#pragma unroll
        for (int i = 0; i < H1; ++i)
#pragma unroll
            for (int m = 0; m < MT; ++m)
                acc[m][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(oa[PAR][m], ob[PAR][i], acc[m][i], 0, 0, 0);
        // the products of step t - 1 beside the scatter's address arithmetic, then those of step t
        // beside its LDS writes
        static_for<MT * (NFT - H1)>([&](auto) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        });
        static_for<MT * H1>([&](auto) __attribute__((always_inline)) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        });
        __builtin_amdgcn_sched_barrier(0);
        // the slot of step t is free (step t was written into its tile during the previous step):
        // it takes step t + RSL
        load_step(t + RSL, rg[U % RSL]);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
    };
    // whole periods only (steps past the segment's end add zeros): a conditional step would give the
    // accumulators a second path, and the compiler would then copy them between register files
    for (int t0 = 0; t0 < n; t0 += PER)
        static_for<PER>([&](auto uc) __attribute__((always_inline)) { step(t0 + decltype(uc)::value, uc); });
    // second half of the last step (odd: the step count is a multiple of PER)
#pragma unroll
    for (int i = H1; i < NFT; ++i)
#pragma unroll
        for (int m = 0; m < MT; ++m)
            acc[m][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(oa[1][m], ob[1][i], acc[m][i], 0, 0, 0);

    // partial dX^T of the segment: lane (l16, q) of tile ft holds feature 16 ft + l16, rows
    // 16 m + 4q .. + 3
#pragma unroll
    for (int i = 0; i < NFT; ++i) {
        const int f = 16 * (wave + NWV * i) + l16;
        if (f < F_s) {
#pragma unroll
            for (int m = 0; m < MT; ++m)
                *reinterpret_cast<float4 *>(pp + (size_t)f * Bp + 16 * m + 4 * q) =
                    make_float4(acc[m][i][0], acc[m][i][1], acc[m][i][2], acc[m][i][3]);
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Forward for small groups as a dense product over scattered weight tiles (bf16):
//   Y[rows, l] = bias[l] + sum over f of X[rows, f] W'[l, f]   (Section 3.2, the forward product;
//   W' as above, here stored label-major).
// The gathers of the small-group forward cost one LDS read per (label's group, slot, row); here a
// step of 32 labels costs one 2-byte write per (label, slot), independent of the rows.  A
// workgroup of 8 waves owns 32 batch rows and a segment of labels; wave (mt, nt, kh) keeps X for
// rows 16 mt .. 16 mt + 15 and the features of K half kh in its registers for the whole segment.
// Per step:
//   - the step's weights are scattered into a zeroed [32 labels][FR] bf16 tile and cleared after
//     use (FR = F_s rounded up to 128);
//   - wave (mt, nt, kh) forms D[labels 16 nt ..][rows 16 mt ..] over its K half with
//     v_mfma_f32_16x16x32_bf16: A = 16-byte reads of the tile's label rows, B = X from registers;
//   - in the next step the K-half-1 wave's partial sums reach its K-half-0 partner through LDS, which
//     adds them to its own (in fixed order) with the bias and puts the bf16 result into a staged
//     [32 rows][64 labels] block that leaves as 128-byte row runs every second step.
// Three tiles rotate (the step's, the next one being written, the previous one being cleared), with
// one barrier per step; at F_s = 768 they and the staging fill the 160 KB of LDS.
// ---------------------------------------------------------------------------------------------
// staged output: [32 rows][64 labels] bf16, 8-byte piece p of row r at piece position p ^ (r mod 16)
constexpr int kFdStage = 32 * 128;
constexpr int kFdRed = 4 * 1024;                 // one step's K-half-1 partial sums: 4 waves x 64 lanes x 16 B
__host__ __device__ constexpr int fd_lds(int fr) { return 3 * 64 * fr + 2 * kFdRed + 2 * kFdStage; }

// KCH: 32-feature K chunks per half (FR = 64 KCH).
template <int KCH, int F_IN, bool HAS_BIAS>
__global__ __launch_bounds__(512) void k_fwd_dn(const bf16_t *__restrict__ X, const int32_t *__restrict__ idx,
                                                const bf16_t *__restrict__ W, const float *__restrict__ bias,
                                                bf16_t *__restrict__ Y, int B, int F_s, int64_t L, int gshift, int nbt,
                                                int64_t lps, const int32_t *__restrict__ spos, int P) {
    constexpr int FR = 64 * KCH;                  // tile columns (features)
    constexpr int TB = 64 * FR;                   // tile bytes: [32 labels][FR] bf16
    constexpr int LPL = 16;                       // lanes per label of a step
    constexpr int E = F_IN / LPL;                 // slots per lane and step
    constexpr int NW = E / 2;                     // dwords of weights per lane and step
    constexpr int RSL = 4;                        // steps whose loads are in flight (ring slots)
    constexpr int PER = 12;                       // unrolled period: RSL, 3 tiles, 2 staged blocks
    static_assert(FR % 128 == 0, "a tile row is whole 16-chunk blocks");
    static_assert(E == 2 || E % 4 == 0, "support loads of 8 or 16 bytes");
    extern __shared__ __align__(16) char fd[];    // 3 tiles, [2] partial sums, [2] staged blocks
    const int w = blockIdx.x, xcd = w % kXcds, jj = w / kXcds;
    const int bt = jj % nbt;
    const int64_t seg = (int64_t)(jj / nbt) * kXcds + xcd;
    const int b0 = bt * 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const int64_t l_begin = seg * lps;
    const int64_t l_end = l_begin + lps < L ? l_begin + lps : L;
    if (l_begin >= l_end) return;                 // workgroup-uniform
    const int n = (int)(((l_end - l_begin + 31) / 32 + PER - 1) / PER * PER);   // steps, whole periods
    const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)fd;
    const uint32_t rbase = lbase + 3 * TB;        // partial sums
    const uint32_t sbase = rbase + 2 * kFdRed;    // staged output
    // the first clear writes here: staged block 1, which is first written in step 3
    const uint32_t dummy = sbase + kFdStage;
    for (int e = tid; e < 3 * TB / 16; e += 512) *(lds_u32x4_t *)(uintptr_t)(lbase + 16 * e) = u32x4_t{0u, 0u, 0u, 0u};

    // ---- X for this wave's rows and K half, in registers for the whole segment ----
    const int mt = wave & 1, nt = (wave >> 1) & 1, kh = wave >> 2;
    const int rows = B - b0 < 32 ? B - b0 : 32;
    bf16x8_t xa[KCH];
    {
        const Buf xb(X + (int64_t)b0 * F_s, (uint32_t)((int64_t)rows * F_s * 2));
        const int r = 16 * mt + l16;
#pragma unroll
        for (int c = 0; c < KCH; ++c) {
            const int f0 = 32 * (kh * KCH + c) + 8 * q;
            const uint32_t off = r < rows && f0 < F_s ? (uint32_t)(((int64_t)r * F_s + f0) * 2) : kOob;
            xa[c] = as_bf16x8(xb.ld16(off));
        }
    }

    // ---- scatter roles (as in backward-feature: 16 lanes per label, 4 labels of distinct 4-byte
    // pairs per wave) ----
    const int gl0 = tid / LPL;
    const int ls = 8 * (gl0 >> 3) + 2 * (gl0 & 3) + ((gl0 >> 2) & 1);
    const int o = tid % LPL;
    const uint32_t lrow = (uint32_t)(ls * FR * 2);
    const uint32_t lsw = (uint32_t)(ls & 15);
    const Buf wseg(W + l_begin * F_IN, (uint32_t)((l_end - l_begin) * F_IN * 2));
    const int64_t g_begin = l_begin >> gshift;
    const Buf iseg(idx + g_begin * F_IN, (uint32_t)(((l_end >> gshift) - g_begin) * F_IN * 4));
    struct Slot {
        uint32_t wv[NW];
        int32_t f[E];
    };
    Slot rg[RSL];
    auto load_step = [&](int st, Slot &r) __attribute__((always_inline)) {
        const int64_t lr = (int64_t)st * 32 + ls;
        const uint32_t wo = (uint32_t)(lr * F_IN * 2 + E * 2 * o);
        if constexpr (NW == 1) {
            r.wv[0] = wseg.ld4(wo);
        } else if constexpr (NW == 2) {
            const uint2 x = wseg.ld8(wo);
            r.wv[0] = x.x;
            r.wv[1] = x.y;
        } else {
#pragma unroll
            for (int i = 0; i < NW / 4; ++i) {
                const uint4 x = wseg.ld16(wo + 16 * i);
                r.wv[4 * i] = x.x;
                r.wv[4 * i + 1] = x.y;
                r.wv[4 * i + 2] = x.z;
                r.wv[4 * i + 3] = x.w;
            }
        }
        const int64_t gl = ((l_begin + lr) >> gshift) - g_begin;
        const uint32_t io = (uint32_t)(gl * F_IN * 4 + E * 4 * o);
        if constexpr (E == 2) {
            const uint2 x = iseg.ld8(io);
            r.f[0] = (int32_t)x.x;
            r.f[1] = (int32_t)x.y;
        } else {
#pragma unroll
            for (int i = 0; i < E / 4; ++i) {
                const uint4 x = iseg.ld16(io + 16 * i);
                r.f[4 * i] = (int32_t)x.x;
                r.f[4 * i + 1] = (int32_t)x.y;
                r.f[4 * i + 2] = (int32_t)x.z;
                r.f[4 * i + 3] = (int32_t)x.w;
            }
        }
    };
    // tile row ls: the 16-byte chunk k (features 8k .. 8k + 7) at chunk position k ^ (ls mod 16)
    uint32_t ca[2][E];
#pragma unroll
    for (int j = 0; j < E; ++j) ca[0][j] = ca[1][j] = dummy;
    auto scatter = [&](const Slot &r, int tb, uint32_t (&c)[E]) __attribute__((always_inline)) {
        const uint32_t base = lbase + (uint32_t)(tb * TB) + lrow;
#pragma unroll
        for (int j = 0; j < E; ++j) {
            const uint32_t f = (uint32_t)r.f[j];
            c[j] = base + ((((f >> 3) ^ lsw) << 4) | ((f & 7u) << 1));
            const uint32_t v = r.wv[j >> 1];
            *(lds_u16_t *)(uintptr_t)c[j] = (uint16_t)((j & 1) ? (v >> 16) : v);
        }
    };
    auto clear = [&](const uint32_t (&c)[E]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < E; ++j) *(lds_u16_t *)(uintptr_t)c[j] = (uint16_t)0;
    };
    // A operand: tile row 16 nt + l16, chunk 4 (kh KCH + c) + q at position chunk ^ l16
    const uint32_t arow = lbase + (uint32_t)((16 * nt + l16) * FR * 2);
    const uint32_t ql = (uint32_t)(q ^ l16);
    // K-half-1 partial sums: wave 4 + j's lane l at j 1024 + 16 l, read by its partner wave j
    const uint32_t rslot = rbase + (uint32_t)((wave & 3) * 1024 + lane * 16);
    f32x4_t dprev = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};   // a K-half-0 wave's partial sums of the last step
    // the partner pair's result of step st: rows 16 mt + l16, labels 16 nt + 4q .. + 3 of the step
    const int srow = 16 * mt + l16;
    auto combine = [&](int st, int par) __attribute__((always_inline)) {
        const f32x4_t p1 = *(__attribute__((address_space(3))) f32x4_t *)(uintptr_t)(rslot + par * kFdRed);
        f32x4_t v = dprev + p1;
        if constexpr (HAS_BIAS) {
            const int64_t lab = l_begin + (int64_t)st * 32 + 16 * nt + 4 * q;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += lab + e < l_end ? bias[lab + e] : 0.0f;
        }
        const int piece = (st & 1) * 8 + 4 * nt + q;
        const uint32_t sb = sbase + (uint32_t)(((st >> 1) & 1) * kFdStage + srow * 128 + ((piece ^ (srow & 15)) << 3));
        *(lds_u32x2_t *)(uintptr_t)sb = u32x2_t{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
    };
    // flush of steps 2k, 2k + 1: thread -> row tid / 16, labels 4 (tid mod 16) .. + 3 (8 bytes);
    // with the positives, the loss gradient of the rounded logits
    const int fr_ = tid >> 4, fp = tid & 15;
    PosCursor tgt;
    if (spos && fr_ < rows) tgt.init(spos + (int64_t)(b0 + fr_) * P, P, l_begin + 4 * fp);
    auto flush = [&](int k) __attribute__((always_inline)) {
        const int64_t lab = l_begin + (int64_t)k * 64 + 4 * fp;
        const int64_t nv = l_end - lab;
        if (fr_ < rows && nv > 0) {
            u32x2_t v = *(lds_u32x2_t *)(uintptr_t)(sbase + (uint32_t)((k & 1) * kFdStage + fr_ * 128 +
                                                                       ((fp ^ (fr_ & 15)) << 3)));
            if (spos) {   // kernel-uniform
                const uint32_t t = tgt.bits(lab, 4);
                v = u32x2_t{bce_pair(v[0], t), bce_pair(v[1], t >> 2)};
            }
            bf16_t *dst = Y + (int64_t)(b0 + fr_) * L + lab;
            if (nv >= 4) *reinterpret_cast<uint2 *>(dst) = make_uint2(v[0], v[1]);
            else *reinterpret_cast<uint32_t *>(dst) = v[0];   // L even: the row's last two labels
        }
    };

#pragma unroll
    for (int i = 0; i < RSL; ++i) load_step(i, rg[i]);
    __syncthreads();                              // tiles zeroed
    scatter(rg[0], 0, ca[0]);                     // step 0
    __syncthreads();

    // step t = t0 + U: tile t mod 3, partial sums t mod 2, ring slot t mod RSL, clear addresses t mod 2
    auto step = [&](int t, auto uc) __attribute__((always_inline)) {
        constexpr int U = decltype(uc)::value;
        constexpr int PAR = U % 2, TBI = U % 3;
        bf16x8_t ob[KCH];
#pragma unroll
        for (int c = 0; c < KCH; ++c)
            ob[c] = *(lds_bf16x8_t *)(uintptr_t)(arow + (uint32_t)(TBI * TB) +
                                                 ((((uint32_t)(4 * (kh * KCH + c))) ^ ql) << 4));
        __builtin_amdgcn_sched_barrier(0);
        // step t - 1's cells (tile (t + 2) mod 3, read before the last barrier) are cleared and step
        // t + 1 is written into tile (t + 1) mod 3 (cleared before the last barrier)
        clear(ca[1 - PAR]);
        scatter(rg[(U + 1) % RSL], (TBI + 1) % 3, ca[1 - PAR]);
        // two independent chains of products (even and odd chunks), so that one's latency is covered
        f32x4_t d[2] = {f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}, f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}};
#pragma unroll
        for (int c = 0; c < KCH; ++c) d[c & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ob[c], xa[c], d[c & 1], 0, 0, 0);
        if (kh == 1) {
            *(__attribute__((address_space(3))) f32x4_t *)(uintptr_t)(rslot + PAR * kFdRed) = d[0] + d[1];
        } else {
            if (t >= 1) combine(t - 1, 1 - PAR);
            dprev = d[0] + d[1];
        }
        if (PAR == 1 && t >= 3) flush((t - 3) >> 1);
        load_step(t + RSL, rg[U % RSL]);          // step t's slot is free (scattered in the last step)
        __syncthreads();
    };
    for (int t0 = 0; t0 < n; t0 += PER)
        static_for<PER>([&](auto uc) __attribute__((always_inline)) { step(t0 + decltype(uc)::value, uc); });
    if (kh == 0) combine(n - 1, (n - 1) & 1);
    __syncthreads();
    flush((n - 2) >> 1);
}

struct DnGeom {
    int nwv, mt, nbt, FR, nft;
    int64_t nseg, lps;
    size_t lds;
};

// Batches of more than 32 rows take 64-row workgroups of 4 waves (one per SIMD, so that the 64 x F_s
// accumulators fit the registers), smaller ones, and 128-slot supports (whose lanes carry twice the
// entries), 32-row workgroups of 8 waves.
static DnGeom dn_geom(const haste::TailArgs &a) {
    DnGeom g;
    g.nwv = a.B > 32 && a.F_in <= 64 ? 4 : 8;
    g.mt = g.nwv == 4 ? 4 : 2;
    g.nbt = (int)haste::cdiv(a.B, 16 * g.mt);
    const int per_wave = (int)haste::cdiv(haste::cdiv(a.F_s, 16), g.nwv);
    // the instantiated tile counts per wave (0: F_s too wide)
    static const int k4[] = {2, 4, 8, 12}, k8[] = {2, 4, 6};
    g.nft = 0;
    if (g.nwv == 4) {
        for (int c : k4)
            if (g.nft == 0 && per_wave <= c) g.nft = c;
    } else {
        for (int c : k8)
            if (g.nft == 0 && per_wave <= c) g.nft = c;
    }
    g.FR = 16 * g.nwv * g.nft;
    // one workgroup per CU (the tiles take most of the LDS): segments x batch tiles ~ 256
    int64_t nseg = haste::round_up(haste::cdiv(kXcds * kCusPerXcd, g.nbt), kXcds);
    const int64_t max_seg = haste::round_up(haste::cdiv(a.L, 64), kXcds);
    g.nseg = nseg < max_seg ? nseg : max_seg;
    g.lps = haste::round_up(haste::cdiv(a.L, g.nseg), 64);
    g.lds = (size_t)dn_lds(g.FR, g.mt);
    return g;
}

template <int NWV, int MT, int F_IN, int NFT>
static hipError_t launch_dn(const haste::TailArgs &a, const DnGeom &g, const int32_t *idx, const void *W,
                            const void *dY, float *part, hipStream_t s) {
    constexpr int PL = 16 * MT * 32 / (64 * NWV);
    auto kern = a.L % PL != 0 ? k_bwd_x_dn<NWV, MT, F_IN, NFT, true> : k_bwd_x_dn<NWV, MT, F_IN, NFT, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)g.lds);
    if (e != hipSuccess) return e;
    const int gshift = a.G == 1 ? 0 : a.G == 2 ? 1 : a.G == 4 ? 2 : 3;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(64 * NWV), g.lds, s, idx, (const bf16_t *)W,
                       (const bf16_t *)dY, part, (int)a.B, g.nbt * 16 * MT, (int)a.F_s, g.FR, a.L, gshift, g.nbt, g.lps);
    return hipGetLastError();
}

template <int F_IN>
static hipError_t dn_f(const haste::TailArgs &a, const DnGeom &g, const int32_t *idx, const void *W, const void *dY,
                       float *part, hipStream_t s) {
    if (g.nwv == 4) {
        switch (g.nft) {
            case 2: return launch_dn<4, 4, F_IN, 2>(a, g, idx, W, dY, part, s);
            case 4: return launch_dn<4, 4, F_IN, 4>(a, g, idx, W, dY, part, s);
            case 8: return launch_dn<4, 4, F_IN, 8>(a, g, idx, W, dY, part, s);
            case 12: return launch_dn<4, 4, F_IN, 12>(a, g, idx, W, dY, part, s);
        }
    } else {
        switch (g.nft) {
            case 2: return launch_dn<8, 2, F_IN, 2>(a, g, idx, W, dY, part, s);
            case 4: return launch_dn<8, 2, F_IN, 4>(a, g, idx, W, dY, part, s);
            case 6: return launch_dn<8, 2, F_IN, 6>(a, g, idx, W, dY, part, s);
        }
    }
    return hipErrorInvalidValue;
}


struct FdGeom {
    int nbt, kch;
    int64_t nseg, lps;
    size_t lds;
};

static FdGeom fd_geom(const haste::TailArgs &a) {
    FdGeom g;
    g.nbt = (int)haste::cdiv(a.B, 32);
    const int fr = (int)haste::round_up(a.F_s, 128);
    g.kch = fr / 64;
    int64_t nseg = haste::round_up(haste::cdiv(kXcds * kCusPerXcd, g.nbt), kXcds);
    const int64_t max_seg = haste::round_up(haste::cdiv(a.L, 64), kXcds);
    g.nseg = nseg < max_seg ? nseg : max_seg;
    g.lps = haste::round_up(haste::cdiv(a.L, g.nseg), 64);
    g.lds = (size_t)fd_lds(fr);
    return g;
}

template <int KCH, int F_IN>
static hipError_t launch_fd(const haste::TailArgs &a, const FdGeom &g, const void *X, const int32_t *idx, const void *W,
                            const float *bias, void *Y, hipStream_t s, const int32_t *spos, int P) {
    auto kern = bias ? k_fwd_dn<KCH, F_IN, true> : k_fwd_dn<KCH, F_IN, false>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)g.lds);
    if (e != hipSuccess) return e;
    const int gshift = a.G == 1 ? 0 : a.G == 2 ? 1 : a.G == 4 ? 2 : 3;
    hipLaunchKernelGGL(kern, dim3((unsigned)(g.nseg * g.nbt)), dim3(512), g.lds, s, (const bf16_t *)X, idx,
                       (const bf16_t *)W, bias, (bf16_t *)Y, (int)a.B, (int)a.F_s, a.L, gshift, g.nbt, g.lps, spos, P);
    return hipGetLastError();
}

template <int F_IN>
static hipError_t fd_f(const haste::TailArgs &a, const FdGeom &g, const void *X, const int32_t *idx, const void *W,
                       const float *bias, void *Y, hipStream_t s, const int32_t *spos, int P) {
    switch (g.kch) {
        case 2: return launch_fd<2, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 4: return launch_fd<4, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 6: return launch_fd<6, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 8: return launch_fd<8, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 10: return launch_fd<10, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 12: return launch_fd<12, F_IN>(a, g, X, idx, W, bias, Y, s, spos, P);
    }
    return hipErrorInvalidValue;
}


// ---------------------------------------------------------------------------------------------
// Backward-weight for groups of 1 or 2 labels as a dense matrix-core product (bf16):
//   dW[l, t] = sum over rows b of dY[b, l] X[b, idx[g(l), t]]   (Section 3.2, the backward-weight
//   product): the entries of D = dY^T X [labels][F_s] at each label's support.
// With one or two labels per group a gather kernel shares a gathered X column among at most two
// labels, and its cost is an LDS gather per (label, slot, row).  Here a workgroup of 8 waves (two
// per SIMD) owns a block of 64 labels at a time and forms D for all F_s features over the whole
// batch: wave w keeps D[64 labels][features 16 NFT w ..] in its matrix-core accumulators (96
// registers at NFT = 6).  Per K step of 32 rows, with v_mfma_f32_16x16x32_bf16 (M = labels,
// N = features, K = rows):
//   A = dY^T: the step's [32 rows][64 labels] block, staged in LDS and read transposed with
//       ds_read_b64_tr_b16 (lane (label l16, q) receives rows 8q .. 8q+7 of its label);
//   B = X^T from the block-major copy (16 bytes per lane: rows 8q .. 8q+7 of one feature; 1 KiB
//       of 16 whole features per wave instruction, L2-resident), the next step's loads issued one
//       per feature tile between the products.
// dY (from HBM) is loaded four steps ahead, after the step's X^T loads, so that waiting for X^T
// (the load counter completes in order) does not wait for it.  The product does F_s / F_in times
// the multiply-adds the layer needs (12x at 64 slots of 768), which the matrix cores absorb; X^T
// is read once per 64 labels, and that stream (384 KB per block at 256 rows, through each CU's L1)
// is what bounds the kernel.  After the batch, the D slices are staged in LDS as [feature][64
// labels] fp32 (rows of 272 bytes: the 16 lanes of one write land on distinct banks), a round of
// WPR waves at a time, and each thread picks out its dW cells (label, slot) whose feature lies in
// the round's range; the cells leave as contiguous rows.  Workgroups are persistent (one per CU):
// the next block's supports, first dY rows and first X^T tiles are loaded before the extraction.
// Rows past B meet zero X^T rows (and are loaded as zeros), and the K steps run in whole periods
// of four (a padded step reads past the X^T copy, i.e. zeros), so the accumulators have one path.
// ---------------------------------------------------------------------------------------------
constexpr int kWdLabels = 64;                     // labels per workgroup
constexpr int kWdYRow = 160;                      // staged dY row: 64 labels + 32 bytes of pad
constexpr int kWdDRow = 272;                      // staged D^T row: 64 labels fp32 + 16 bytes of pad
// waves per extraction round: their D^T slices (NWV waves x 16 NFT features) within 104 KB
__host__ __device__ constexpr int wd_wpr(int nwv, int nft) { return nwv * nft <= 24 ? nwv : nwv * nft <= 48 ? nwv / 2 : nwv / 4; }
__host__ __device__ constexpr int wd_stage(int nwv, int nft) {   // dY staging, then the D^T rounds
    return wd_wpr(nwv, nft) * 16 * nft * kWdDRow > 2 * 32 * kWdYRow ? wd_wpr(nwv, nft) * 16 * nft * kWdDRow : 2 * 32 * kWdYRow;
}
__host__ __device__ constexpr int wd_lds(int nwv, int nft, int f_in) { return wd_stage(nwv, nft) + kWdLabels * f_in * 4; }   // + supports

// NWV: waves (4: one per SIMD; 8: two).  NFT: 16-feature tiles per wave (NWV x 16 NFT >= F_s).
// TAILP: L is not a multiple of 8, so the last block's last 8-label piece of a row is read dword by
// dword (nothing past the row).
template <int NWV, int NFT, int F_IN, bool WITH_DB, bool TAILP>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * NWV, 64 * NWV), amdgpu_waves_per_eu(NWV / 4, NWV / 4)))
void k_bwd_w_dn(const bf16_t *__restrict__ Xb, const int32_t *__restrict__ idx, const bf16_t *__restrict__ dY,
                float *__restrict__ dW, float *__restrict__ dbias, int beta, int B, int Bp, int F_s, int64_t L,
                int gshift, int64_t nblk) {
    constexpr int T = 64 * NWV;                   // threads
    constexpr int NC = kWdLabels * F_IN / T;       // dW cells per thread
    constexpr int WPR = wd_wpr(NWV, NFT);
    constexpr int FPW = 16 * NFT;                  // features per wave
    extern __shared__ __align__(16) char wd[];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, q = lane >> 4;
    const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)wd;
    typedef __attribute__((address_space(3))) int lds_i32_t;
    typedef __attribute__((address_space(3))) float lds_f32_t;

    // this thread's dW cells of a block: label e / F_IN, slot e mod F_IN (e = tid + 256 i); their
    // features wait in LDS (behind the staging area) until the extraction
    const uint32_t fbase = lbase + (uint32_t)wd_stage(NWV, NFT);
    auto load_fe = [&](int64_t lab0, int nlab, int (&fe)[NC]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int e = tid + T * i, l = e / F_IN;
            fe[i] = l < nlab ? idx[((lab0 + l) >> gshift) * F_IN + e % F_IN] : -1;
        }
    };
    auto store_fe = [&](const int (&fe)[NC]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < NC; ++i) *(lds_i32_t *)(uintptr_t)(fbase + 4 * (tid + T * i)) = fe[i];
    };

    // dY of K step k of a block: thread -> row tid / 8, labels 8 (tid mod 8) .. + 7 (a block of no
    // labels reads nothing); with 8 waves, waves 4 .. 7 stage nothing
    const bool ystage = NWV == 4 || tid < 256;
    const int yr = (tid >> 3) & 31, yc = tid & 7;
    const uint32_t yst = lbase + (uint32_t)(yr * kWdYRow + 16 * yc);
    auto load_y = [&](int64_t lab0, int nlab, int k) __attribute__((always_inline)) -> u32x4_t {
        const int b0 = 32 * k;
        const int rows = B - b0 < 32 ? B - b0 : 32;   // none past the batch (and past the padded step)
        const Buf yb(dY + (int64_t)(rows > 0 ? b0 : 0) * L + lab0,
                     rows > 0 ? (uint32_t)(((int64_t)(rows - 1) * L + nlab) * 2) : 0u);
        const int nv = nlab - 8 * yc;                  // labels of this piece in the block
        const uint32_t o = ystage && yr < rows && nv > 0 ? (uint32_t)(((int64_t)yr * L + 8 * yc) * 2) : kOob;
        if constexpr (!TAILP) {
            const uint4 v = yb.ld16(o);
            return u32x4_t{v.x, v.y, v.z, v.w};
        } else {
            u32x4_t v;
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = yb.ld4(nv > 2 * j ? o + 4 * j : kOob);
            return v;
        }
    };
    // X^T of K step k: lane -> feature FPW wave + 16 nt + l16, rows 8q .. 8q + 7 (a lane offset plus
    // a scalar one per tile and step).  Features past F_s read the next block's rows or, past the
    // copy, zeros: finite values in columns of D that no support names.
    const Buf xb(Xb, (uint32_t)((int64_t)Bp * F_s * 2));
    const int xo = ((FPW * wave + l16) * 32 + 8 * q) * 2;
    auto load_x = [&](int k, bf16x8_t (&bo)[NFT]) __attribute__((always_inline)) {
        const int kb = k * F_s * 64;
#pragma unroll
        for (int nt = 0; nt < NFT; ++nt)
            bo[nt] = as_bf16x8(__builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xb.r, xo, kb + 1024 * nt, 0)));
    };
    // A operand source lanes (ds_read_b64_tr_b16): 16-lane group q names rows 8q + (l16 >> 2) (+ 4),
    // labels 16 m + 4 (l16 & 3) .. + 3
    const uint32_t asrc = lbase + (uint32_t)((8 * q + (l16 >> 2)) * kWdYRow + (l16 & 3) * 8);
    // (the LDS byte address becomes an LDS pointer directly: through a generic pointer, address 0
    // would turn into the LDS null value)
    auto read_a = [&](uint32_t slot, int m) __attribute__((always_inline)) -> bf16x8_t {
        const uint32_t p = asrc + slot + 32 * m;
        const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t *)(uintptr_t)p);
        const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t *)(uintptr_t)(p + 4 * kWdYRow));
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        return as_bf16x8(make_uint4(l2.x, l2.y, h2.x, h2.y));
    };

    f32x4_t acc[4][NFT];
    f32x4_t db;                                    // dbias of M tile `wave` (ones as B)
    const bf16x8_t ones = as_bf16x8(make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u));
    constexpr uint32_t SB = 32 * kWdYRow;          // one staged step
    // K steps in whole periods of four (the dY ring below; a padded step reads zeros)
    const int nk = Bp / 32;
    const int nkp = (nk + 3) & ~3;
    // X^T of steps k and k + 1: step s in bo[s mod XR], loaded XR - 1 steps ahead (a deeper ring
    // with one wave per SIMD ran out of registers and was three times slower)
    constexpr int XR = 2;
    bf16x8_t bo[XR][NFT];
    u32x4_t yv[4];         // dY of steps k + 1 .. k + 4, step s in yv[s mod 4]
    int fe[NC];

    // The workgroup runs blocks blockIdx.x, + gridDim.x, ... (one workgroup per CU).  A block's
    // first loads (supports, dY of steps 0 .. 4, X^T of step 0) are issued before the previous
    // block's extraction, so that their latency is hidden behind it.
    int64_t blk = blockIdx.x;
    int64_t lab0 = blk * kWdLabels;
    int nlab = L - lab0 < kWdLabels ? (int)(L - lab0) : kWdLabels;
    {
        load_fe(lab0, nlab, fe);
        const u32x4_t y0 = load_y(lab0, nlab, 0);
#pragma unroll
        for (int j = 1; j <= 4; ++j) yv[j & 3] = load_y(lab0, nlab, j);
#pragma unroll
        for (int j = 0; j < XR - 1; ++j) load_x(j, bo[j]);
        if (ystage) *(lds_u32x4_t *)(uintptr_t)yst = y0;
        store_fe(fe);
        __syncthreads();                           // step 0 and the supports staged
    }
    for (;;) {
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int nt = 0; nt < NFT; ++nt) acc[m][nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        db = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        // Step k (U = k mod 4): its dY is in staging slot k mod 2 and its X^T in bo[k mod XR].  It
        // stages step k + 1's dY (loaded four steps earlier) into the other slot, whose step k - 1
        // was read before the last barrier, and loads step k + 5's dY in its place; step k + 1's X^T
        // loads are issued one per feature tile between the products (issued together, the waves'
        // 48 loads queue at the texture unit and each wave waits there before its first product).
        auto step = [&](int k, auto uc) __attribute__((always_inline)) {
            constexpr int U = decltype(uc)::value;
            constexpr int PAR = U & 1, J = (U + 1) & 3;
            bf16x8_t a[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) a[m] = read_a(PAR * SB, m);
            bf16x8_t ad;
            if constexpr (WITH_DB) ad = read_a(PAR * SB, wave & 3);
            if (ystage) *(lds_u32x4_t *)(uintptr_t)(yst + (1 - PAR) * SB) = yv[J];
            yv[J] = load_y(lab0, nlab, k + 5);
            __builtin_amdgcn_sched_barrier(0);
            constexpr int XC = U % XR, XN = (U + XR - 1) % XR;   // this step's slot; the one step k - 1 freed
            const int kb = (k + XR - 1) * F_s * 64;
#pragma unroll
            for (int nt = 0; nt < NFT; ++nt) {
                bo[XN][nt] = as_bf16x8(__builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xb.r, xo, kb + 1024 * nt, 0)));
#pragma unroll
                for (int m = 0; m < 4; ++m) acc[m][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[m], bo[XC][nt], acc[m][nt], 0, 0, 0);
            }
            if constexpr (WITH_DB) db = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad, ones, db, 0, 0, 0);
            static_for<NFT>([&](auto) __attribute__((always_inline)) {
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one X^T load
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);   // four products
            });
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
        };
        for (int k0 = 0; k0 < nkp; k0 += 4)
            static_for<4>([&](auto uc) __attribute__((always_inline)) { step(k0 + decltype(uc)::value, uc); });

        // the next block's first loads (none past the last block: a block of no labels)
        const int64_t nb = blk + gridDim.x;
        const int64_t lab0n = nb < nblk ? nb * kWdLabels : lab0;
        const int nlabn = nb < nblk ? (L - lab0n < kWdLabels ? (int)(L - lab0n) : kWdLabels) : 0;
        // (128-slot supports: the next block's support ids are loaded after the extraction, whose
        // registers they would otherwise crowd)
        constexpr bool PRE_FE = F_IN <= 64;
        int fen[NC];
        if constexpr (PRE_FE) load_fe(lab0n, nlabn, fen);
        const u32x4_t y0 = load_y(lab0n, nlabn, 0);
#pragma unroll
        for (int j = 1; j <= 4; ++j) yv[j & 3] = load_y(lab0n, nlabn, j);
#pragma unroll
        for (int j = 0; j < XR - 1; ++j) load_x(j, bo[j]);

        // extraction: round r stages the slices of waves WPR r .. WPR r + WPR - 1 (features
        // FPW WPR r .. + FPW WPR - 1) as D^T [feature][label]; lane (l16, q) of tile (m, nt) holds
        // feature 16 nt + l16 of its wave, labels 16 m + 4q .. + 3
        constexpr int NR = NWV / WPR;
        float dv[NC];
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            fe[i] = *(lds_i32_t *)(uintptr_t)(fbase + 4 * (tid + T * i));
            dv[i] = 0.0f;
        }
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            if (r > 0) __syncthreads();            // the previous round's picks are done
            if (wave / WPR == r) {
                const uint32_t drow = lbase + (uint32_t)(((wave % WPR) * FPW + l16) * kWdDRow + 16 * q);
#pragma unroll
                for (int nt = 0; nt < NFT; ++nt)
#pragma unroll
                    for (int m = 0; m < 4; ++m)
                        *(lds_u32x4_t *)(uintptr_t)(drow + 16 * nt * kWdDRow + 64 * m) =
                            __builtin_bit_cast(u32x4_t, acc[m][nt]);
            }
            __syncthreads();
            const int lo = FPW * WPR * r;
#pragma unroll
            for (int i = 0; i < NC; ++i) {
                const int fr = fe[i] - lo;
                if (fr >= 0 && fr < FPW * WPR) {
                    const int l = (tid + T * i) / F_IN;
                    dv[i] = *(lds_f32_t *)(uintptr_t)(lbase + (uint32_t)(fr * kWdDRow + 4 * l));
                }
            }
        }
        float *wrow = dW + lab0 * F_IN;
#pragma unroll
        for (int i = 0; i < NC; ++i) {
            const int e = tid + T * i;
            if (e / F_IN < nlab) wrow[e] = beta ? wrow[e] + dv[i] : dv[i];
        }
        if constexpr (WITH_DB) {
            if (l16 == 0 && wave < 4) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int l = 16 * wave + 4 * q + i;
                    if (l < nlab) dbias[lab0 + l] = (beta ? dbias[lab0 + l] : 0.0f) + db[i];
                }
            }
        }
        if (nb >= nblk) break;                     // workgroup-uniform
        if constexpr (!PRE_FE) load_fe(lab0n, nlabn, fen);
        __syncthreads();                           // the picks are done: the LDS takes the next block
        if (ystage) *(lds_u32x4_t *)(uintptr_t)yst = y0;
        store_fe(fen);
        __syncthreads();
        blk = nb;
        lab0 = lab0n;
        nlab = nlabn;
    }
}

static int wd_nft(int F_s) { return F_s <= 256 ? 4 : F_s <= 512 ? 8 : F_s <= 768 ? 12 : 0; }

template <int NWV, int NFT, int F_IN>
static hipError_t launch_wd(const haste::TailArgs &a, const void *Xb, const int32_t *idx, const void *dY, float *dW,
                            float *dbias, int beta, int Bp, hipStream_t s) {
    const bool tailp = a.L % 8 != 0;
    auto go = [&](auto kern) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, wd_lds(NWV, NFT, F_IN));
        if (e != hipSuccess) return e;
        const int gshift = a.G == 1 ? 0 : 1;
        const int64_t nblk = haste::cdiv(a.L, kWdLabels);
        const int64_t grid = nblk < kXcds * kCusPerXcd ? nblk : kXcds * kCusPerXcd;   // one workgroup per CU
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * NWV), wd_lds(NWV, NFT, F_IN), s, (const bf16_t *)Xb, idx,
                           (const bf16_t *)dY, dW, dbias, beta, (int)a.B, Bp, (int)a.F_s, a.L, gshift, nblk);
        return hipGetLastError();
    };
    if (dbias) return tailp ? go(k_bwd_w_dn<NWV, NFT, F_IN, true, true>) : go(k_bwd_w_dn<NWV, NFT, F_IN, true, false>);
    return tailp ? go(k_bwd_w_dn<NWV, NFT, F_IN, false, true>) : go(k_bwd_w_dn<NWV, NFT, F_IN, false, false>);
}

template <int F_IN>
static hipError_t wd_f(const haste::TailArgs &a, const void *Xb, const int32_t *idx, const void *dY, float *dW,
                       float *dbias, int beta, int Bp, hipStream_t s) {
    switch (wd_nft((int)a.F_s)) {
        case 4: return launch_wd<8, 2, F_IN>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
        case 8: return launch_wd<8, 4, F_IN>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
        case 12: return launch_wd<8, 6, F_IN>(a, Xb, idx, dY, dW, dbias, beta, Bp, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

namespace haste {

// bf16, G in {1, 2, 4, 8}, F_in in {32, 64, 128}; F_s up to 768 (three [768][32] tiles fill the
// LDS); dY rows dword-aligned (L even) and a workgroup's rows within the 31-bit range of a buffer offset;
// a segment's weight and support offsets within that range too.
bool bwd_x_dn_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2 || a.G == 4 || a.G == 8)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || a.F_in == 128)) return false;
    if (a.F_s <= 0 || a.L % 2 != 0 || a.L * 64 * 2 >= ((int64_t)1 << 31)) return false;
    const DnGeom g = dn_geom(a);
    return g.nft != 0 && g.lds <= 160 * 1024 && (g.lps + 1024) * a.F_in * 4 < ((int64_t)1 << 31);
}

size_t bwd_x_dn_ws(const TailArgs &a) {
    const DnGeom g = dn_geom(a);
    return (size_t)round_up(g.nseg * a.F_s * (g.nbt * 16 * g.mt) * 4, 256);
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
    return reduce_fmajor(part, (int)g.nseg, g.nbt * 16 * g.mt, a.B, a.F_s, dX, beta, s);
}

// forward: bf16, G in {1, 2} (larger groups share their gathers, which the small-group kernel then
// does more cheaply), F_in in {32, 64, 128}, F_s a multiple of 8 up to 768 (X rows read 16 bytes at
// a time; two [32][768] tiles beside the staging), L even (the output leaves in label pairs).
bool fwd_dn_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || a.F_in == 128)) return false;
    if (a.F_s <= 0 || a.F_s % 8 != 0 || a.F_s > 768 || a.L % 2 != 0) return false;
    const FdGeom g = fd_geom(a);
    return g.lds <= 160 * 1024 && (g.lps + 1024) * a.F_in * 4 < ((int64_t)1 << 31);
}

hipError_t fwd_dn(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias, void *Y,
                  hipStream_t s, const int32_t *spos, int P) {
    const FdGeom g = fd_geom(a);
    switch (a.F_in) {
        case 32: return fd_f<32>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 64: return fd_f<64>(a, g, X, idx, W, bias, Y, s, spos, P);
        case 128: return fd_f<128>(a, g, X, idx, W, bias, Y, s, spos, P);
    }
    return hipErrorInvalidValue;
}

// backward-weight: bf16, G in {1, 2}, F_in in {32, 64, 128}, F_s a multiple of 8 up to 768 (the
// eight waves' accumulators); dY rows dword-aligned (L even) and 32 rows of them within the 31-bit
// range of a buffer offset, and the whole X^T copy (read past by a padded step) within that range
// too.  The X^T copy of the workspace is the other backward-weight kernels'.
bool bwd_w_dn_supported(const TailArgs &a) {
    if (a.dtype != HASTE_DTYPE_BF16 || !(a.G == 1 || a.G == 2)) return false;
    if (!(a.F_in == 32 || a.F_in == 64 || a.F_in == 128)) return false;
    return a.F_s > 0 && a.F_s % 8 == 0 && a.F_s <= 768 && a.L % 2 == 0 && (a.L * 32 + 1024) * 2 < ((int64_t)1 << 31) &&
           (round_up(a.B, 128) + 128) * a.F_s * 2 < ((int64_t)1 << 31);
}

hipError_t bwd_w_dn(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW, float *dbias,
                    int beta, void *ws, hipStream_t s) {
    const int Bp = (int)round_up(a.B, 32);
    hipError_t e = transpose_x(a, X, ws, s);
    if (e != hipSuccess) return e;
    switch (a.F_in) {
        case 32: return wd_f<32>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
        case 64: return wd_f<64>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
        case 128: return wd_f<128>(a, ws, idx, dY, dW, dbias, beta, Bp, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace haste
