// Dense head over the frequent labels (paper Section 3.3, a^H = W_head h_head) and its backward.
//
// All three products are plain GEMMs C[M,N] = A[M,K] B[K,N] whose operands arrive in different
// layouts:
//   forward   Y_h  = X  W_head^T    A = X      (K contiguous), B = W_head^T (K contiguous)
//   dW_head   dW_h = dY_h^T X       A = dY_h^T (M contiguous), B = X        (N contiguous)
//   dX        dX  += dY_h W_head    A = dY_h   (K contiguous), B = W_head   (N contiguous), K = H
// The bf16 kernel stages 128x32 tiles of both operands in LDS with K contiguous (operands that
// are contiguous along M/N are transposed while being written to LDS) and runs
// v_mfma_f32_32x32x16_bf16 on a 2x2 grid of waves, each owning a 64x64 block.  dX contracts over
// the H head labels, so it is split over K and the partials are reduced in a fixed order.
#include <initializer_list>

#include "common.hpp"

namespace {

// EPI_BF16_BCE: the loss gradient sigmoid(logit) - T of the bias-added logits, in bf16 (256 kernel)
enum { EPI_BF16_BIAS = 0, EPI_F32 = 1, EPI_F32_PART = 2, EPI_BF16_BCE = 3 };

constexpr int TM = 128, TN = 128, TK = 32;
constexpr int LS = TK + 8;  // LDS row stride (bf16): 80 bytes keeps 16-byte rows aligned

// 8 consecutive elements along the operand's contiguous dimension, zero outside [0, lim)
__device__ __forceinline__ uint4 load8(const bf16_t *__restrict__ p, int64_t pos, int64_t lim) {
    if (pos + 8 <= lim && ((reinterpret_cast<uintptr_t>(p) & 15) == 0)) return *reinterpret_cast<const uint4 *>(p);
    bf16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = (pos + i < lim) ? p[i] : (bf16_t)0;
    return make_uint4(pack2(e[0], e[1]), pack2(e[2], e[3]), pack2(e[4], e[5]), pack2(e[6], e[7]));
}

// Stage a 128 x 32 operand tile into LDS as tile[r][k] (k contiguous).  Element (r, k) of the
// operand lives at base + r*sr + k*sk; exactly one of sr, sk is 1 (KC: k contiguous).
template <bool KC>
__device__ __forceinline__ void stage(bf16_t *tile, const bf16_t *__restrict__ base, int64_t sr, int64_t sk,
                                      int64_t r0, int64_t rlim, int64_t k0, int64_t klim) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int c = threadIdx.x + 256 * q;
        if (KC) {
            const int r = c >> 2, kc = (c & 3) * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (r0 + r < rlim) v = load8(base + (r0 + r) * sr + (k0 + kc), k0 + kc, klim);
            *reinterpret_cast<uint4 *>(tile + r * LS + kc) = v;
        } else {
            const int k = c >> 4, rc = (c & 15) * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (k0 + k < klim) v = load8(base + (k0 + k) * sk + (r0 + rc), r0 + rc, rlim);
            const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                tile[(rc + 2 * h) * LS + k] = (bf16_t)(u[h] & 0xffffu);
                tile[(rc + 2 * h + 1) * LS + k] = (bf16_t)(u[h] >> 16);
            }
        }
    }
}

template <bool AK, bool BK, int EPI>
__global__ __launch_bounds__(256) void k_gemm_bf16(const bf16_t *__restrict__ A, int64_t sam, int64_t sak,
                                                   const bf16_t *__restrict__ Bm, int64_t sbk, int64_t sbn,
                                                   void *__restrict__ C, int64_t ldc, const float *__restrict__ bias,
                                                   int64_t M, int64_t N, int64_t K, int64_t kchunk) {
    __shared__ __align__(16) bf16_t As[TM * LS];
    __shared__ __align__(16) bf16_t Bs[TN * LS];
    const int64_t n0 = (int64_t)blockIdx.x * TN, m0 = (int64_t)blockIdx.y * TM;
    const int64_t kb = (int64_t)blockIdx.z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int ln = lane & 31, hh = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{0};

    for (int64_t k0 = kb; k0 < ke; k0 += TK) {
        // A(m, k) at A + m*sam + k*sak ; B(k, n) at Bm + k*sbk + n*sbn
        stage<AK>(As, A, sam, sak, m0, M, k0, ke);
        stage<BK>(Bs, Bm, sbn, sbk, n0, N, k0, ke);
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < TK / 16; ++ks) {
            uint4 av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *reinterpret_cast<const uint4 *>(As + (wm * 64 + i * 32 + ln) * LS + ks * 16 + 8 * hh);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bv[j] = *reinterpret_cast<const uint4 *>(Bs + (wn * 64 + j * 32 + ln) * LS + ks * 16 + 8 * hh);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x16(as_bf16x8(av[i]), as_bf16x8(bv[j]), acc[i][j]);
        }
        __syncthreads();
    }
    // D[m = 8r + 4hh + q][n = ln] per 32x32 block
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 64 + j * 32 + ln;
            if (n >= N) continue;
            const float bv = (EPI == EPI_BF16_BIAS && bias) ? bias[n] : 0.0f;
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t m = m0 + wm * 64 + i * 32 + 8 * r + 4 * hh + q;
                    if (m >= M) continue;
                    const float v = acc[i][j][4 * r + q];
                    if (EPI == EPI_BF16_BIAS) {
                        reinterpret_cast<bf16_t *>(C)[m * ldc + n] = f32_to_bf16(v + bv);
                    } else if (EPI == EPI_F32) {
                        reinterpret_cast<float *>(C)[m * ldc + n] = v;
                    } else {
                        reinterpret_cast<float *>(C)[(int64_t)blockIdx.z * M * N + m * N + n] = v;
                    }
                }
        }
}

// ---------------------------------------------------------------------------------------------
// bf16 GEMM, double buffered.  128x128 output tile, K in steps of 64, 4 waves in a 2x2 grid each
// owning a 64x64 block (v_mfma_f32_32x32x16_bf16).  Each operand tile is staged in LDS in its
// global layout, loaded with coalesced 16-byte loads:
//   K contiguous      -> LDS [row][k], fragments read 16 bytes (8 k) per lane;
//   M/N contiguous    -> LDS [k][row], fragments read with ds_read_b64_tr_b16, which returns to
//                        lane i of a 16-lane group 4 consecutive k of row i when source lane 4a + b
//                        addresses k0 + a, rows 4b .. 4b+3 (two reads give the 8 k of a fragment).
// One barrier per K step: the next step's tiles are loaded into registers while the current
// step computes, then written to the other LDS buffer.
// ---------------------------------------------------------------------------------------------
constexpr int G2K = 64;                 // K step
constexpr int G2KC = G2K + 8;           // [row][k] row stride (bf16): 144 bytes
constexpr int G2RC = TM + 16;           // [k][row] row stride (bf16): 288 bytes
constexpr int G2TILE = (TM * G2KC > G2K * G2RC ? TM * G2KC : G2K * G2RC);  // bf16 per operand tile

// One operand: rows r0 .. r0+127 (M or N) by k0 .. k0+63, element (r, k) at base + r*sr + k*sk,
// with sk == 1 (KC) or sr == 1.  The whole matrix spans `bytes` (buffer bound: zero outside).
template <bool KC>
struct G2Operand {
    Buf buf;
    int64_t sr, sk;
    uint4 v[4];  // this thread's 4 x 16 bytes of the next tile
    __device__ __forceinline__ void load(int64_t r0, int64_t rlim, int64_t k0, int64_t klim) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = threadIdx.x + 256 * q;
            int64_t r, k;
            if (KC) { r = r0 + (c >> 3); k = k0 + (c & 7) * 8; }
            else    { k = k0 + (c >> 4); r = r0 + (c & 15) * 8; }
            // rows/k past the limits read as zero (limits are multiples of 8 along the contiguous dim)
            const bool ok = r < rlim && k < klim;
            const int64_t off = (r * sr + k * sk) * 2;
            v[q] = buf.ld16(ok ? (uint32_t)off : kOob);
        }
    }
    __device__ __forceinline__ void store(bf16_t *tile) const {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int c = threadIdx.x + 256 * q;
            if (KC) *reinterpret_cast<uint4 *>(tile + (c >> 3) * G2KC + (c & 7) * 8) = v[q];
            else    *reinterpret_cast<uint4 *>(tile + (c >> 4) * G2RC + (c & 15) * 8) = v[q];
        }
    }
    // MFMA operand fragment: rows rb .. rb+31 (lane ln), k = ks*16 + 8hh .. +7
    __device__ __forceinline__ uint4 frag(const bf16_t *tile, int rb, int ks, int lane) const {
        const int ln = lane & 31, hh = lane >> 5;
        if (KC) return *reinterpret_cast<const uint4 *>(tile + (rb + ln) * G2KC + ks * 16 + 8 * hh);
        const int g = lane >> 4, i = lane & 15;               // 16-lane group, lane in group
        const int rr = rb + 16 * (g & 1) + 4 * (i & 3);        // rows of this source lane
        const int kk = ks * 16 + 8 * (g >> 1) + (i >> 2);      // k row of this source lane
        const uint2 lo = lds_read_tr(tile + kk * G2RC + rr);
        const uint2 hi = lds_read_tr(tile + (kk + 4) * G2RC + rr);
        return make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
};

template <bool AK, bool BK, int EPI>
__global__ __launch_bounds__(256, 2) void k_gemm2(const bf16_t *__restrict__ A, int64_t sam, int64_t sak,
                                                  uint32_t a_bytes, const bf16_t *__restrict__ Bm, int64_t sbk,
                                                  int64_t sbn, uint32_t b_bytes, void *__restrict__ C, int64_t ldc,
                                                  const float *__restrict__ bias, int64_t M, int64_t N, int64_t K,
                                                  int64_t kchunk) {
    extern __shared__ __align__(16) bf16_t g2s[];   // [2 stages][A tile, B tile]
    const int64_t n0 = (int64_t)blockIdx.x * TN, m0 = (int64_t)blockIdx.y * TM;
    const int64_t kb = (int64_t)blockIdx.z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ln = lane & 31, hh = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    G2Operand<AK> oa{Buf(A, a_bytes), sam, sak, {}};
    G2Operand<BK> ob{Buf(Bm, b_bytes), sbn, sbk, {}};
    auto tileA = [&](int st) { return g2s + st * 2 * G2TILE; };
    auto tileB = [&](int st) { return g2s + st * 2 * G2TILE + G2TILE; };

    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{0};

    oa.load(m0, M, kb, ke);
    ob.load(n0, N, kb, ke);
    oa.store(tileA(0));
    ob.store(tileB(0));
    __syncthreads();
    int st = 0;
    for (int64_t k0 = kb; k0 < ke; k0 += G2K) {
        // next step's tiles (past the end: out of range, zero, never used)
        oa.load(m0, M, k0 + G2K, ke);
        ob.load(n0, N, k0 + G2K, ke);
        const bf16_t *ta = tileA(st), *tb = tileB(st);
#pragma unroll
        for (int ks = 0; ks < G2K / 16; ++ks) {
            uint4 av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) av[i] = oa.frag(ta, wm * 64 + i * 32, ks, lane);
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = ob.frag(tb, wn * 64 + j * 32, ks, lane);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32x32x16(as_bf16x8(av[i]), as_bf16x8(bv[j]), acc[i][j]);
        }
        st ^= 1;
        oa.store(tileA(st));
        ob.store(tileB(st));
        __syncthreads();
    }
    // D[m = 8r + 4hh + q][n = ln] per 32x32 block
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t n = n0 + wn * 64 + j * 32 + ln;
            if (n >= N) continue;
            const float bv = (EPI == EPI_BF16_BIAS && bias) ? bias[n] : 0.0f;
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int64_t m = m0 + wm * 64 + i * 32 + 8 * r + 4 * hh + q;
                    if (m >= M) continue;
                    const float v = acc[i][j][4 * r + q];
                    if (EPI == EPI_BF16_BIAS) {
                        reinterpret_cast<bf16_t *>(C)[m * ldc + n] = f32_to_bf16(v + bv);
                    } else if (EPI == EPI_F32) {
                        reinterpret_cast<float *>(C)[m * ldc + n] = v;
                    } else {
                        reinterpret_cast<float *>(C)[(int64_t)blockIdx.z * M * N + m * N + n] = v;
                    }
                }
        }
}

constexpr size_t kG2Lds = (size_t)4 * G2TILE * 2;   // two stages of two operand tiles

// ---------------------------------------------------------------------------------------------
// bf16 GEMM for large tiles: 256 x BN output tile (BN = 256 or 128), 4 waves in a 2x2 grid each
// owning a 128 x BN/2 block (4 x BN/64 v_mfma_f32_32x32x16_bf16 accumulators).  K advances in
// steps of 32 through a ring of LDS stages filled by direct global-to-LDS loads
// (buffer_load_dwordx4 ... lds: 64 lanes x 16 bytes land contiguously at the address in M0), so
// the next steps are in flight while one is multiplied, without staging registers: 4 stages and
// one workgroup per CU at BN = 256; 3 stages and two workgroups per CU at BN = 128 (the head's
// products use 128), so that one workgroup's epilogue overlaps the other's products.  The loads are
// issued from inline assembly and waited for explicitly (s_waitcnt vmcnt): issued through the
// compiler's builtin, every LDS read would first wait for all of them.
// Stage layouts carry an XOR swizzle of their 16-byte chunks instead of padding, so that a load
// instruction still fills 1 KB of contiguous LDS:
//   K-contiguous operand  [256 rows][32 k]:  chunk c of row r sits at c ^ ((r >> 1) & 3);
//   M/N-contiguous        [32 k][256 rows]:  chunk c of k-row k sits at c ^ 2 (k & 3).
// Both keep the fragment reads (16-byte row reads, and ds_read_b64_tr_b16 over 4 k-rows) free of
// bank conflicts.  The products are formed as D^T = B^T A^T (the B tile is the MFMA A operand),
// so a result lane holds 4 consecutive output columns of one row: 8-byte (bf16) or 16-byte
// (fp32) stores.  Tiles that share an operand tile are placed on one XCD back to back.
// ---------------------------------------------------------------------------------------------
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int G4T = 256;                  // output tile rows (M)
constexpr int kHeadBN = 128;              // output tile columns (N) of the head's products
constexpr int G4K = 32;                   // K step

// the tile's column count BN (256 or 128) fixes the rest: LDS stages (one workgroup per CU at 256,
// two at 128), bytes of the two operands' stage tiles, and the LDS the kernel takes
__host__ __device__ constexpr int g4_stages(int bn) { return bn == 256 ? 4 : 3; }
__host__ __device__ constexpr int g4_stage_bytes(int bn) { return (G4T + bn) * G4K * 2; }
__host__ __device__ constexpr size_t g4_lds(int bn) { return (size_t)g4_stages(bn) * g4_stage_bytes(bn); }

// one direct global-to-LDS load: this lane's 16 bytes at byte offset voff of the buffer land at
// LDS address lds + 16 * lane
__device__ __forceinline__ void lds_dma16(const Buf &b, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(lds), "v"(voff), "s"(b.r) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// One operand tile of R rows (R = 256 or 128) and 32 k per stage, R / 16 load instructions of
// 1 KB, R / 64 per wave: wave w issues instructions i = (R / 64) w + t.  K-contiguous: rows 16i ..
// 16i+15 (4 lanes per 64-byte row); M/N-contiguous: 512 / R k-rows of 2R bytes per instruction.
template <bool KC, int R>
struct G4Operand {
    static constexpr int NI = R / 64;    // load instructions per wave and stage
    static constexpr int LPK = R / 8;    // lanes per k-row (M/N-contiguous)
    Buf buf;
    int64_t ld;         // elements between consecutive rows (KC) or k-rows (M/N contiguous)
    int64_t r0, rlim;   // tile rows and the operand's row count (M or N)
    int64_t klim;       // end of this workgroup's K range
    __device__ __forceinline__ void issue(int64_t k0, uint32_t lds_stage, int wave, int lane) const {
#pragma unroll
        for (int t = 0; t < NI; ++t) issue1(k0, lds_stage, wave, lane, t);
    }
    __device__ __forceinline__ void issue1(int64_t k0, uint32_t lds_stage, int wave, int lane, int t) const {
        const int i = NI * wave + t;
        uint32_t off;
        if (KC) {
            const int row = 16 * i + (lane >> 2), c = (lane & 3) ^ ((row >> 1) & 3);
            const int64_t k = k0 + 8 * c;
            const bool ok = r0 + row < rlim && k < klim;   // klim is a multiple of 8
            off = ok ? (uint32_t)(((r0 + row) * ld + k) * 2) : kOob;
        } else {
            const int kr = (512 / R) * i + lane / LPK, c = (lane % LPK) ^ ((kr & 3) << 1);
            const int64_t r = r0 + 8 * c;
            const bool ok = k0 + kr < klim && r < rlim;    // rlim is a multiple of 8
            off = ok ? (uint32_t)(((k0 + kr) * ld + r) * 2) : kOob;
        }
        lds_dma16(buf, off, __builtin_amdgcn_readfirstlane(lds_stage + i * 1024));
    }
    // MFMA operand fragment: rows rb .. rb+31 (lane ln), k = ks*16 + 8hh .. +7 of the stage
    __device__ __forceinline__ uint4 frag(const char *stage, int rb, int ks, int lane) const {
        const int ln = lane & 31, hh = lane >> 5;
        if (KC) {
            const int row = rb + ln, c = (2 * ks + hh) ^ ((row >> 1) & 3);
            return *reinterpret_cast<const uint4 *>(stage + row * 64 + c * 16);
        }
        const int g = lane >> 4, i = lane & 15;                 // 16-lane group, lane in group
        const int rr = rb + 16 * (g & 1) + 4 * (i & 3);          // rows of this source lane
        const int kk = ks * 16 + 8 * (g >> 1) + (i >> 2);        // k-row of this source lane
        const char *p = stage + kk * (2 * R) + (((rr >> 3) ^ ((kk & 3) << 1)) * 16) + (rr & 7) * 2;
        const uint2 lo = lds_read_tr(p);
        const uint2 hi = lds_read_tr(p + 4 * (2 * R));           // k-row kk + 4: same swizzle
        return make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
};

template <int BN, bool AK, bool BK, int EPI>
__global__ __launch_bounds__(256, BN <= 128 ? 2 : 1) void k_gemm4(
    const bf16_t *__restrict__ A, int64_t sa, uint32_t a_bytes, const bf16_t *__restrict__ Bm, int64_t sb,
    uint32_t b_bytes, void *__restrict__ C, int64_t ldc, const float *__restrict__ bias, int64_t M, int64_t N,
    int64_t K, int64_t kchunk, int MT, int NT, int Z, const int32_t *__restrict__ pos, int P) {
    constexpr int S = g4_stages(BN);
    constexpr int NB = BN / 64;                  // 32-column blocks per wave
    constexpr int LPW = 4 + NB;                  // loads per wave and stage (A: 4, B: NB)
    constexpr int SB = g4_stage_bytes(BN);
    extern __shared__ __align__(16) char g4s[];   // [stage][A tile, B tile]
    // tile order: the workgroups that share an operand tile run on one XCD back to back
    const int w = blockIdx.x, xcd = w % kXcds, local = w / kXcds;
    int mt, nt, z = 0;
    if (Z > 1) {
        const int per = MT * NT, r = local % per;
        z = (local / per) * kXcds + xcd;
        mt = r / NT;
        nt = r % NT;
        if (z >= Z) return;
    } else if (MT <= NT) {
        nt = (local / MT) * kXcds + xcd;
        mt = local % MT;
        if (nt >= NT) return;
    } else {
        mt = (local / NT) * kXcds + xcd;
        nt = local % NT;
        if (mt >= MT) return;
    }
    const int64_t m0 = (int64_t)mt * G4T, n0 = (int64_t)nt * BN;
    const int64_t kb = (int64_t)z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int ln = lane & 31, hh = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    const G4Operand<AK, G4T> oa{Buf(A, a_bytes), sa, m0, M, ke};
    const G4Operand<BK, BN> ob{Buf(Bm, b_bytes), sb, n0, N, ke};
    const uint32_t lds0 = (uint32_t)reinterpret_cast<uintptr_t>(g4s);
    auto stA = [&](int st) { return lds0 + (uint32_t)(st * SB); };
    auto stB = [&](int st) { return lds0 + (uint32_t)(st * SB + G4T * G4K * 2); };

    f32x16_t acc[NB][4];   // [n block j][m block i]: D^T[n][m]
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[j][i] = f32x16_t{0};

    const int nsteps = (int)((ke - kb + G4K - 1) / G4K);
    auto frags = [&](int st, int ks, uint4 (&av)[4], uint4 (&bv)[NB]) {
        const char *ta = g4s + st * SB, *tb = ta + G4T * G4K * 2;
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = oa.frag(ta, wm * 128 + i * 32, ks, lane);
#pragma unroll
        for (int jn = 0; jn < NB; ++jn) bv[jn] = ob.frag(tb, wn * (BN / 2) + jn * 32, ks, lane);
    };
    auto products = [&](const uint4 (&av)[4], const uint4 (&bv)[NB]) {
#pragma unroll
        for (int jn = 0; jn < NB; ++jn)
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[jn][i] = mfma32x32x16(as_bf16x8(bv[jn]), as_bf16x8(av[i]), acc[jn][i]);
    };
    // Software pipeline over K steps of two 16-deep halves (h0, h1).  Iteration j: read h1 of step
    // j while h0's products run; wait for step j + 1 and barrier (stage j % S is then fully read
    // into registers by every wave); then h1's products, with the loads that refill stage j % S
    // with step j + S and the reads of h0 of step j + 1 spread between them.  Issued as one burst
    // after the barrier, the four waves' loads queue at the texture unit and hold up the products
    // behind them; spread out, they overlap.  Steps past the end are loaded out of range into
    // stages that are never read.
#pragma unroll
    for (int s = 0; s < S; ++s) {
        oa.issue(kb + (int64_t)s * G4K, stA(s), wave, lane);
        ob.issue(kb + (int64_t)s * G4K, stB(s), wave, lane);
    }
    uint4 a0[4], b0[NB], a1[4], b1[NB];
    wait_vmcnt<LPW * (S - 1)>();   // this wave's loads of step 0 have landed
    __syncthreads();               // everyone's have
    frags(0, 0, a0, b0);
    constexpr int NP = 4 * NB;                   // products of a half step
    constexpr int NA = 8 + 2 * NB;               // loads and fragment reads to spread over them
    for (int j = 0; j < nsteps; ++j) {
        const int st = j % S;
        frags(st, 1, a1, b1);
        __builtin_amdgcn_sched_barrier(0);   // the reads go ahead of the products they overlap
        products(a0, b0);
        __builtin_amdgcn_sched_barrier(0);
        wait_vmcnt<LPW * (S - 2)>();   // this wave's loads of step j + 1 have landed
        __syncthreads();               // everyone's have; stage j % S is read out
        const char *ta = g4s + ((j + 1) % S) * SB, *tb = ta + G4T * G4K * 2;
        const int64_t kn = kb + (int64_t)(j + S) * G4K;
#pragma unroll
        for (int s = 0; s < NP; ++s) {
            const int jn = s / 4, i = s % 4;
            acc[jn][i] = mfma32x32x16(as_bf16x8(b1[jn]), as_bf16x8(a1[i]), acc[jn][i]);
#pragma unroll
            for (int a = s * NA / NP; a < (s + 1) * NA / NP; ++a) {
                if (a < 4) oa.issue1(kn, stA(st), wave, lane, a);
                else if (a < 4 + NB) ob.issue1(kn, stB(st), wave, lane, a - 4);
                else if (a < 8 + NB) a0[a - 4 - NB] = oa.frag(ta, wm * 128 + (a - 4 - NB) * 32, 0, lane);   // past the
                else b0[a - 8 - NB] = ob.frag(tb, wn * (BN / 2) + (a - 8 - NB) * 32, 0, lane);          // last: unused
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // the epilogue issues ahead of the other workgroup's products on a shared SIMD, so that it
    // ends sooner and frees its LDS and the next tile starts (measured: forward with the loss
    // gradient 81 -> 77 us on the 65K head)
    __builtin_amdgcn_s_setprio(1);
    wait_vmcnt<0>();   // no load may still be writing LDS
    __syncthreads();   // and no wave still reads a stage: the LDS now stages the output

    // Loss gradient (EPI_BF16_BCE): the tile's targets as a bitmap [256 rows][BN / 32 words]
    // behind the staged half-tile (ids outside [n0, n0 + BN) or [0, N) ignored, repeats set the
    // same bit); the sigmoid is taken while staging.
    constexpr int TW = BN / 32;                          // target words per row
    uint32_t *tbits = reinterpret_cast<uint32_t *>(g4s + 128 * BN * 2);
    if constexpr (EPI == EPI_BF16_BCE) {
        for (int e = threadIdx.x; e < G4T * TW; e += 256) tbits[e] = 0u;
        __syncthreads();
        // one row per thread; its ids 8 at a time, all 8 loads in flight before any is used
        const int r = threadIdx.x;
        const bool live = m0 + r < M;
        const int32_t *pr = pos + (live ? (m0 + r) * P : 0);
        for (int p0 = 0; p0 < P; p0 += 8) {
            int id[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) id[u] = live && p0 + u < P ? pr[p0 + u] : -1;
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (id[u] >= n0 && id[u] < n0 + BN && id[u] < N) {
                    const int c = (int)(id[u] - n0);
                    atomicOr(&tbits[r * TW + (c >> 5)], 1u << (c & 31));
                }
        }
        __syncthreads();   // the bitmap is complete
    }

    // Output: one 128-row half of the tile at a time goes through LDS as [128 rows][BN columns]
    // (16-byte chunk c of row r at c ^ (r % XM + 1): the rows one store-to-LDS instruction touches
    // spread over the banks), then leaves as whole row pieces of BN elements, 1 KB per store
    // instruction.
    constexpr bool BF = EPI == EPI_BF16_BIAS || EPI == EPI_BF16_BCE;   // bf16 output
    constexpr int OB = BF ? 2 : 4;                      // output bytes per element
    constexpr int RB = BN * OB;                         // bytes per staged row
    constexpr int XM = RB / 16 - 1 < 31 ? RB / 16 - 1 : 31;   // chunk swizzle mask
    constexpr int RPI = 1024 / RB;                      // rows per store instruction
    char *eb = g4s;
    float *Cf = reinterpret_cast<float *>(C) + (EPI == EPI_F32_PART ? (int64_t)z * M * N : 0);
    bf16_t *Cb = reinterpret_cast<bf16_t *>(C);
    const int64_t ldo = EPI == EPI_F32_PART ? N : ldc;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if (wm == h) {
            // D^T[n = 8r + 4hh + q][m = ln] per 32x32 block: 4 consecutive columns per lane and r
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int nl = wn * (BN / 2) + j * 32 + 8 * r + 4 * hh;
                    float4 b = make_float4(0.f, 0.f, 0.f, 0.f);
                    if (BF && bias && n0 + nl < N)
                        b = *reinterpret_cast<const float4 *>(bias + n0 + nl);   // 16-byte aligned
                    const int byte = nl * OB;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int ml = i * 32 + ln;
                        const f32x16_t &d = acc[j][i];
                        char *p = eb + ml * RB + ((((byte >> 4) ^ (ml & XM)) << 4) | (byte & 15));
                        float4 v = make_float4(d[4 * r + 0] + b.x, d[4 * r + 1] + b.y, d[4 * r + 2] + b.z,
                                               d[4 * r + 3] + b.w);
                        if constexpr (EPI == EPI_BF16_BCE) {   // sigmoid, minus the targets of these 4 columns
                            const uint32_t tb = tbits[(128 * h + ml) * TW + (nl >> 5)] >> (nl & 31);
                            v = make_float4(sigmoid_f32(v.x), sigmoid_f32(v.y), sigmoid_f32(v.z), sigmoid_f32(v.w));
                            v.x -= (float)(tb & 1u);
                            v.y -= (float)((tb >> 1) & 1u);
                            v.z -= (float)((tb >> 2) & 1u);
                            v.w -= (float)((tb >> 3) & 1u);
                        }
                        if (BF)
                            *reinterpret_cast<uint2 *>(p) = make_uint2(pack_bf16(v.x, v.y), pack_bf16(v.z, v.w));
                        else
                            *reinterpret_cast<float4 *>(p) = v;
                    }
                }
        }
        __syncthreads();
        // 128 rows, RPI per instruction, spread over the 4 waves; columns past N are not stored
        // (N is a multiple of 8: a 16-byte chunk is all in or all out)
        const int rl = lane / (64 / RPI), c = lane % (64 / RPI);
        const int64_t n = n0 + (int64_t)c * (16 / OB);
        constexpr int NI = 128 / RPI / 4;                   // store instructions per wave
        constexpr int NBAT = NI < 8 ? NI : 8;               // issued in batches: reads, then stores
#pragma unroll
        for (int t0 = 0; t0 < NI; t0 += NBAT) {
            uint4 v[NBAT];
#pragma unroll
            for (int t = 0; t < NBAT; ++t) {
                const int row = RPI * (4 * (t0 + t) + wave) + rl;
                v[t] = *reinterpret_cast<const uint4 *>(eb + row * RB + ((c ^ (row & XM)) << 4));
            }
#pragma unroll
            for (int t = 0; t < NBAT; ++t) {
                const int64_t m = m0 + 128 * h + RPI * (4 * (t0 + t) + wave) + rl;
                if (m < M && n < N) {
                    // outputs written once and not read again soon: streaming stores
                    const u32x4_t wv = __builtin_bit_cast(u32x4_t, v[t]);
                    if (BF)
                        __builtin_nontemporal_store(wv, reinterpret_cast<u32x4_t *>(Cb + m * ldo + n));
                    else if (EPI == EPI_F32)
                        __builtin_nontemporal_store(wv, reinterpret_cast<u32x4_t *>(Cf + m * ldo + n));
                    else
                        *reinterpret_cast<uint4 *>(Cf + m * ldo + n) = v[t];
                }
            }
        }
        __syncthreads();
    }
}

// fp32 GEMM on the vector ALUs (fp32 heads): 64x64 tiles, 4x4 outputs per thread.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float *__restrict__ A, int64_t sam, int64_t sak,
                                                  const float *__restrict__ Bm, int64_t sbk, int64_t sbn,
                                                  void *__restrict__ C, int64_t ldc, const float *__restrict__ bias,
                                                  int64_t M, int64_t N, int64_t K, int64_t kchunk) {
    __shared__ float As[16][64 + 4];
    __shared__ float Bs[16][64 + 4];
    const int64_t n0 = (int64_t)blockIdx.x * 64, m0 = (int64_t)blockIdx.y * 64;
    const int64_t kb = (int64_t)blockIdx.z * kchunk;
    const int64_t ke = kb + kchunk < K ? kb + kchunk : K;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    float acc[4][4] = {};
    for (int64_t k0 = kb; k0 < ke; k0 += 16) {
        for (int e = threadIdx.x; e < 16 * 64; e += 256) {
            const int k = e >> 6, r = e & 63;
            As[k][r] = (m0 + r < M && k0 + k < ke) ? A[(m0 + r) * sam + (k0 + k) * sak] : 0.0f;
            Bs[k][r] = (n0 + r < N && k0 + k < ke) ? Bm[(k0 + k) * sbk + (n0 + r) * sbn] : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m >= M || n >= N) continue;
            const float v = acc[i][j];
            if (EPI == EPI_BF16_BIAS) {
                reinterpret_cast<float *>(C)[m * ldc + n] = v + (bias ? bias[n] : 0.0f);
            } else if (EPI == EPI_F32) {
                reinterpret_cast<float *>(C)[m * ldc + n] = v;
            } else {
                reinterpret_cast<float *>(C)[(int64_t)blockIdx.z * M * N + m * N + n] = v;
            }
        }
}

// split of the H contraction of dX for output tiles of tm x tn: enough workgroups to cover the
// chip (about `target`), never below 256 head labels per chunk.  at_most: never more than
// `target` workgroups, for the 256x256 kernel, which holds a whole CU (its LDS allows one
// workgroup per CU): one workgroup past the CU count would run in a second round on its own.
int64_t head_splits(int64_t B, int64_t F_s, int64_t H, int64_t tm, int64_t tn, int64_t target, bool at_most) {
    const int64_t tiles = haste::cdiv(B, tm) * haste::cdiv(F_s, tn) < 1 ? 1 : haste::cdiv(B, tm) * haste::cdiv(F_s, tn);
    int64_t S = at_most ? target / tiles : haste::cdiv(target, tiles);
    const int64_t maxS = haste::cdiv(H, 256);
    if (S > maxS) S = maxS;
    return S < 1 ? 1 : S;
}
int64_t head_splits_for(int64_t B, int64_t F_s, int64_t H, int32_t dtype, bool big) {
    if (dtype != HASTE_DTYPE_BF16) return head_splits(B, F_s, H, 64, 64, 512, false);
    return big ? head_splits(B, F_s, H, G4T, kHeadBN, kXcds * kCusPerXcd * (kHeadBN == 128 ? 2 : 1), true)
               : head_splits(B, F_s, H, TM, TN, 512, false);
}

// The double-buffered kernel needs 16-byte aligned rows along every operand's contiguous
// dimension (F_s and H multiples of 8) and operands within the 31-bit buffer range.
bool gemm2_ok(int64_t B, int64_t F_s, int64_t H) {
    const int64_t lim = ((int64_t)1 << 31) - 1;
    return F_s % 8 == 0 && H % 8 == 0 && B * F_s * 2 < lim && H * F_s * 2 < lim && B * H * 2 < lim;
}

// the 256x256 kernel loads and stores 16 bytes per lane and reads the bias 4 floats at a time:
// every pointer 16-byte aligned
bool gemm4_ok(int64_t B, int64_t F_s, int64_t H, std::initializer_list<const void *> ptrs) {
    if (!gemm2_ok(B, F_s, H)) return false;
    for (const void *p : ptrs)
        if ((reinterpret_cast<uintptr_t>(p) & 15) != 0) return false;
    return true;
}

// C[M, N] (+)= A B over K, split into Z chunks of kchunk (a multiple of the K step); sa, sb are
// the operands' row strides (elements).  256 x kHeadBN output tiles, or 256 x 64 where the wider
// ones would leave CUs idle (a 16K-label head over 256 rows: 128 tiles against 256 CUs).
template <int BN, bool AK, bool BK, int EPI>
hipError_t launch_gemm4_bn(hipStream_t s, const bf16_t *A, int64_t sa, int64_t a_elems, const bf16_t *Bm, int64_t sb,
                           int64_t b_elems, void *C, int64_t ldc, const float *bias, int64_t M, int64_t N, int64_t K,
                           int64_t kchunk, int Z, const int32_t *pos, int P) {
    const int MT = (int)haste::cdiv(M, G4T), NT = (int)haste::cdiv(N, BN);
    const int64_t grid = Z > 1 ? haste::round_up(Z, kXcds) * MT * NT
                               : (MT <= NT ? haste::round_up(NT, kXcds) * MT : haste::round_up(MT, kXcds) * NT);
    auto kern = k_gemm4<BN, AK, BK, EPI>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)g4_lds(BN));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(256), g4_lds(BN), s, A, sa, (uint32_t)(a_elems * 2), Bm, sb,
                       (uint32_t)(b_elems * 2), C, ldc, bias, M, N, K, kchunk, MT, NT, Z, pos, P);
    return hipGetLastError();
}

template <bool AK, bool BK, int EPI>
hipError_t launch_gemm4(hipStream_t s, const bf16_t *A, int64_t sa, int64_t a_elems, const bf16_t *Bm, int64_t sb,
                        int64_t b_elems, void *C, int64_t ldc, const float *bias, int64_t M, int64_t N, int64_t K,
                        int64_t kchunk, int Z, const int32_t *pos = nullptr, int P = 0) {
    const int64_t tiles = haste::cdiv(M, G4T) * haste::cdiv(N, kHeadBN) * Z;
    if (tiles < kXcds * kCusPerXcd && N % 64 == 0)
        return launch_gemm4_bn<64, AK, BK, EPI>(s, A, sa, a_elems, Bm, sb, b_elems, C, ldc, bias, M, N, K, kchunk, Z,
                                                pos, P);
    return launch_gemm4_bn<kHeadBN, AK, BK, EPI>(s, A, sa, a_elems, Bm, sb, b_elems, C, ldc, bias, M, N, K, kchunk, Z,
                                                 pos, P);
}

template <bool AK, bool BK, int EPI>
hipError_t launch_gemm2(dim3 grid, hipStream_t s, const bf16_t *A, int64_t sam, int64_t sak, int64_t a_elems,
                        const bf16_t *Bm, int64_t sbk, int64_t sbn, int64_t b_elems, void *C, int64_t ldc,
                        const float *bias, int64_t M, int64_t N, int64_t K, int64_t kchunk) {
    auto kern = k_gemm2<AK, BK, EPI>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)kG2Lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, dim3(256), kG2Lds, s, A, sam, sak, (uint32_t)(a_elems * 2), Bm, sbk, sbn,
                       (uint32_t)(b_elems * 2), C, ldc, bias, M, N, K, kchunk);
    return hipGetLastError();
}

}  // namespace

namespace haste {

size_t head_ws(int64_t B, int64_t F_s, int64_t H, int32_t dtype) {
    // either tile size may run (it also depends on the output's alignment): room for the larger split
    const int64_t S0 = head_splits_for(B, F_s, H, dtype, false), S1 = head_splits_for(B, F_s, H, dtype, true);
    return (size_t)(S0 > S1 ? S0 : S1) * (size_t)B * (size_t)F_s * 4 + 256;
}

hipError_t head_fwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const float *bias_h, void *Yh, hipStream_t s) {
    // M = B, N = H, K = F_s;  A(m,k) = X[m*F_s + k];  B(k,n) = Wh[n*F_s + k]
    if (dtype == HASTE_DTYPE_BF16) {
        if (gemm4_ok(B, F_s, H, {X, Wh, Yh, bias_h}))
            return launch_gemm4<true, true, EPI_BF16_BIAS>(s, (const bf16_t *)X, F_s, B * F_s, (const bf16_t *)Wh, F_s,
                                                           H * F_s, Yh, H, bias_h, B, H, F_s, F_s, 1);
        const dim3 grid((unsigned)cdiv(H, TN), (unsigned)cdiv(B, TM), 1);
        if (gemm2_ok(B, F_s, H))
            return launch_gemm2<true, true, EPI_BF16_BIAS>(grid, s, (const bf16_t *)X, F_s, 1, B * F_s,
                                                           (const bf16_t *)Wh, 1, F_s, H * F_s, Yh, H, bias_h, B, H,
                                                           F_s, F_s);
        hipLaunchKernelGGL((k_gemm_bf16<true, true, EPI_BF16_BIAS>), grid, dim3(256), 0, s, (const bf16_t *)X, F_s,
                           (int64_t)1, (const bf16_t *)Wh, (int64_t)1, F_s, Yh, H, bias_h, B, H, F_s, F_s);
    } else {
        const dim3 grid((unsigned)cdiv(H, 64), (unsigned)cdiv(B, 64), 1);
        hipLaunchKernelGGL((k_gemm_f32<EPI_BF16_BIAS>), grid, dim3(256), 0, s, (const float *)X, F_s, (int64_t)1,
                           (const float *)Wh, (int64_t)1, F_s, Yh, H, bias_h, B, H, F_s, F_s);
    }
    return hipGetLastError();
}

// dY_h = sigmoid(X W_head^T + bias_h) - T: the 256 kernel with the loss gradient in its epilogue
// where it applies (the logits never reach memory), else the logits into dY_h and the gradient in
// place
hipError_t head_fwd_bce(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                        const float *bias_h, const int32_t *pos, int P, void *dYh, hipStream_t s) {
    if (dtype == HASTE_DTYPE_BF16 && gemm4_ok(B, F_s, H, {X, Wh, dYh, bias_h}))
        return launch_gemm4<true, true, EPI_BF16_BCE>(s, (const bf16_t *)X, F_s, B * F_s, (const bf16_t *)Wh, F_s,
                                                      H * F_s, dYh, H, bias_h, B, H, F_s, F_s, 1, pos, P);
    const hipError_t e = head_fwd(B, F_s, H, dtype, X, Wh, bias_h, dYh, s);
    if (e != hipSuccess) return e;
    return bce_grad(B, H, dtype, dYh, pos, P, dYh, s);
}

hipError_t head_bwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const void *dYh, float *dWh, float *dX, int beta_dx, void *ws, hipStream_t s) {
    const bool bf = dtype == HASTE_DTYPE_BF16;
    if (dWh) {
        // M = H, N = F_s, K = B;  A(m,k) = dYh[k*H + m];  B(k,n) = X[k*F_s + n]
        if (bf && gemm4_ok(B, F_s, H, {X, dYh, dWh})) {
            // A(m, k) = dYh[k][m] (k-rows of H), B(k, n) = X[k][n] (k-rows of F_s)
            hipError_t e = launch_gemm4<false, false, EPI_F32>(s, (const bf16_t *)dYh, H, B * H, (const bf16_t *)X, F_s,
                                                               B * F_s, (void *)dWh, F_s, nullptr, H, F_s, B, B, 1);
            if (e != hipSuccess) return e;
        } else if (bf) {
            const dim3 grid((unsigned)cdiv(F_s, TN), (unsigned)cdiv(H, TM), 1);
            if (gemm2_ok(B, F_s, H)) {
                hipError_t e = launch_gemm2<false, false, EPI_F32>(grid, s, (const bf16_t *)dYh, 1, H, B * H,
                                                                   (const bf16_t *)X, F_s, 1, B * F_s, (void *)dWh,
                                                                   F_s, nullptr, H, F_s, B, B);
                if (e != hipSuccess) return e;
            } else {
                hipLaunchKernelGGL((k_gemm_bf16<false, false, EPI_F32>), grid, dim3(256), 0, s, (const bf16_t *)dYh,
                                   (int64_t)1, H, (const bf16_t *)X, F_s, (int64_t)1, (void *)dWh, F_s,
                                   (const float *)nullptr, H, F_s, B, B);
            }
        } else {
            const dim3 grid((unsigned)cdiv(F_s, 64), (unsigned)cdiv(H, 64), 1);
            hipLaunchKernelGGL((k_gemm_f32<EPI_F32>), grid, dim3(256), 0, s, (const float *)dYh, (int64_t)1, H,
                               (const float *)X, F_s, (int64_t)1, (void *)dWh, F_s, (const float *)nullptr, H, F_s,
                               B, B);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dX) {
        // M = B, N = F_s, K = H;  A(m,k) = dYh[m*H + k];  B(k,n) = Wh[k*F_s + n]; split over K
        float *part = reinterpret_cast<float *>(ws);
        const bool big = bf && gemm4_ok(B, F_s, H, {dYh, Wh, part});
        const int64_t S = head_splits_for(B, F_s, H, dtype, big);
        const int64_t kchunk = round_up(cdiv(H, S), 32);
        const int64_t Sx = cdiv(H, kchunk);
        if (big) {
            // A(m, k) = dYh[m][k] (rows of H), B(k, n) = Wh[k][n] (k-rows of F_s)
            hipError_t e = launch_gemm4<true, false, EPI_F32_PART>(s, (const bf16_t *)dYh, H, B * H, (const bf16_t *)Wh,
                                                                   F_s, H * F_s, (void *)part, F_s, nullptr, B, F_s, H,
                                                                   kchunk, (int)Sx);
            if (e != hipSuccess) return e;
        } else if (bf) {
            const dim3 grid((unsigned)cdiv(F_s, TN), (unsigned)cdiv(B, TM), (unsigned)Sx);
            if (gemm2_ok(B, F_s, H)) {
                hipError_t e = launch_gemm2<true, false, EPI_F32_PART>(grid, s, (const bf16_t *)dYh, H, 1, B * H,
                                                                       (const bf16_t *)Wh, F_s, 1, H * F_s,
                                                                       (void *)part, F_s, nullptr, B, F_s, H, kchunk);
                if (e != hipSuccess) return e;
            } else {
                hipLaunchKernelGGL((k_gemm_bf16<true, false, EPI_F32_PART>), grid, dim3(256), 0, s,
                                   (const bf16_t *)dYh, H, (int64_t)1, (const bf16_t *)Wh, F_s, (int64_t)1,
                                   (void *)part, F_s, (const float *)nullptr, B, F_s, H, kchunk);
            }
        } else {
            const dim3 grid((unsigned)cdiv(F_s, 64), (unsigned)cdiv(B, 64), (unsigned)Sx);
            hipLaunchKernelGGL((k_gemm_f32<EPI_F32_PART>), grid, dim3(256), 0, s, (const float *)dYh, H, (int64_t)1,
                               (const float *)Wh, F_s, (int64_t)1, (void *)part, F_s, (const float *)nullptr, B, F_s,
                               H, kchunk);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return reduce_rmajor(part, (int)Sx, B, F_s, dX, beta_dx, s);
    }
    return hipSuccess;
}

}  // namespace haste
