// Internal declarations shared by the HIP translation units of libhaste.so (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "haste.h"

typedef uint16_t bf16_t;  // bf16 bit pattern

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

// Hardware layout facts used by every kernel (CDNA4, 64-wide wavefronts).
constexpr int kWave = 64;
constexpr int kXcds = 8;          // MI355X: 8 XCDs, workgroups dispatched round-robin over them
constexpr int kCusPerXcd = 32;    // 256 CUs in total
constexpr int kMaxFs = 1024;      // widest input feature dimension the on-chip tiles are sized for

__device__ __forceinline__ float bf16_to_f32(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// fp32 -> bf16, round to nearest even (finite inputs; the hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    __bf16 h = (__bf16)f;
    return __builtin_bit_cast(bf16_t, h);
}

__device__ __forceinline__ float load_f32(const float *p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_f32(const bf16_t *p, int64_t i) { return bf16_to_f32(p[i]); }
__device__ __forceinline__ void store_out(float *p, int64_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_out(bf16_t *p, int64_t i, float v) { p[i] = f32_to_bf16(v); }

// ds_read_b64_tr_b16: within each 16-lane group, lane r names an 8-byte word M[r] (4 bf16);
// result lane i receives M[4j + i/4][i % 4] as element j (j = 0..3).  p must be 8-byte aligned
// and point into LDS.
__device__ __forceinline__ uint2 lds_read_tr(const void *p) {
    const bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t *)(p));
    return __builtin_bit_cast(uint2, v);
}

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16).
// Lane l holds A[l % 32][8*(l/32) .. +7], B[8*(l/32) .. +7][l % 32] and
// D[8*i + 4*(l/32) + j][l % 32] in register 4*i + j.
__device__ __forceinline__ f32x16_t mfma32x32x16(const bf16x8_t &a, const bf16x8_t &b, const f32x16_t &c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// f(integral_constant<int, I>) for I = 0 .. N - 1, unrolled at compile time
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ uint32_t pack2(bf16_t lo, bf16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16 pair (round to nearest even; one v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// registers r0..r0+7 of an MFMA result as one bf16x8 operand
__device__ __forceinline__ uint4 pack8(const f32x16_t &d, int r0) {
    return make_uint4(pack_bf16(d[r0 + 0], d[r0 + 1]), pack_bf16(d[r0 + 2], d[r0 + 3]),
                      pack_bf16(d[r0 + 4], d[r0 + 5]), pack_bf16(d[r0 + 6], d[r0 + 7]));
}

// Bounds-checked buffer access (raw buffer resource, stride 0).  Loads at byte offsets at or past
// `bytes` return zero and stores there are dropped by the hardware, so masked lanes simply use
// kOob: no branch around the memory instruction, which keeps the count of outstanding memory
// operations the same on every path (the compiler can then wait for exactly the loads a use
// needs).  `base` must be wave-uniform; offsets are 32-bit.
constexpr uint32_t kOob = 0x80000000u;
constexpr int kRawBufferWord3 = 0x00020000;  // gfx9-family raw buffer format word

constexpr int kStreaming = 2;  // non-temporal ("nt") cache policy of a buffer access

struct Buf {
    __amdgpu_buffer_rsrc_t r;
    __device__ __forceinline__ Buf(const void *base, uint32_t bytes)
        : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0,
                                              (int)(bytes < kOob ? bytes : kOob - 1), kRawBufferWord3)) {}
    __device__ __forceinline__ uint32_t ld4(uint32_t off) const {
        return __builtin_bit_cast(uint32_t, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
    }
    __device__ __forceinline__ uint2 ld8(uint32_t off) const {
        return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0));
    }
    __device__ __forceinline__ uint4 ld16(uint32_t off) const {
        return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
    }
    // POLICY: cache-policy bits of the instruction (kStreaming marks data not read again soon)
    template <int POLICY = 0>
    __device__ __forceinline__ void st8(uint2 v, uint32_t off) const {
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b64(r, 0, 0, 0)), v),
                                              r, (int)off, 0, POLICY);
    }
    template <int POLICY = 0>
    __device__ __forceinline__ void st16(uint4 v, uint32_t off) const {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(r, 0, 0, 0)), v),
                                               r, (int)off, 0, POLICY);
    }
};

// The backward-feature accumulator dX^T[F_s][32 rows] (fp32) in LDS: row f is 128 bytes, and its
// 16-byte chunk c (rows 4c .. 4c + 3) sits at chunk position c ^ (f mod 8).  A matrix-core result
// tile writes one chunk of 16 rows at a time (lane l16 -> row f_l16), so the XOR spreads those
// rows over the banks without padding (less LDS than 36- or 40-float rows, and fewer conflicts
// than either on the 16-row tiles of random supports).  acc_row(f): the row's byte offset with
// its swizzle, so that chunk c of the row is at acc_row(f) ^ (c << 4).
__host__ __device__ constexpr uint32_t acc_row(int f) { return (uint32_t)f * 128u | (((uint32_t)f & 7u) << 4); }
__host__ __device__ constexpr int acc_index(int f, int r) {   // float index of row r of accumulator row f
    return f * 32 + ((((r >> 2) ^ f) & 7) << 2) + (r & 3);
}

// Slot order of a group's support for the backward-feature accumulator.  Rows of distinct
// residue mod 8 fall in distinct banks for the 8 lanes an access serves together, so slots are
// ordered by (occurrence of the residue so far, row mod 8), which deals the residues round-robin
// over the runs of 8 positions: a residue held by at most F_in / 8 slots never appears twice in a
// run (measured on 16-row tiles of random 64-slot supports: 1.4x the conflict-free read time
// against 2.2x for sorted order).  For the slots t = lane and
// t = lane + 64 (those below F_in) of support `sup`: f = the feature (-1 past F_in) and pos = its
// position (-1 past F_in).  Wave-level: every lane of the wave must call it.
__device__ __forceinline__ void slot_positions(const int32_t *sup, int F_in, int lane, int (&f)[2], int (&pos)[2]) {
    int cls[2], occ[2] = {0, 0};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int t = lane + 64 * i;
        f[i] = t < F_in ? sup[t] : -1;
        cls[i] = f[i] >= 0 ? (f[i] & 7) : -1;
    }
    const uint64_t lt = __lanemask_lt();
    int cnt[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) {
        const uint64_t m0 = __ballot(cls[0] == v), m1 = __ballot(cls[1] == v);
        if (cls[0] == v) occ[0] = __popcll(m0 & lt);
        if (cls[1] == v) occ[1] = __popcll(m0) + __popcll(m1 & lt);
        cnt[v] = __popcll(m0) + __popcll(m1);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        pos[i] = -1;
        if (cls[i] < 0) continue;
        const int r = cls[i], o = occ[i];
        int rank = 0;                             // slots with a smaller (occurrence, residue)
#pragma unroll
        for (int v = 0; v < 8; ++v) rank += (cnt[v] < o ? cnt[v] : o) + (v < r && cnt[v] > o ? 1 : 0);
        pos[i] = rank;
    }
}

// Gradient of the binary cross-entropy of sigmoid(z) against a 0/1 target with respect to the
// logit z (Section 3.3 objective): sigmoid(z) - y, in fp32.  exp(-z) overflows to +inf for very
// negative z, which gives sigmoid 0 as it should.
__device__ __forceinline__ float sigmoid_f32(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

__device__ __forceinline__ float bce_grad_f32(float z, bool positive) {
    const float sg = sigmoid_f32(z);
    return positive ? sg - 1.0f : sg;
}

// The loss-gradient targets of one batch row over an increasing sequence of label windows, read
// from the row's positives sorted ascending (INT32_MAX past the last; sort_positives): `cur` is
// the first positive not yet passed.  Windows must not go back.
struct PosCursor {
    const int32_t *p;
    int P, cur;
    int32_t nxt;
    // start at the first positive >= first (binary search)
    __device__ __forceinline__ void init(const int32_t *row, int P_, int64_t first) {
        p = row;
        P = P_;
        int lo = 0, hi = P_;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if ((int64_t)row[mid] < first) lo = mid + 1;
            else hi = mid;
        }
        cur = lo;
        nxt = cur < P ? p[cur] : INT32_MAX;
    }
    // bit e set where label lab + e (e < n <= 32) is a positive of the row
    __device__ __forceinline__ uint32_t bits(int64_t lab, int n) {
        uint32_t t = 0;
        while (nxt != INT32_MAX && (int64_t)nxt < lab + n) {
            if ((int64_t)nxt >= lab) t |= 1u << (uint32_t)(nxt - lab);
            ++cur;
            nxt = cur < P ? p[cur] : INT32_MAX;
        }
        return t;
    }
};

// bf16 pair -> the loss gradients of both logits (targets bit 0 and bit 1 of t), as a bf16 pair
__device__ __forceinline__ uint32_t bce_pair(uint32_t w, uint32_t t) {
    return pack_bf16(bce_grad_f32(__uint_as_float(w << 16), t & 1u), bce_grad_f32(__uint_as_float(w & 0xffff0000u), (t >> 1) & 1u));
}

// One step of SGD with momentum on one weight (the classification layer's optimizer, Section 4):
// velocity m <- momentum * m + (g + weight_decay * w), then w_next = w - lr * m.  Explicit fused
// multiply-adds, so that every kernel that applies the step rounds it the same way.
__device__ __forceinline__ void sgd_step(float w, float g, float &m, float &w_next, float lr, float momentum,
                                         float weight_decay) {
    m = __fmaf_rn(momentum, m, __fmaf_rn(weight_decay, w, g));
    w_next = __fmaf_rn(-lr, m, w);
}

// ---- host-side launchers (one translation unit each) -----------------------------------------
namespace haste {

struct TailArgs {
    int64_t B, F_s, L, G, F_in;
    int32_t dtype;
};

// records the calling thread's haste_last_error() message and returns code (abi.hip)
int report(int code, const char *fmt, ...);

// tail, MFMA (bf16)
bool fwd_mfma_supported(const TailArgs &a);
hipError_t fwd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s);
// forward for small groups (G = 1, 2, 4, 8), 16 / G groups per matrix tile
bool fwd_sg_supported(const TailArgs &a);
// spos (optional): the rows' positives sorted by sort_positives; the output is then the loss
// gradient sigmoid(Y) - T of the bf16 logits, bit for bit as bce_grad computes it
hipError_t fwd_sg(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias, void *Y,
                  hipStream_t s, const int32_t *spos = nullptr, int P = 0);
// backward-weight for small groups (G = 1, 2, 4, 8), on the workspace's X^T copy (bwd_w_mfma_ws)
bool bwd_w_sg_supported(const TailArgs &a);
hipError_t bwd_w_sg(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW, float *dbias,
                    int beta, void *ws, hipStream_t s);
hipError_t transpose_x(const TailArgs &a, const void *X, void *ws, hipStream_t s);
// backward-feature for small groups (G = 1, 2, 4, 8), 32 consecutive labels per matrix-core K step
bool bwd_x_sg_supported(const TailArgs &a);
size_t bwd_x_sg_ws(const TailArgs &a);
hipError_t bwd_x_sg(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta, void *ws,
                    hipStream_t s);
// backward-feature for small groups (G = 1, 2, 4, 8, F_s <= 800) as a dense product over each
// 32-label step's weights scattered into an LDS tile
bool bwd_x_dn_supported(const TailArgs &a);
size_t bwd_x_dn_ws(const TailArgs &a);
hipError_t bwd_x_dn(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta, void *ws,
                    hipStream_t s);
// forward for groups of 1 or 2 labels (F_s <= 768) as a dense product over each 32-label step's
// weights scattered into an LDS tile
bool fwd_dn_supported(const TailArgs &a);
hipError_t fwd_dn(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias, void *Y,
                  hipStream_t s, const int32_t *spos = nullptr, int P = 0);
// backward-weight for groups of 1 or 2 labels (F_s <= 768) as the dense product dY^T X of 64-label
// blocks, the supports' entries picked out of it (X^T copy in the workspace)
bool bwd_w_dn_supported(const TailArgs &a);
hipError_t bwd_w_dn(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW, float *dbias,
                    int beta, void *ws, hipStream_t s);
bool bwd_w_mfma_supported(const TailArgs &a);
size_t bwd_w_mfma_ws(const TailArgs &a);
hipError_t bwd_w_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, void *ws, hipStream_t s);
// the tail's training pass in two kernels' worth of work: fused forward + loss gradient + dW, then
// backward-feature reading the transposed weights the first one wrote (groups of 32 labels)
bool tail_step_fused(const TailArgs &a, int P);
size_t tail_step_ws(const TailArgs &a, int P);
hipError_t tail_step_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                          const int32_t *pos, int P, void *dY, float *dW, float *dbias, int beta, float *dX,
                          int beta_dx, void *ws, hipStream_t s);
hipError_t tail_step_sgd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                              const int32_t *pos, int P, void *dY, float *dbias, const haste_sgd_t &opt, float *m,
                              void *W_next, float *dX, int beta_dx, void *ws, size_t fb_ws_bytes, hipStream_t s);
bool bwd_x_mfma_supported(const TailArgs &a);
size_t bwd_x_mfma_ws(const TailArgs &a);
hipError_t bwd_x_mfma(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s);

// forward with the BCE-gradient epilogue, optionally fused with backward-weight (bf16, MFMA); the
// workspace query provides for rows of up to kFusedPosWs positives
constexpr int kFusedPosWs = 1024;
bool fwd_bce_mfma_supported(const TailArgs &a, int P);
size_t fwd_bce_mfma_ws(const TailArgs &a, int P);   // P: positives per row
hipError_t fwd_bce_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                        const int32_t *pos, int P, void *dY, float *dW, float *dbias, int beta, void *ws,
                        hipStream_t s);
// forward + BCE gradient + backward-weight with the momentum step applied to W in place of storing dW
hipError_t fwd_bce_sgd_mfma(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                            const int32_t *pos, int P, void *dY, float *dbias, const haste_sgd_t &opt, float *m,
                            void *W_next, void *ws, hipStream_t s);
// momentum step over n weights: m and W_next updated (W_next may alias W)
hipError_t sgd_momentum(int64_t n, int32_t dtype, const void *W, const float *g, float *m, const haste_sgd_t &opt,
                        void *W_next, hipStream_t s);
// group-shared rewiring (Alg. 3); n_prune >= 1
bool rewire_supported(const TailArgs &a);
size_t rewire_ws(const TailArgs &a);
hipError_t rewire(const TailArgs &a, int32_t *idx, void *W, float *m, int64_t n_prune, int init_random, uint64_t seed,
                  void *ws, hipStream_t s);
// semantic grouping of labels (Alg. 2) on int8 unit embeddings
bool group_supported(int64_t N, int64_t D, int64_t G, int64_t beta);
size_t group_ws(int64_t N, int64_t D, int64_t G, int64_t beta);
hipError_t group_labels(int64_t N, int64_t D, const int8_t *E, int64_t G, int64_t beta, int64_t iters, uint64_t seed,
                        int32_t *order, int32_t *gsize, int64_t *n_groups, int32_t *cluster, void *ws, hipStream_t s);
// spos[b][0..P): row b's positives in [0, N) sorted ascending, the rest INT32_MAX (P <= kSortPosMax)
constexpr int kSortPosMax = 256;
hipError_t sort_positives(int64_t B, int64_t N, const int32_t *pos, int P, int32_t *spos, hipStream_t s);
// dY[b, n] = sigmoid(Y[b, n]) - T[b, n] elementwise (Y and dY may alias)
hipError_t bce_grad(int64_t B, int64_t N, int32_t dtype, const void *Y, const int32_t *pos, int P, void *dY,
                    hipStream_t s);

// tail, VALU (fp32 and bf16, any G including per-label fixed fan-in)
bool valu_supported(const TailArgs &a);
hipError_t fwd_valu(const TailArgs &a, const void *X, const int32_t *idx, const void *W, const float *bias,
                    void *Y, hipStream_t s);
hipError_t bwd_w_valu(const TailArgs &a, const void *X, const int32_t *idx, const void *dY, float *dW,
                      float *dbias, int beta, hipStream_t s);
size_t bwd_x_valu_ws(const TailArgs &a);
hipError_t bwd_x_valu(const TailArgs &a, const int32_t *idx, const void *W, const void *dY, float *dX, int beta,
                      void *ws, hipStream_t s);

// dense head
size_t head_ws(int64_t B, int64_t F_s, int64_t H, int32_t dtype);
hipError_t head_fwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const float *bias_h, void *Yh, hipStream_t s);
// dY_h = sigmoid(X W_head^T + bias_h) - T (T from pos[B, P] as in bce_grad)
hipError_t head_fwd_bce(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                        const float *bias_h, const int32_t *pos, int P, void *dYh, hipStream_t s);
hipError_t head_bwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X, const void *Wh,
                    const void *dYh, float *dWh, float *dX, int beta_dx, void *ws, hipStream_t s);

// utilities
hipError_t fill_f32(float *p, int64_t n, float v, hipStream_t s);
// dX[b, f] = beta*dX[b, f] + sum_s part[s][f][b]   (part is [S][F_s][ldp], feature-major)
hipError_t reduce_fmajor(const float *part, int S, int64_t ldp, int64_t B, int64_t F_s, float *dX, int beta,
                         hipStream_t s);
// C[m, n] = beta*C[m, n] + sum_s part[s][m][n]     (part is [S][M][N], row-major)
hipError_t reduce_rmajor(const float *part, int S, int64_t M, int64_t N, float *C, int beta, hipStream_t s);
hipError_t validate_idx(const int32_t *idx, int64_t rows, int64_t F_in, int64_t F_s, int32_t *n_bad,
                        hipStream_t s);
hipError_t debug_gather(const void *X, int32_t dtype, const int32_t *idx, int64_t B, int64_t F_s, int64_t F_in,
                        int64_t k0, int64_t nk, void *out, hipStream_t s);

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

}  // namespace haste
