/*
 * haste.h - C ABI of libhaste.so, the MI355X (gfx950) implementation of the group-shared fixed
 * fan-in (GS-FFI) output layer and its dense head.
 *
 * The layer (paper, Section 3.1): L labels are split into K = L/G groups of exactly G labels.
 * Labels of a group are contiguous, so label l belongs to group g(l) = l / G.  Group k owns one
 * support I_k of F_in input features, stored as row k of idx[K, F_in].  Label l keeps its own
 * weight vector W[l, 0..F_in-1]; slot t of that vector multiplies feature idx[g(l), t].
 * G = 1 is standard (per-label) fixed fan-in: idx then has L rows.
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller, dense, row-major, and aligned
 *     to at least 16 bytes.  The library never allocates, frees or copies them.
 *   - "dtype" selects the storage type of X, W, Y, dY (and W_head, Y_h, dY_h):
 *       HASTE_DTYPE_F32  - IEEE fp32, all arithmetic fp32;
 *       HASTE_DTYPE_BF16 - bf16 storage, products accumulated in fp32, bf16 outputs rounded to
 *                          nearest-even.
 *     bias, dbias, dW, dX and dW_head are always fp32.
 *   - idx is int32.  Every row must be strictly increasing and lie in [0, F_s): a precondition,
 *     not checked per call (haste_validate_idx checks it).
 *   - "stream" is a hipStream_t passed as void* (NULL = the default stream).  Every call only
 *     enqueues work on that stream and returns; a kernel fault surfaces at the caller's next
 *     synchronisation.  Calls never synchronise the device.
 *   - "ws" is caller-owned device scratch of ws_bytes bytes; the required size is given by
 *     haste_workspace_bytes / haste_head_workspace_bytes.  Concurrent calls must use distinct
 *     workspaces.
 *   - Return value: HASTE_OK, or an error code; on error nothing is launched and
 *     haste_last_error() describes the cause (per calling thread).
 *   - 64-bit sizes throughout; B * L may exceed 2^31.
 */
#ifndef HASTE_H_
#define HASTE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum haste_dtype { HASTE_DTYPE_F32 = 0, HASTE_DTYPE_BF16 = 1 };

enum haste_status {
    HASTE_OK = 0,
    HASTE_ERR_INVALID = 1,      /* bad shape, null pointer, misalignment, L % G != 0 ...   */
    HASTE_ERR_UNSUPPORTED = 2,  /* valid arguments outside what the kernels implement      */
    HASTE_ERR_WORKSPACE = 3,    /* ws_bytes smaller than the reported requirement           */
    HASTE_ERR_HIP = 4           /* the HIP runtime refused a launch                         */
};

/* Workspace-query operation codes. */
enum haste_op {
    HASTE_OP_FWD = 0, HASTE_OP_BWD_W = 1, HASTE_OP_BWD_X = 2, HASTE_OP_FWD_BCE = 3, HASTE_OP_FWD_BCE_SGD = 4,
    HASTE_OP_REWIRE = 5, HASTE_OP_TAIL_STEP = 6, HASTE_OP_TAIL_STEP_SGD = 7
};

/* Hyper-parameters of one step of SGD with momentum (see haste_sgd_momentum). */
typedef struct haste_sgd {
    float lr;            /* learning rate                                               */
    float momentum;      /* velocity decay, in [0, 1)                                   */
    float weight_decay;  /* L2 coefficient added to the gradient (0 = none)             */
    int32_t reserved;    /* must be 0                                                   */
} haste_sgd_t;

/* Shape of one sparse tail layer. */
typedef struct haste_desc {
    int64_t B;      /* batch rows (>= 0)                                         */
    int64_t F_s;    /* input feature width (> 0)                                 */
    int64_t L;      /* tail labels (>= 0), a multiple of G                       */
    int64_t G;      /* labels per group (> 0)                                    */
    int64_t F_in;   /* support size per group, fixed fan-in (1 <= F_in <= F_s)   */
    int32_t dtype;  /* enum haste_dtype                                          */
    int32_t reserved;  /* must be 0                                              */
} haste_desc_t;

/*
 * Forward logits of the tail (Section 3.1 logit; Section 3.2 "gather-once and dense MMA"):
 *   Y[b, l] = bias[l] + sum_{t < F_in} X[b, idx[l/G, t]] * W[l, t]
 * X[B, F_s], idx[L/G, F_in] int32, W[L, F_in], bias[L] fp32 or NULL (no bias), Y[B, L] (dtype),
 * overwritten.
 */
int haste_fwd(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
              const float *bias, void *Y, void *ws, size_t ws_bytes, void *stream);

/*
 * Backward-weight of the tail (Section 3.2: grad W_k = (grad Z_k)^T H_k, formed only on the
 * support of each group):
 *   dW[l, t] = beta * dW[l, t] + sum_b dY[b, l] * X[b, idx[l/G, t]]
 *   dbias[l] = beta * dbias[l] + sum_b dY[b, l]            (skipped when dbias is NULL)
 * dY[B, L] (dtype); dW[L, F_in] fp32; beta is 0 (overwrite) or 1 (accumulate).
 */
int haste_bwd_w(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *dY,
                float *dW, float *dbias, int beta, void *ws, size_t ws_bytes, void *stream);

/*
 * Backward-feature of the tail (Section 3.2: grad h_{:, I_k} += grad Z_k W_k, reduced over all
 * groups with a split over the label dimension):
 *   dX[b, f] = beta * dX[b, f] + sum_k sum_{t : idx[k,t] = f} sum_{j < G} dY[b, kG+j] * W[kG+j, t]
 * dX[B, F_s] fp32; beta is 0 (overwrite) or 1 (accumulate).  Partial sums over label segments
 * live in ws and are reduced in a fixed segment order; on the bf16 matrix-core path ws also
 * holds a group-transposed copy of W (about L * F_in * 2 bytes), rebuilt by every call.
 */
int haste_bwd_x(const haste_desc_t *desc, const int32_t *idx, const void *W, const void *dY,
                float *dX, int beta, void *ws, size_t ws_bytes, void *stream);

/*
 * Forward of the tail with the gradient of the binary cross-entropy objective as its epilogue
 * (Section 3.1 logit; Section 3.3 objective, whose derivative in a logit z is sigmoid(z) - y),
 * optionally fused with the backward-weight product of that gradient (Section 3.2):
 *   z[b, l]  = bias[l] + sum_{t < F_in} X[b, idx[l/G, t]] * W[l, t]        (not stored)
 *   dY[b, l] = sigmoid(z[b, l]) - T[b, l]                                  (dtype, overwritten)
 *   T[b, l]  = 1 if l occurs among pos[b, 0..P-1], else 0
 *   if dW != NULL:    dW[l, t] = beta * dW[l, t] + sum_b dY[b, l] * X[b, idx[l/G, t]]
 *   if dbias != NULL: dbias[l] = beta * dbias[l] + sum_b dY[b, l]          (needs dW)
 * The dW and dbias sums use dY as stored (rounded to dtype); they equal haste_bwd_w on the
 * returned dY.
 * pos[B, P] int32 holds each row's positive tail labels as column ids; entries outside [0, L)
 * (e.g. -1 padding) are ignored and a repeated id counts once.  P >= 0; pos may be NULL when
 * P == 0.  bias as in haste_fwd; beta is 0 (overwrite) or 1 (accumulate).
 * bf16 layers whose groups are whole 16-label tiles, with F_s <= 1024, run one fused kernel (the
 * logits never reach memory), for any number of positives per row: rows of more than 64 are first
 * bucketed by workgroup and batch slab in the workspace, whose queried size provides for up to
 * 1024 per row (2 F_s round_up(B, 32) + 8 (L B / 512) + 4 B P bytes about; a larger P fuses when
 * ws holds that much, else composes).  Other layers run haste_fwd into dY, the gradient in place
 * (for bf16 the sigmoid then sees the logits rounded to bf16), and haste_bwd_w; for bf16 groups of
 * 1, 2, 4 or 8 labels with rows of up to 256 positives the forward kernel itself stores that same
 * gradient (bit for bit), after sorting each row's positives into the workspace (B * P * 4 bytes
 * after the X^T copy; the queried size provides for 256 per row).
 * ws: haste_workspace_bytes(desc, HASTE_OP_FWD_BCE) bytes.
 */
int haste_fwd_bce(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
                  const float *bias, const int32_t *pos, int32_t P, void *dY, float *dW,
                  float *dbias, int beta, void *ws, size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): haste_fwd_bce with its scratch in a device array the library owns, so
 * the call takes no workspace and allocates nothing.  Arguments, results and errors are those of
 * haste_fwd_bce, bit for bit, without ws / ws_bytes.
 * Limit: the call's scratch (the X^T copy, 2 F_s round_up(B, 32) + 256 bytes on the matrix-core
 * path, plus on the fused kernel's shapes the bucketed positives of rows of more than 64) must not
 * exceed haste_fwd_bce_static_max_bytes() (8 MiB); a larger call gives HASTE_ERR_UNSUPPORTED and
 * launches nothing.
 * Each GPU holds one such array for the life of the process, shared by every call on that GPU and
 * left holding the last call's data (each call writes all it reads): calls that overlap on one GPU
 * (other streams or threads) race on it, and the caller must serialise them.  The array's device
 * address is looked up on the first call on each device; the current device must be the one the
 * stream belongs to.
 */
int haste_fwd_bce_static(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
                         const float *bias, const int32_t *pos, int32_t P, void *dY, float *dW,
                         float *dbias, int beta, void *stream);

/* Bytes of scratch haste_fwd_bce_static holds per device (its limit). */
size_t haste_fwd_bce_static_max_bytes(void);

/*
 * haste_fwd_bce followed by one step of SGD with momentum on W (the classification layer's
 * optimizer, Section 4), with the step applied where the backward-weight product is formed, so
 * that dW never reaches memory:
 *   dY as in haste_fwd_bce;  dW as in haste_fwd_bce (not stored);
 *   m[l, t]      = momentum * m[l, t] + (dW[l, t] + weight_decay * W[l, t])     (fp32, updated)
 *   W_next[l, t] = W[l, t] - lr * m[l, t]                                         (dtype)
 * m[L, F_in] fp32 (zeros before the first step); W_next[L, F_in] in the dtype of W, and it must
 * not overlap W (the backward-feature call of the same step still reads W).  dbias: optional
 * gradient output as in haste_fwd_bce (the bias's own step is a haste_sgd_momentum call).
 * The fp32 arithmetic of the step is that of haste_sgd_momentum, so the result equals
 * haste_fwd_bce + haste_sgd_momentum bit for bit.  Layers outside the fused kernel's shapes (those
 * of haste_fwd_bce) run exactly that composition, with dW in ws.  On the fused shapes rows of more
 * than 1024 positives need more workspace than the query gives (HASTE_ERR_WORKSPACE names it).
 * B == 0 applies the step with a zero gradient.
 * ws: haste_workspace_bytes(desc, HASTE_OP_FWD_BCE_SGD) bytes.
 */
int haste_fwd_bce_sgd(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
                      const float *bias, const int32_t *pos, int32_t P, void *dY, float *dbias,
                      const haste_sgd_t *opt, float *m, void *W_next, void *ws, size_t ws_bytes,
                      void *stream);

/*
 * One step of SGD with momentum (Section 4: the classification layer is trained with SGD and
 * momentum), in the common form without dampening or look-ahead, over n weights:
 *   m[i]      = momentum * m[i] + (grad[i] + weight_decay * W[i])
 *   W_next[i] = W[i] - lr * m[i]
 * W, W_next [n] in dtype (W_next may be W: an in-place step); grad [n] (NULL: a zero gradient) and
 * m [n] fp32, m updated.  momentum must lie in [0, 1).
 * Arithmetic: fp32 fused multiply-adds; a bf16 W_next is rounded to nearest even.
 */
int haste_sgd_momentum(int64_t n, int32_t dtype, const void *W, const float *grad, float *m,
                       const haste_sgd_t *opt, void *W_next, void *stream);

/*
 * Group-shared rewiring (Alg. 3; the discrete phase of the alternating training loop, Section 3.3), in place:
 *   1. score[k, j] = sum over the G labels l of group k of |W[l, j]|, fp32, labels in order (the
 *      algorithm's mean, scaled by the common factor G, which orders the scores identically);
 *   2. prune the m = floor(K * F_in * rho) smallest scores over all groups, ties to the lower
 *      flat index k * F_in + j;
 *   3. each pruned slot of group k, in ascending slot order, takes a feature drawn uniformly from
 *      [0, F_s) minus the features the group keeps and those drawn before it (rows stay sets);
 *      then row k is re-sorted, each slot carrying its weight column W[kG .. kG+G-1, j] and its
 *      velocity m[.., j] with it;
 *   4. pruned slots' weights: 0 (init_random = 0) or uniform in [-1/sqrt(F_in), 1/sqrt(F_in)]
 *      (init_random = 1), stored in the dtype of W; their velocity is set to 0.
 * Draws: SplitMix64 (Steele, Lea and Flood, 2014) in counter form, output i of the stream seeded
 * with `seed`: the new feature of slot j of group k is the (out(k F + j) mod n_free)-th free
 * feature in ascending order; label l's new weight at slot j is ((2 n - 2^24) as fp32) *
 * (fp32(1/sqrt(F_in)) * 2^-24) with n = out(K F + l F + j) >> 40.
 * idx [K, F_in] int32 (strictly increasing rows, precondition), W [L, F_in] (dtype) and m
 * [L, F_in] fp32 (or NULL) are updated in place.  rho in [0, 1); *n_pruned (host, or NULL)
 * receives m.  F_in <= 256.  ws: haste_workspace_bytes(desc, HASTE_OP_REWIRE) bytes; desc->B is
 * not used.
 */
int haste_rewire(const haste_desc_t *desc, int32_t *idx, void *W, float *m, double rho, int32_t init_random,
                 uint64_t seed, int64_t *n_pruned, void *ws, size_t ws_bytes, void *stream);

/* Options of haste_group_labels. */
typedef struct haste_group_opts {
    int64_t G;       /* group size (1 .. 256)                                         */
    int64_t beta;    /* bucket factor: C = max(1, floor(N / (beta * G))) clusters      */
    int64_t iters;   /* k-means iterations (>= 0)                                      */
    uint64_t seed;   /* SplitMix64 seed of the initial centres and the group seeds      */
} haste_group_opts_t;

/*
 * Semantic grouping of labels (Alg. 2; Section 3.1, "Label Grouping"), before training: coarse
 * spherical k-means into C clusters, then, inside each cluster, greedy groups: a random unassigned
 * seed together with its top-(G - 1) unassigned neighbours by cosine similarity, until the cluster
 * is used up.  The seed always belongs to its own group.
 *   - E [N, D] int8: label embeddings (unit vectors scaled by 127 and rounded); every row must be
 *     non-zero (a precondition).  Similarity is the cosine of the stored rows.
 *   - k-means: a centre is the normalised mean of its members, held exactly as the integer sum s
 *     of their rows; a label e goes to the centre maximising e.s / |s| (its cosine up to the
 *     label's own norm), formed in fp64 from the exact integer e.s and |s| = sqrt of the exact
 *     |s|^2 rounded once, ties to the lower centre.  Centres start as the first C labels of a
 *     partial Fisher-Yates shuffle of [0, N) (swap partner of i: i + out(i) mod (N - i)); `iters`
 *     full Lloyd iterations follow (assign every label, then move every non-empty cluster's centre
 *     to its members' sum; a zero sum keeps the centre), then a final assignment.  (The paper runs
 *     mini-batch k-means, a CPU economy; full passes of the [N, D] x [D, C] product are cheap on
 *     the GPU.)
 *   - groups: cluster by cluster; the t-th seed of cluster c is the (out(N + c N + t) mod
 *     n_unassigned)-th unassigned member in ascending label order; the other members are the
 *     unassigned labels of largest cosine (e_i.e_s) / sqrt(|e_i|^2 |e_s|^2) in fp64, ties to the
 *     lower label; a group lists its labels in ascending order.  The last group of a cluster may
 *     have fewer than G labels (the layout needs L % G == 0: pad with zero-weight labels).
 *   out(i) is SplitMix64 (Steele, Lea and Flood, 2014) output i of the stream seeded with seed.
 * order [N] int32 receives the labels group after group; gsize [N] int32 the group sizes (first
 * *n_groups entries); n_groups is a DEVICE int64; cluster [N] int32 (device, or NULL) the final
 * cluster of each label.  D % 16 == 0, D <= 1024, N < 2^24, N D < 2^31, 4 C D < 2^31; otherwise
 * HASTE_ERR_UNSUPPORTED.
 * ws: haste_group_workspace_bytes(N, D, opts) bytes.
 */
int haste_group_labels(int64_t N, int64_t D, const int8_t *E, const haste_group_opts_t *opts, int32_t *order,
                       int32_t *gsize, int64_t *n_groups, int32_t *cluster, void *ws, size_t ws_bytes,
                       void *stream);

/*
 * The tail's training pass (Section 3.2 forward and both backward products, with the gradient of
 * the Section 3.3 objective): haste_fwd_bce (dY, dW, dbias as documented there) followed by
 *   dX = beta_dx * dX + scatter(dY W)        as haste_bwd_x, on the dY just formed.
 * Same arguments and rules as those two calls; beta applies to dW and dbias, beta_dx to dX.
 * Results equal the two calls' bit for bit.  For groups of 32 labels on the fused path the
 * forward kernel also writes the transposed weights and lane-ordered supports the backward-feature
 * kernel reads, into the workspace, so that pass skips its own transposition of W.  dX NULL runs
 * haste_fwd_bce alone.  ws: haste_workspace_bytes(desc, HASTE_OP_TAIL_STEP) bytes (holds both
 * calls' workspaces side by side); too small gives HASTE_ERR_WORKSPACE and launches nothing.
 */
int haste_tail_step(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
                    const float *bias, const int32_t *pos, int32_t P, void *dY, float *dW,
                    float *dbias, int beta, float *dX, int beta_dx, void *ws, size_t ws_bytes,
                    void *stream);

/*
 * The same pass with the optimizer step (Section 4: SGD with momentum): haste_fwd_bce_sgd (dY, m,
 * W_next, dbias as documented there; dW never stored) followed by haste_bwd_x on its dY with the
 * step's W (not W_next), bit-identical to the two calls.  W_next must not overlap W.
 * ws: haste_workspace_bytes(desc, HASTE_OP_TAIL_STEP_SGD) bytes.
 */
int haste_tail_step_sgd(const haste_desc_t *desc, const void *X, const int32_t *idx, const void *W,
                        const float *bias, const int32_t *pos, int32_t P, void *dY, float *dbias,
                        const haste_sgd_t *opt, float *m, void *W_next, float *dX, int beta_dx,
                        void *ws, size_t ws_bytes, void *stream);

/* Bytes of workspace haste_group_labels needs (0 for invalid arguments). */
size_t haste_group_workspace_bytes(int64_t N, int64_t D, const haste_group_opts_t *opts);

/*
 * Gradient of the binary cross-entropy objective at stored logits (Section 3.3), for the dense
 * head or any [B, N] logit block:
 *   dY[b, n] = sigmoid(Y[b, n]) - T[b, n],  T from pos[B, P] as in haste_fwd_bce (ids in [0, N)).
 * Y and dY are [B, N] in dtype and may be the same buffer (in-place).  Arithmetic is fp32.
 */
int haste_bce_grad(int64_t B, int64_t N, int32_t dtype, const void *Y, const int32_t *pos,
                   int32_t P, void *dY, void *stream);

/*
 * Dense head forward (Section 3.3: a^H = W_head h_head):
 *   Y_h[b, h] = bias_h[h] + sum_f X[b, f] * W_head[h, f]
 * X[B, F_s], W_head[H, F_s] (dtype), bias_h[H] fp32 or NULL, Y_h[B, H] (dtype) overwritten.
 */
int haste_head_fwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X,
                   const void *W_head, const float *bias_h, void *Y_h, void *stream);

/*
 * Dense head forward fused with the gradient of the binary cross-entropy objective (Section 3.3,
 * head branch):
 *   dY_h[b, h] = sigmoid(bias_h[h] + sum_f X[b, f] * W_head[h, f]) - T[b, h]
 * with T from pos[B, P] as in haste_bce_grad (ids in [0, H); -1 padding and repeats allowed).
 * The logits are not stored.  On bf16 layers whose pointers are 16-byte aligned and whose F_s
 * and H are multiples of 8 the sigmoid is taken of the fp32 logit inside the GEMM's epilogue and
 * sigmoid - T is rounded once to bf16; otherwise the logits are written into dY_h (rounded to
 * dtype) and the gradient is formed there in place, as haste_head_fwd + haste_bce_grad would.
 * X[B, F_s], W_head[H, F_s] (dtype), bias_h[H] fp32 (16-byte aligned) or NULL, dY_h[B, H] (dtype)
 * overwritten.  Errors: HASTE_ERR_INVALID for a bad dtype, negative sizes or P, a NULL pointer
 * that is needed, or an unaligned bias_h; nothing is launched then.
 */
int haste_head_fwd_bce(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X,
                       const void *W_head, const float *bias_h, const int32_t *pos, int32_t P,
                       void *dY_h, void *stream);

/*
 * Dense head backward (Section 3.3 objective, head branch):
 *   dW_h[h, f] = sum_b dY_h[b, h] * X[b, f]                        (overwritten, fp32)
 *   dX[b, f]   = beta_dx * dX[b, f] + sum_h dY_h[b, h] * W_head[h, f]
 * beta_dx = 1 adds the head's input gradient onto an existing one (e.g. the tail's when both
 * branches read the same X).  dW_h or dX may be NULL to skip that product.  ws holds the
 * split-K partials of dX (haste_head_workspace_bytes).
 */
int haste_head_bwd(int64_t B, int64_t F_s, int64_t H, int32_t dtype, const void *X,
                   const void *W_head, const void *dY_h, float *dW_h, float *dX, int beta_dx,
                   void *ws, size_t ws_bytes, void *stream);

/* Bytes of workspace `op` (enum haste_op) needs for this layer; 0 if none.  Never fails; for an
 * invalid descriptor it returns 0 and the call itself reports the error. */
size_t haste_workspace_bytes(const haste_desc_t *desc, int op);

/* Bytes of workspace haste_head_bwd needs. */
size_t haste_head_workspace_bytes(int64_t B, int64_t F_s, int64_t H, int32_t dtype);

/*
 * Debug check of the idx precondition (Section 3.1: each group's support I_k is a set of exactly
 * F_in input features, a subset of the F_s features of h; stored sorted, a set is a strictly
 * increasing row): *n_bad_rows (device int32, overwritten) receives the number of rows of
 * idx[n_rows, F_in] that are not strictly increasing within [0, F_s).
 * n_rows = L/G (or L when G = 1).
 */
int haste_validate_idx(const haste_desc_t *desc, const int32_t *idx, int32_t *n_bad_rows,
                       void *stream);

/*
 * Debug export of the gather step (Section 3.2, H_k = h_{:, I_k}): for groups k in [k0, k0+nk)
 *   out[k - k0, b, t] = X[b, idx[k, t]]      out is [nk, B, F_in] in the dtype of X (bit copy).
 */
int haste_debug_gather(const haste_desc_t *desc, const void *X, const int32_t *idx, int64_t k0,
                       int64_t nk, void *out, void *stream);

/* Human-readable name of a status code (static storage). */
const char *haste_status_str(int status);

/* Message for the last error on the calling thread ("" if none). */
const char *haste_last_error(void);

/* Library version string. */
const char *haste_version(void);

#ifdef __cplusplus
}
#endif
#endif /* HASTE_H_ */
