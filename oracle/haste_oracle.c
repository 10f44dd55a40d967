/*
 * CPU oracle for the group-shared fixed fan-in (GS-FFI) output layer and its dense head.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously-correct statement of what
 * the GPU path computes.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  It shares no code, header, table or helper with the GPU library.
 *
 * Definitions (paper, Section 3.1 "Representation", Section 3.2 "Kernels", Section 3.3 Eq.
 * "head_tail_objective"):
 *   - labels are partitioned into K = L/G contiguous groups; label l belongs to group g(l) = l/G;
 *   - group k has one support I_k = idx[k, 0..F_in-1] (features of the input h);
 *   - label l keeps its own weights w_l = W[l, 0..F_in-1], slot t lives on feature idx[g(l), t];
 *   - logit   z_l(x) = <w_l, h_{I_g(l)}>                      (Section 3.1)
 *   - dW      grad W_k = (grad Z_k)^T H_k,  H_k = h_{:, I_k}     (Section 3.2, backward-weight)
 *   - dX      grad h_{:, I_k} += grad Z_k W_k, summed over k     (Section 3.2, backward-feature)
 *   - head    a^H = W_head h_head                                (Section 3.3)
 *   - BCE     d/dz of the binary cross-entropy of sigmoid(z)      (Section 3.3 objective)
 *   - SGD     momentum step of the classification layer's optimizer (Section 4)
 *   - rewire  group-shared rewiring of the supports (Alg. 3)
 *   - group   semantic grouping of labels (Alg. 2)
 *
 * Arithmetic: inputs are decoded exactly to double (bf16 -> fp64 and fp32 -> fp64 are exact);
 * every sum is accumulated in double in the order the definition states (no blocking, no
 * reordering).  Outputs are fp64 and are never rounded to the GPU's storage types.
 *
 * Parity pins: see the tests (brute-force dense zero-masked matrix, worked Fig. 2 instances,
 * special cases, finite differences, adjoint identity, one-hot gathers).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define DT_F32 0
#define DT_BF16 1

/* element i of a stored buffer, decoded exactly */
static double ld(const void *p, int64_t i, int dtype) {
    if (dtype == DT_BF16) {
        uint32_t u = ((uint32_t)((const uint16_t *)p)[i]) << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return (double)((const float *)p)[i];
}

static int bad_layer(int64_t B, int64_t F_s, int64_t L, int64_t G, int64_t F_in, int dtype) {
    if (B < 0 || F_s <= 0 || L < 0 || G <= 0 || F_in <= 0) return 1;
    if (L % G != 0) return 1;
    if (dtype != DT_F32 && dtype != DT_BF16) return 1;
    return 0;
}

int haste_oracle_num_threads(void) { return omp_get_max_threads(); }

/* ---------------------------------------------------------------------------------------------
 * Tail forward (Section 3.1):  Y[b, l] = bias[l] + sum_t X[b, idx[g(l), t]] * W[l, t]
 * for labels l in [l0, l1) and all rows b; Y is [B, l1-l0] row-major.
 * ------------------------------------------------------------------------------------------- */
int haste_oracle_fwd(int64_t B, int64_t F_s, int64_t L, int64_t G, int64_t F_in, int dtype,
                     const void *X, const int32_t *idx, const void *W, const float *bias,
                     int64_t l0, int64_t l1, double *Y) {
    if (bad_layer(B, F_s, L, G, F_in, dtype) || l0 < 0 || l1 > L || l0 > l1) return 1;
    const int64_t n = l1 - l0;
#pragma omp parallel for schedule(static)
    for (int64_t l = l0; l < l1; ++l) {
        const int64_t g = l / G;                 /* g(l): labels of a group are contiguous */
        for (int64_t b = 0; b < B; ++b) {
            double z = bias ? (double)bias[l] : 0.0;
            for (int64_t t = 0; t < F_in; ++t) {
                const int64_t f = idx[g * F_in + t];
                z += ld(X, b * F_s + f, dtype) * ld(W, l * F_in + t, dtype);
            }
            Y[b * n + (l - l0)] = z;
        }
    }
    return 0;
}

/* Forward logits at explicit (b, l) sample points. */
int haste_oracle_fwd_at(int64_t B, int64_t F_s, int64_t L, int64_t G, int64_t F_in, int dtype,
                        const void *X, const int32_t *idx, const void *W, const float *bias,
                        int64_t n, const int64_t *bs, const int64_t *ls, double *out) {
    if (bad_layer(B, F_s, L, G, F_in, dtype)) return 1;
    for (int64_t i = 0; i < n; ++i)
        if (bs[i] < 0 || bs[i] >= B || ls[i] < 0 || ls[i] >= L) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const int64_t b = bs[i], l = ls[i], g = l / G;
        double z = bias ? (double)bias[l] : 0.0;
        for (int64_t t = 0; t < F_in; ++t)
            z += ld(X, b * F_s + idx[g * F_in + t], dtype) * ld(W, l * F_in + t, dtype);
        out[i] = z;
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Tail backward-weight (Section 3.2):  dW[l, t] = sum_b dY[b, l] * X[b, idx[g(l), t]]
 * only on the F_in support slots; dbias[l] = sum_b dY[b, l].  Labels in [l0, l1).
 * dW is [l1-l0, F_in], dbias is [l1-l0] (may be NULL).
 * ------------------------------------------------------------------------------------------- */
int haste_oracle_bwd_w(int64_t B, int64_t F_s, int64_t L, int64_t G, int64_t F_in, int dtype,
                       const void *X, const int32_t *idx, const void *dY,
                       int64_t l0, int64_t l1, double *dW, double *dbias) {
    if (bad_layer(B, F_s, L, G, F_in, dtype) || l0 < 0 || l1 > L || l0 > l1) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t l = l0; l < l1; ++l) {
        const int64_t g = l / G;
        for (int64_t t = 0; t < F_in; ++t) {
            const int64_t f = idx[g * F_in + t];
            double s = 0.0;
            for (int64_t b = 0; b < B; ++b)
                s += ld(dY, b * L + l, dtype) * ld(X, b * F_s + f, dtype);
            dW[(l - l0) * F_in + t] = s;
        }
        if (dbias) {
            double s = 0.0;
            for (int64_t b = 0; b < B; ++b) s += ld(dY, b * L + l, dtype);
            dbias[l - l0] = s;
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Tail backward-feature (Section 3.2):
 *   dX[b, f] = sum_k sum_{t : idx[k,t] = f} sum_{j < G} dY[b, kG + j] * W[kG + j, t]
 * written as a per-row scatter over labels: every label's contribution is added to the feature
 * its slot lives on.  Rows b in [b0, b1); dX is [b1-b0, F_s] (overwritten).
 * ------------------------------------------------------------------------------------------- */
int haste_oracle_bwd_x(int64_t B, int64_t F_s, int64_t L, int64_t G, int64_t F_in, int dtype,
                       const int32_t *idx, const void *W, const void *dY,
                       int64_t b0, int64_t b1, double *dX) {
    if (bad_layer(B, F_s, L, G, F_in, dtype) || b0 < 0 || b1 > B || b0 > b1) return 1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = b0; b < b1; ++b) {
        double *row = dX + (b - b0) * F_s;
        for (int64_t f = 0; f < F_s; ++f) row[f] = 0.0;
        for (int64_t l = 0; l < L; ++l) {
            const double d = ld(dY, b * L + l, dtype);
            const int64_t g = l / G;
            for (int64_t t = 0; t < F_in; ++t)
                row[idx[g * F_in + t]] += d * ld(W, l * F_in + t, dtype);
        }
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Dense head (Section 3.3):  Yh[b, h] = bias_h[h] + sum_f X[b, f] * Wh[h, f], heads in [h0, h1).
 * Yh is [B, h1-h0].
 * ------------------------------------------------------------------------------------------- */
int haste_oracle_head_fwd(int64_t B, int64_t F_s, int64_t H, int dtype, const void *X,
                          const void *Wh, const float *bias_h, int64_t h0, int64_t h1, double *Yh) {
    if (B < 0 || F_s <= 0 || H < 0 || h0 < 0 || h1 > H || h0 > h1) return 1;
    if (dtype != DT_F32 && dtype != DT_BF16) return 1;
    const int64_t n = h1 - h0;
#pragma omp parallel for schedule(static)
    for (int64_t h = h0; h < h1; ++h)
        for (int64_t b = 0; b < B; ++b) {
            double z = bias_h ? (double)bias_h[h] : 0.0;
            for (int64_t f = 0; f < F_s; ++f) z += ld(X, b * F_s + f, dtype) * ld(Wh, h * F_s + f, dtype);
            Yh[b * n + (h - h0)] = z;
        }
    return 0;
}

/* dWh[h, f] = sum_b dYh[b, h] * X[b, f] for heads in [h0, h1); dWh is [h1-h0, F_s]. */
int haste_oracle_head_bwd_w(int64_t B, int64_t F_s, int64_t H, int dtype, const void *X,
                            const void *dYh, int64_t h0, int64_t h1, double *dWh) {
    if (B < 0 || F_s <= 0 || H < 0 || h0 < 0 || h1 > H || h0 > h1) return 1;
    if (dtype != DT_F32 && dtype != DT_BF16) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t h = h0; h < h1; ++h)
        for (int64_t f = 0; f < F_s; ++f) {
            double s = 0.0;
            for (int64_t b = 0; b < B; ++b) s += ld(dYh, b * H + h, dtype) * ld(X, b * F_s + f, dtype);
            dWh[(h - h0) * F_s + f] = s;
        }
    return 0;
}

/* dXh[b, f] = sum_h dYh[b, h] * Wh[h, f] for rows in [b0, b1); dXh is [b1-b0, F_s]. */
int haste_oracle_head_bwd_x(int64_t B, int64_t F_s, int64_t H, int dtype, const void *Wh,
                            const void *dYh, int64_t b0, int64_t b1, double *dXh) {
    if (B < 0 || F_s <= 0 || H < 0 || b0 < 0 || b1 > B || b0 > b1) return 1;
    if (dtype != DT_F32 && dtype != DT_BF16) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t b = b0; b < b1; ++b)
        for (int64_t f = 0; f < F_s; ++f) {
            double s = 0.0;
            for (int64_t h = 0; h < H; ++h) s += ld(dYh, b * H + h, dtype) * ld(Wh, h * F_s + f, dtype);
            dXh[(b - b0) * F_s + f] = s;
        }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Gradient of the binary cross-entropy objective with respect to the logits (Section 3.3: the
 * objective sums the BCE of sigmoid(z) against the 0/1 targets over labels; its derivative in z
 * is sigmoid(z) - y):
 *   dY[b, n] = 1 / (1 + exp(-Z[b, n])) - T[b, n]
 *   T[b, n]  = 1 if n occurs among pos[b, 0..P-1], else 0
 * Entries of pos outside [0, N) (e.g. -1 padding) are ignored; a repeated entry counts once (the
 * target is set, not added).  Z and dY are [B, N] row-major doubles.
 * ------------------------------------------------------------------------------------------- */
static double sigmoid(double z) { return 1.0 / (1.0 + exp(-z)); }

int haste_oracle_bce_grad(int64_t B, int64_t N, const double *Z, const int32_t *pos, int64_t P, double *dY) {
    if (B < 0 || N < 0 || P < 0) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < B; ++b) {
        for (int64_t n = 0; n < N; ++n) dY[b * N + n] = sigmoid(Z[b * N + n]);
        for (int64_t p = 0; p < P; ++p) {
            const int64_t c = pos[b * P + p];
            if (c >= 0 && c < N) dY[b * N + c] = sigmoid(Z[b * N + c]) - 1.0;
        }
    }
    return 0;
}

/* The same gradient at explicit (b, n) points: z[i] is the logit of (bs[i], ns[i]). */
int haste_oracle_bce_grad_at(int64_t B, int64_t N, const int32_t *pos, int64_t P, int64_t n, const int64_t *bs,
                             const int64_t *ns, const double *z, double *out) {
    if (B < 0 || N < 0 || P < 0) return 1;
    for (int64_t i = 0; i < n; ++i)
        if (bs[i] < 0 || bs[i] >= B || ns[i] < 0 || ns[i] >= N) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double y = 0.0;
        for (int64_t p = 0; p < P; ++p)
            if (pos[bs[i] * P + p] == ns[i]) y = 1.0;
        out[i] = sigmoid(z[i]) - y;
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * SGD with momentum, the optimizer the paper trains the classification layer with (Section 4,
 * implementation details), in the common form without dampening or look-ahead:
 *   velocity  m <- momentum * m + (grad + weight_decay * W)
 *   weights   W_next = W - lr * m
 * W is read in its storage dtype; grad, m (in/out) and W_next are doubles.
 * ------------------------------------------------------------------------------------------- */
int haste_oracle_sgd_momentum(int64_t n, int dtype, const void *W, const double *grad, double *m, double lr,
                              double momentum, double weight_decay, double *W_next) {
    if (n < 0 || (dtype != DT_F32 && dtype != DT_BF16)) return 1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        const double w = ld(W, i, dtype);
        m[i] = momentum * m[i] + (grad[i] + weight_decay * w);
        W_next[i] = w - lr * m[i];
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Group-shared rewiring (Alg. 3, the discrete phase of the alternating training loop in Section 3.3):
 *   1. score every (group k, slot j) by the |w| of the group's labels at that slot;
 *   2. mark the m = floor(K F rho) smallest scores over all groups;
 *   3. give each marked slot a new feature;
 *   4. reinitialise the marked slots' weights (zero, or uniform in [-1/sqrt(F), 1/sqrt(F)]).
 * Readings where the algorithm is silent or leaves the layout's invariants open:
 *   - the score is the sum over the G labels, accumulated in fp32 in label order (the mean of the
 *     algorithm divides every score by the same G, which orders them identically); both this and
 *     the GPU take the selection decision in that fp32 arithmetic;
 *   - ties in the selection go to the lower flat index k F + j;
 *   - a marked slot draws its feature uniformly from those not kept by its group and not drawn
 *     before it (slots in ascending j), so every support stays a set; the row is then re-sorted,
 *     carrying each slot's weight column (and velocity) with it;
 *   - randomness: SplitMix64 (Steele, Lea and Flood, 2014) in counter form, output i of the stream
 *     seeded with `seed`: draw r = out(k F + j) picks the (r mod n_free)-th free feature in
 *     ascending order; label l's reinitialised slot j takes n = out(K F + l F + j) >> 40 (24 bits)
 *     and the value ((2 n - 2^24) as fp32) * (a 2^-24), a = fp32(1 / sqrt(F)), stored in the
 *     weights' dtype (bf16 rounded to nearest even);
 *   - a velocity array, if given, moves with its weights and is zero on reinitialised slots.
 * idx [K, F] (strictly increasing rows, in/out), W [K G, F] in its storage dtype (in/out), m
 * [K G, F] doubles or NULL (in/out); mask [K F] receives the marked slots by their old position.
 * ------------------------------------------------------------------------------------------- */
static uint64_t splitmix64_at(uint64_t s, uint64_t i) {
    uint64_t z = s + (i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

uint64_t haste_oracle_splitmix64(uint64_t seed, uint64_t i) { return splitmix64_at(seed, i); }

static uint16_t bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

typedef struct { float s; int64_t i; } score_t;

static int by_score(const void *a, const void *b) {
    const score_t *x = (const score_t *)a, *y = (const score_t *)b;
    if (x->s < y->s) return -1;
    if (x->s > y->s) return 1;
    return (x->i > y->i) - (x->i < y->i);
}

typedef struct { int32_t f; int32_t src; } slot_t;

static int by_feature(const void *a, const void *b) {
    const slot_t *x = (const slot_t *)a, *y = (const slot_t *)b;
    return (x->f > y->f) - (x->f < y->f);
}

int haste_oracle_rewire(int64_t K, int64_t G, int64_t F, int64_t H, int dtype, int32_t *idx, void *W, double *m,
                        double rho, int init_random, uint64_t seed, int64_t *n_pruned, uint8_t *mask) {
    if (K < 0 || G <= 0 || F <= 0 || H < F || rho < 0.0 || rho >= 1.0) return 1;
    if (dtype != DT_F32 && dtype != DT_BF16) return 1;
    const int64_t KF = K * F;
    const int64_t npr = (int64_t)floor((double)K * (double)F * rho);
    *n_pruned = npr;
    memset(mask, 0, (size_t)KF);
    if (npr == 0) return 0;
    /* 1. scores, fp32, labels in order */
    score_t *sc = (score_t *)malloc((size_t)KF * sizeof(score_t));
    if (!sc) return 2;
    for (int64_t k = 0; k < K; ++k)
        for (int64_t j = 0; j < F; ++j) {
            float s = 0.0f;
            for (int64_t g = 0; g < G; ++g) s += fabsf((float)ld(W, (k * G + g) * F + j, dtype));
            sc[k * F + j].s = s;
            sc[k * F + j].i = k * F + j;
        }
    /* 2. the npr smallest, ties to the lower index */
    qsort(sc, (size_t)KF, sizeof(score_t), by_score);
    for (int64_t r = 0; r < npr; ++r) mask[sc[r].i] = 1;
    free(sc);
    /* 3-4. per group: draws, re-sort, weights */
    const float a = (float)(1.0 / sqrt((double)F));
    const float scale = a * 5.9604644775390625e-08f; /* a * 2^-24, exact */
    uint8_t *used = (uint8_t *)malloc((size_t)H);
    slot_t *row = (slot_t *)malloc((size_t)F * sizeof(slot_t));
    double *tmp = (double *)malloc((size_t)F * sizeof(double));
    if (!used || !row || !tmp) { free(used); free(row); free(tmp); return 2; }
    for (int64_t k = 0; k < K; ++k) {
        int any = 0;
        for (int64_t j = 0; j < F; ++j) any |= mask[k * F + j];
        if (!any) continue;
        memset(used, 0, (size_t)H);
        int64_t n_used = 0;
        for (int64_t j = 0; j < F; ++j)
            if (!mask[k * F + j]) { used[idx[k * F + j]] = 1; ++n_used; }
        for (int64_t j = 0; j < F; ++j) {
            int32_t f = idx[k * F + j];
            if (mask[k * F + j]) {
                const int64_t t = (int64_t)(splitmix64_at(seed, (uint64_t)(k * F + j)) % (uint64_t)(H - n_used));
                int64_t c = -1;
                for (f = 0; f < H; ++f)
                    if (!used[f] && ++c == t) break;
                used[f] = 1;
                ++n_used;
            }
            row[j].f = f;
            row[j].src = (int32_t)j;
        }
        qsort(row, (size_t)F, sizeof(slot_t), by_feature);
        for (int64_t p = 0; p < F; ++p) idx[k * F + p] = row[p].f;
        for (int64_t g = 0; g < G; ++g) {
            const int64_t l = k * G + g;
            for (int64_t p = 0; p < F; ++p) {
                const int64_t j = row[p].src;
                if (mask[k * F + j]) {
                    double v = 0.0;
                    if (init_random) {
                        const uint64_t n = splitmix64_at(seed, (uint64_t)(KF + l * F + j)) >> 40;
                        v = (double)((float)((int64_t)(2 * n) - (1LL << 24)) * scale);
                    }
                    tmp[p] = v;
                } else {
                    tmp[p] = ld(W, l * F + j, dtype);
                }
            }
            for (int64_t p = 0; p < F; ++p) {
                if (dtype == DT_BF16) ((uint16_t *)W)[l * F + p] = bf16_rne((float)tmp[p]);
                else ((float *)W)[l * F + p] = (float)tmp[p];
            }
            if (m) {
                for (int64_t p = 0; p < F; ++p) tmp[p] = mask[k * F + row[p].src] ? 0.0 : m[l * F + row[p].src];
                for (int64_t p = 0; p < F; ++p) m[l * F + p] = tmp[p];
            }
        }
    }
    free(used); free(row); free(tmp);
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Semantic label grouping (Alg. 2): coarse spherical k-means into C = max(1, floor(N / (beta G)))
 * clusters, then, inside each cluster, greedy groups: a random unassigned seed together with its
 * top-(G - 1) unassigned neighbours by cosine similarity (Section 3.1, "Label Grouping").
 * Readings:
 *   - embeddings are stored as int8 (unit vectors x 127, rounded); similarity is the cosine of the
 *     stored vectors, cos(u, v) = u.v / (|u| |v|) (Eq. grouping-objective's sim);
 *   - spherical k-means: a centre is the normalised mean of its members, i.e. the direction of
 *     their sum s (an exact integer vector).  The cosine of e with that centre is e.s / (|e| |s|);
 *     |e| is the same for every centre and does not change the argmax, so a label goes to the
 *     centre maximising e.s / |s|.  e.s is an exact integer, |s|^2 an exact integer rounded once to
 *     double, and the quotient takes one correctly rounded square root and one correctly rounded
 *     division in fp64: the decision is taken in fp64 on the exact inputs.  Ties go to the lower
 *     centre.  Initial centres are single labels (s = e); an empty cluster, or one whose members
 *     sum to zero, keeps its centre;
 *   - k-means runs `iters` full Lloyd iterations (assign every label, then move every centre),
 *     then a final assignment; the paper's mini-batch variant is a CPU economy;
 *   - the greedy stage: the seed always belongs to its own group; the other k - 1 members are the
 *     unassigned labels of largest cos(e_i, e_s) = (e_i.e_s) / sqrt(|e_i|^2 |e_s|^2), formed in
 *     fp64 the same way (|e_i|^2 |e_s|^2 < 2^53 is exact), ties to the lower label;
 *   - initial centres: the first C entries of a partial Fisher-Yates shuffle of [0, N) whose i-th
 *     swap partner is i + out(i) mod (N - i); the t-th seed of cluster c is the
 *     (out(N + c N + t) mod n_unassigned)-th unassigned member in ascending label order
 *     (out = SplitMix64 in counter form, as for rewiring);
 *   - a group lists its labels in ascending order; groups are emitted cluster by cluster, in the
 *     order they are formed.
 * E [N, D] int8; order [N] receives the labels group after group, gsize the group sizes,
 * *n_groups their count, cluster [N] (or NULL) the final cluster of each label.
 * ------------------------------------------------------------------------------------------- */
static int64_t dot8(const int8_t *a, const int8_t *b, int64_t D) {
    int64_t s = 0;
    for (int64_t d = 0; d < D; ++d) s += (int64_t)a[d] * (int64_t)b[d];
    return s;
}

/* |s| of an integer vector: the exact sum of squares (128-bit), rounded once to double, then a
 * correctly rounded square root */
static double exact_norm(const int64_t *s, int64_t D) {
    unsigned __int128 q = 0;
    for (int64_t d = 0; d < D; ++d) q += (unsigned __int128)((__int128)s[d] * (__int128)s[d]);
    return sqrt((double)q);
}

static void assign_all(int64_t N, int64_t D, int64_t C, const int8_t *E, const int64_t *cs, const double *cn,
                       int32_t *cl) {
#pragma omp parallel for schedule(static)
    for (int64_t l = 0; l < N; ++l) {
        int64_t best = -1;
        double bv = 0.0;
        for (int64_t c = 0; c < C; ++c) {
            int64_t dot = 0;
            for (int64_t d = 0; d < D; ++d) dot += (int64_t)E[l * D + d] * cs[c * D + d];
            const double v = (double)dot / cn[c];
            if (best < 0 || v > bv) { bv = v; best = c; }
        }
        cl[l] = (int32_t)best;
    }
}

typedef struct { double sim; int32_t id; } cand_t;

static int by_sim(const void *a, const void *b) {
    const cand_t *x = (const cand_t *)a, *y = (const cand_t *)b;
    if (x->sim != y->sim) return x->sim > y->sim ? -1 : 1;
    return (x->id > y->id) - (x->id < y->id);
}

static int by_id(const void *a, const void *b) {
    const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

int haste_oracle_group_labels(int64_t N, int64_t D, const int8_t *E, int64_t G, int64_t beta, int64_t iters,
                              uint64_t seed, int32_t *order, int32_t *gsize, int64_t *n_groups, int32_t *cluster) {
    if (N <= 0 || D <= 0 || G <= 0 || beta <= 0 || iters < 0) return 1;
    int64_t C = N / (beta * G);
    if (C < 1) C = 1;
    int32_t *a = (int32_t *)malloc((size_t)N * sizeof(int32_t));
    int64_t *cs = (int64_t *)malloc((size_t)(C * D) * sizeof(int64_t));   /* centre directions (sums) */
    double *cn = (double *)malloc((size_t)C * sizeof(double));            /* their norms */
    int32_t *cl = (int32_t *)malloc((size_t)N * sizeof(int32_t));
    int64_t *sum = (int64_t *)malloc((size_t)D * sizeof(int64_t));
    cand_t *cand = (cand_t *)malloc((size_t)N * sizeof(cand_t));
    if (!a || !cs || !cn || !cl || !sum || !cand) {
        free(a); free(cs); free(cn); free(cl); free(sum); free(cand);
        return 2;
    }
    for (int64_t i = 0; i < N; ++i) a[i] = (int32_t)i;
    for (int64_t i = 0; i < C; ++i) {
        const int64_t j = i + (int64_t)(splitmix64_at(seed, (uint64_t)i) % (uint64_t)(N - i));
        const int32_t t = a[i]; a[i] = a[j]; a[j] = t;
        for (int64_t d = 0; d < D; ++d) cs[i * D + d] = E[(int64_t)a[i] * D + d];
        cn[i] = exact_norm(cs + i * D, D);
    }
    for (int64_t it = 0; it < iters; ++it) {
        assign_all(N, D, C, E, cs, cn, cl);
        for (int64_t c = 0; c < C; ++c) {
            memset(sum, 0, (size_t)D * sizeof(int64_t));
            int64_t cnt = 0;
            for (int64_t l = 0; l < N; ++l)
                if (cl[l] == c) { ++cnt; for (int64_t d = 0; d < D; ++d) sum[d] += E[l * D + d]; }
            const double nrm = exact_norm(sum, D);
            if (cnt == 0 || nrm == 0.0) continue;   /* the centre stays where it was */
            memcpy(cs + c * D, sum, (size_t)D * sizeof(int64_t));
            cn[c] = nrm;
        }
    }
    assign_all(N, D, C, E, cs, cn, cl);
    if (cluster) memcpy(cluster, cl, (size_t)N * sizeof(int32_t));
    int64_t pos = 0, ng = 0;
    for (int64_t c = 0; c < C; ++c) {
        int64_t nu = 0;   /* unassigned members, ascending */
        for (int64_t l = 0; l < N; ++l)
            if (cl[l] == c) a[nu++] = (int32_t)l;
        for (int64_t t = 0; nu > 0; ++t) {
            const int64_t r = (int64_t)(splitmix64_at(seed, (uint64_t)(N + c * N + t)) % (uint64_t)nu);
            const int32_t s = a[r];
            const int64_t ns = dot8(E + (int64_t)s * D, E + (int64_t)s * D, D);
            int64_t nc = 0;   /* the other unassigned members, by cosine to the seed */
            for (int64_t i = 0; i < nu; ++i) {
                if (i == r) continue;
                const int8_t *e = E + (int64_t)a[i] * D;
                const int64_t ni = dot8(e, e, D);
                cand[nc].sim = (double)dot8(e, E + (int64_t)s * D, D) / sqrt((double)(ni * ns));
                cand[nc].id = a[i];
                ++nc;
            }
            qsort(cand, (size_t)nc, sizeof(cand_t), by_sim);
            const int64_t k = nu < G ? nu : G;
            order[pos] = s;
            for (int64_t i = 0; i + 1 < k; ++i) order[pos + 1 + i] = cand[i].id;
            qsort(order + pos, (size_t)k, sizeof(int32_t), by_id);
            gsize[ng++] = (int32_t)k;
            pos += k;
            /* the rest stay unassigned, ascending */
            int64_t rr = 0;
            for (int64_t i = k - 1; i < nc; ++i) a[rr++] = cand[i].id;
            qsort(a, (size_t)rr, sizeof(int32_t), by_id);
            nu = rr;
        }
    }
    *n_groups = ng;
    free(a); free(cs); free(cn); free(cl); free(sum); free(cand);
    return 0;
}
