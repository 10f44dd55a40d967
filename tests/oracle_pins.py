"""Pins of the CPU oracle against facts fixed outside the oracle itself.

Every ``pin_*`` takes an oracle object (the real one, or a build with a planted mistake) and
raises AssertionError when the oracle disagrees with:

* the paper's worked instances of the two index formats (Figure 2(c) and 2(d));
* a brute-force dense layer whose full weight matrix is zero outside each group's support
  (the sparse layer of Section 3.1 is exactly that matrix), evaluated with ``np.matmul``;
* special cases with textbook answers (F_in = F_s with identity supports is a dense layer;
  G = 1 is standard per-label fixed fan-in; G = L is one gathered GEMM);
* finite differences of the Section 3.3 BCE objective and of the bilinear pairing, and of the
  objective with respect to the logits for the BCE-gradient function;
* closed forms of the momentum step (constant gradient, weight decay alone) and its convergence on a
  quadratic;
* the rewiring of Alg. 3 on a hand-checked layer, its tie rule, its invariants on random layers,
  the uniformity of its draws, and the published outputs of its generator;
* the grouping of Alg. 2 on planted directions (exact groups) and planted clusters (recovered),
  against its brute-force statement with NumPy cosines, and its seed rule on near-duplicates;
* the moments and bins of rewiring's random reinitialisation (Alg. 3's uniform law);
* the adjoint identity <dY, Y - bias> = <dX, X> = <dW, W> (bilinearity);
* exact one-hot gathers/scatters and the group-permutation invariance.
"""
from __future__ import annotations

import json
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
F32, BF16 = synth.DT_F32, synth.DT_BF16


# ------------------------------------------------------------------------------------------
# independent helpers (NumPy only)
# ------------------------------------------------------------------------------------------
def dense_masked(idx, W, G, F_s):
    """W_full[L, F_s]: W_full[l, idx[l//G, t]] += W[l, t]; zero elsewhere (duplicates add)."""
    W = np.asarray(W, dtype=np.float64)
    L, F_in = W.shape
    Wf = np.zeros((L, F_s), dtype=np.float64)
    rows = np.repeat(np.arange(L), F_in)
    cols = idx[np.arange(L) // G].reshape(-1)
    np.add.at(Wf, (rows, cols), W.reshape(-1))
    return Wf


def rand_layer(rng, B, F_s, L, G, F_in, dtype, distinct=True, bias=True):
    X = rng.standard_normal((B, F_s)).astype(np.float32)
    W = (rng.standard_normal((L, F_in)) / np.sqrt(F_in)).astype(np.float32)
    dY = rng.standard_normal((B, L)).astype(np.float32)
    K = L // G
    if distinct:
        idx = np.stack([np.sort(rng.choice(F_s, F_in, replace=False)) for _ in range(K)]).astype(np.int32)
    else:
        idx = rng.integers(0, F_s, size=(K, F_in)).astype(np.int32)
    b = rng.standard_normal(L).astype(np.float32) if bias else None
    if dtype == BF16:
        X, W, dY = synth.bf16_bits(X), synth.bf16_bits(W), synth.bf16_bits(dY)
    return X, idx, W, b, dY


def f64(a, dtype):
    return synth.to_f64(a, dtype)


def close(a, b, rtol=1e-12, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    scale = max(1.0, float(np.abs(b).max()) if b.size else 1.0)
    err = float(np.abs(a - b).max()) if a.size else 0.0
    assert err <= rtol * scale, f"{what}: max abs err {err:.3e} > {rtol:.1e} * {scale:.3e}"


def _load_fig2():
    with open(os.path.join(GOLDEN, "fig2_formats.json")) as fh:
        return json.load(fh)


def _grid(panel, n_labels, n_features):
    # drawn values rounded to the fp32 storage type the layer holds them in
    D = np.zeros((n_labels, n_features))
    for l, f, v in panel["grid"]:
        D[l, f] = float(np.float32(v))
    return D


# ------------------------------------------------------------------------------------------
# pins
# ------------------------------------------------------------------------------------------
def pin_fig2_gs(o):
    """Figure 2(d): supports {0,2} and {1,3} for groups of 3 labels; logits with X = I are the grid."""
    g = _load_fig2()
    p = g["gs"]
    nl, nf, G = g["n_labels"], g["n_features"], p["group_size"]
    idx = np.array(p["index_rows_slot_major"], dtype=np.int32).T.copy()   # [K, F]
    W = np.array(p["weight_rows_slot_major"], dtype=np.float32).T.copy()  # [L, F]
    D = _grid(p, nl, nf)
    close(dense_masked(idx, W, G, nf), D, 0, "fig2(d) decode")
    # forward with one-hot rows: Y[f, l] = W_full[l, f]
    Y = o.fwd(np.eye(nf, dtype=np.float32), idx, W, None, G, F32)
    close(Y, D.T, 0, "fig2(d) fwd")
    # backward-feature with one-hot upstream rows: dX[l, f] = W_full[l, f]
    dX = o.bwd_x(idx, W, np.eye(nl, dtype=np.float32), G, nf, F32)
    close(dX, D, 0, "fig2(d) bwd_x")
    # backward-weight with X = I and dY = grid^T returns each label's own weights
    dW, _ = o.bwd_w(np.eye(nf, dtype=np.float32), idx, D.T.astype(np.float32), G, idx.shape[1], F32)
    close(dW, W, 0, "fig2(d) bwd_w")


def pin_fig2_ffi(o):
    """Figure 2(c): per-label supports (G = 1) decode to the drawn grid."""
    g = _load_fig2()
    p = g["ffi"]
    nl, nf = g["n_labels"], g["n_features"]
    idx = np.array(p["index_rows_slot_major"], dtype=np.int32).T.copy()   # [L, F]
    W = np.array(p["weight_rows_slot_major"], dtype=np.float32).T.copy()
    D = _grid(p, nl, nf)
    close(dense_masked(idx, W, 1, nf), D, 0, "fig2(c) decode")
    close(o.fwd(np.eye(nf, dtype=np.float32), idx, W, None, 1, F32), D.T, 0, "fig2(c) fwd")
    close(o.bwd_x(idx, W, np.eye(nl, dtype=np.float32), 1, nf, F32), D, 0, "fig2(c) bwd_x")


_SHAPES = [
    # B, F_s, L, G, F_in
    (5, 17, 24, 4, 3),
    (7, 40, 48, 8, 6),
    (3, 9, 6, 1, 4),       # G = 1 (per-label fixed fan-in)
    (4, 12, 10, 10, 5),    # G = L (one group)
    (6, 16, 32, 4, 16),    # F_in = F_s
    (1, 33, 64, 16, 7),    # single row
]


def pin_bruteforce(o):
    """fwd, dW, dbias, dX equal the dense zero-masked layer (np.matmul, fp64)."""
    rng = np.random.default_rng(1234)
    for dtype in (F32, BF16):
        for (B, F_s, L, G, F_in) in _SHAPES:
            X, idx, W, b, dY = rand_layer(rng, B, F_s, L, G, F_in, dtype)
            Wf = dense_masked(idx, f64(W, dtype), G, F_s)
            Xd, dYd = f64(X, dtype), f64(dY, dtype)
            Y = o.fwd(X, idx, W, b, G, dtype)
            close(Y, Xd @ Wf.T + b.astype(np.float64), 1e-12, f"fwd {B,F_s,L,G,F_in}")
            dW, db = o.bwd_w(X, idx, dY, G, F_in, dtype, with_dbias=True)
            full = dYd.T @ Xd                                  # dense gradient [L, F_s]
            close(dW, full[np.arange(L)[:, None], idx[np.arange(L) // G]], 1e-12, "bwd_w")
            close(db, dYd.sum(0), 1e-12, "dbias")
            close(o.bwd_x(idx, W, dY, G, F_s, dtype), dYd @ Wf, 1e-12, "bwd_x")


def pin_duplicate_indices(o):
    """A support with repeated features still equals the masked matrix (contributions add)."""
    rng = np.random.default_rng(7)
    X, idx, W, b, dY = rand_layer(rng, 4, 5, 12, 3, 6, F32, distinct=False)
    Wf = dense_masked(idx, W, 3, 5)
    close(o.fwd(X, idx, W, b, 3, F32), X.astype(np.float64) @ Wf.T + b, 1e-12, "dup fwd")
    close(o.bwd_x(idx, W, dY, 3, 5, F32), dY.astype(np.float64) @ Wf, 1e-12, "dup bwd_x")


def pin_dense_special_case(o):
    """F_in = F_s with idx[k] = 0..F_s-1 is the dense layer Y = X W^T."""
    rng = np.random.default_rng(3)
    B, F_s, L, G = 6, 10, 14, 7
    X = rng.standard_normal((B, F_s)).astype(np.float32)
    W = rng.standard_normal((L, F_s)).astype(np.float32)
    dY = rng.standard_normal((B, L)).astype(np.float32)
    idx = np.tile(np.arange(F_s, dtype=np.int32), (L // G, 1))
    Xd, Wd, dYd = X.astype(np.float64), W.astype(np.float64), dY.astype(np.float64)
    close(o.fwd(X, idx, W, None, G, F32), Xd @ Wd.T, 1e-12, "dense fwd")
    close(o.bwd_w(X, idx, dY, G, F_s, F32)[0], dYd.T @ Xd, 1e-12, "dense dW")
    close(o.bwd_x(idx, W, dY, G, F_s, F32), dYd @ Wd, 1e-12, "dense dX")


def pin_group_equals_expanded_ffi(o):
    """GS with (idx, G) equals standard fixed fan-in with idx_ffi[l] = idx[l // G] (G = 1)."""
    rng = np.random.default_rng(11)
    B, F_s, L, G, F_in = 5, 30, 40, 8, 5
    X, idx, W, b, dY = rand_layer(rng, B, F_s, L, G, F_in, F32)
    idx1 = idx[np.arange(L) // G]
    close(o.fwd(X, idx, W, b, G, F32), o.fwd(X, idx1, W, b, 1, F32), 0, "G vs FFI fwd")
    close(o.bwd_w(X, idx, dY, G, F_in, F32)[0], o.bwd_w(X, idx1, dY, 1, F_in, F32)[0], 0, "G vs FFI dW")
    close(o.bwd_x(idx, W, dY, G, F_s, F32), o.bwd_x(idx1, W, dY, 1, F_s, F32), 1e-14, "G vs FFI dX")


def _bce(Y, T):
    # sum of binary cross-entropies of sigmoid(Y) against targets T (Section 3.3 objective, unscaled)
    return float(np.sum(np.logaddexp(0.0, Y) - T * Y))


def pin_finite_differences(o):
    """Central differences of the BCE objective and of <dY, Y> match dX and dW."""
    rng = np.random.default_rng(5)
    B, F_s, L, G, F_in = 4, 12, 16, 4, 5
    X, idx, W, b, _ = rand_layer(rng, B, F_s, L, G, F_in, F32)
    T = (rng.random((B, L)) < 0.2).astype(np.float64)
    Y = o.fwd(X, idx, W, b, G, F32)
    dY = (1.0 / (1.0 + np.exp(-Y)) - T).astype(np.float32)        # BCE gradient, fp32 upstream
    # with dY rounded to fp32 the exact derivative of phi(X, W) = <dY, Y> is what we compare
    dX = o.bwd_x(idx, W, dY, G, F_s, F32)
    dW, _ = o.bwd_w(X, idx, dY, G, F_in, F32)
    phi = lambda Xv, Wv: float(np.sum(dY.astype(np.float64) * o.fwd(Xv, idx, Wv, b, G, F32)))
    for (bb, ff) in [(0, int(idx[0, 0])), (1, int(idx[1, 2])), (3, int(idx[3, 4])), (2, 0), (0, F_s - 1)]:
        Xp, Xm = X.copy(), X.copy()
        Xp[bb, ff] += np.float32(0.5)
        Xm[bb, ff] -= np.float32(0.5)
        fd = (phi(Xp, W) - phi(Xm, W)) / (float(Xp[bb, ff]) - float(Xm[bb, ff]))
        assert abs(fd - dX[bb, ff]) <= 1e-10 * max(1.0, abs(dX[bb, ff])), f"FD dX[{bb},{ff}] {fd} vs {dX[bb, ff]}"
    for (l, t) in [(0, 0), (5, 3), (15, 4), (9, 1)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[l, t] += np.float32(0.25)
        Wm[l, t] -= np.float32(0.25)
        fd = (phi(X, Wp) - phi(X, Wm)) / (float(Wp[l, t]) - float(Wm[l, t]))
        assert abs(fd - dW[l, t]) <= 1e-10 * max(1.0, abs(dW[l, t])), f"FD dW[{l},{t}] {fd} vs {dW[l, t]}"
    # the BCE objective itself (nonlinear): O(eps^2) truncation
    dY64 = 1.0 / (1.0 + np.exp(-Y)) - T
    dY32 = dY64.astype(np.float32)
    dX_bce = o.bwd_x(idx, W, dY32, G, F_s, F32)
    for (bb, ff) in [(0, int(idx[0, 0])), (2, int(idx[2, 1]))]:
        Xp, Xm = X.copy(), X.copy()
        Xp[bb, ff] += np.float32(1e-3)
        Xm[bb, ff] -= np.float32(1e-3)
        fd = (_bce(o.fwd(Xp, idx, W, b, G, F32), T) - _bce(o.fwd(Xm, idx, W, b, G, F32), T)) / (
            float(Xp[bb, ff]) - float(Xm[bb, ff]))
        assert abs(fd - dX_bce[bb, ff]) <= 1e-5 * max(1.0, abs(fd)), f"BCE FD dX[{bb},{ff}] {fd} vs {dX_bce[bb, ff]}"


def pin_adjoint_identity(o):
    """<dY, Y - bias> = <dX, X> = <dW, W> (the layer is bilinear in (X, W))."""
    rng = np.random.default_rng(9)
    for dtype in (F32, BF16):
        B, F_s, L, G, F_in = 9, 50, 96, 8, 12
        X, idx, W, b, dY = rand_layer(rng, B, F_s, L, G, F_in, dtype)
        Y = o.fwd(X, idx, W, b, G, dtype)
        dX = o.bwd_x(idx, W, dY, G, F_s, dtype)
        dW, _ = o.bwd_w(X, idx, dY, G, F_in, dtype)
        a = float(np.sum(f64(dY, dtype) * (Y - b)))
        c = float(np.sum(dX * f64(X, dtype)))
        d = float(np.sum(dW * f64(W, dtype)))
        scale = float(np.sum(np.abs(f64(dY, dtype) * (Y - b))))
        assert abs(a - c) <= 1e-12 * scale and abs(a - d) <= 1e-12 * scale, f"adjoint {a} {c} {d}"


def pin_one_hot(o):
    """One-hot weights / upstream rows turn the three products into exact gathers and scatters."""
    rng = np.random.default_rng(21)
    B, F_s, L, G, F_in = 6, 20, 24, 4, 5
    X, idx, _, _, dY = rand_layer(rng, B, F_s, L, G, F_in, F32, bias=False)
    g = np.arange(L) // G
    for t0 in range(F_in):
        W = np.zeros((L, F_in), np.float32)
        W[:, t0] = 1
        close(o.fwd(X, idx, W, None, G, F32), X[:, idx[g, t0]], 0, f"one-hot fwd t0={t0}")
    b0 = 4
    dYo = np.zeros((B, L), np.float32)
    dYo[b0] = 1
    close(o.bwd_w(X, idx, dYo, G, F_in, F32)[0], X[b0][idx[g]], 0, "one-hot bwd_w")
    l0, t0 = 9, 3
    W = np.zeros((L, F_in), np.float32)
    W[l0, t0] = 1
    dX = o.bwd_x(idx, W, dY, G, F_s, F32)
    exp = np.zeros((B, F_s))
    exp[:, idx[l0 // G, t0]] = dY[:, l0]
    close(dX, exp, 0, "one-hot bwd_x")
    # features outside every support get exactly +0.0
    W = rng.standard_normal((L, F_in)).astype(np.float32)
    used = np.zeros(F_s, bool)
    used[idx.reshape(-1)] = True
    dX = o.bwd_x(idx, W, dY, G, F_s, F32)
    assert np.all(dX[:, ~used] == 0.0), "untouched features must stay zero"


def pin_group_permutation(o):
    """Permuting groups (their labels and idx rows together) permutes Y columns and dW rows."""
    rng = np.random.default_rng(31)
    B, F_s, L, G, F_in = 5, 25, 36, 6, 4
    X, idx, W, b, dY = rand_layer(rng, B, F_s, L, G, F_in, F32)
    K = L // G
    pk = rng.permutation(K)
    lab = (pk[:, None] * G + np.arange(G)[None, :]).reshape(-1)   # new label n holds old label lab[n]
    Y = o.fwd(X, idx, W, b, G, F32)
    Yp = o.fwd(X, idx[pk], W[lab], b[lab], G, F32)
    close(Yp, Y[:, lab], 0, "perm fwd")
    dW = o.bwd_w(X, idx, dY, G, F_in, F32)[0]
    close(o.bwd_w(X, idx[pk], dY[:, lab], G, F_in, F32)[0], dW[lab], 0, "perm dW")
    close(o.bwd_x(idx[pk], W[lab], dY[:, lab], G, F_s, F32), o.bwd_x(idx, W, dY, G, F_s, F32), 1e-13, "perm dX")


def pin_label_ranges(o):
    """Label-range, row-range and sampled entry points agree with the full computation."""
    rng = np.random.default_rng(41)
    B, F_s, L, G, F_in = 7, 30, 64, 8, 6
    X, idx, W, b, dY = rand_layer(rng, B, F_s, L, G, F_in, BF16)
    Y = o.fwd(X, idx, W, b, G, BF16)
    close(o.fwd(X, idx, W, b, G, BF16, 13, 41), Y[:, 13:41], 0, "fwd range")
    bs = np.array([0, 6, 3, 3]); ls = np.array([0, 63, 17, 40])
    close(o.fwd_at(X, idx, W, b, G, BF16, bs, ls), Y[bs, ls], 0, "fwd_at")
    dW, db = o.bwd_w(X, idx, dY, G, F_in, BF16, with_dbias=True)
    dW2, db2 = o.bwd_w(X, idx, dY, G, F_in, BF16, 8, 24, with_dbias=True)
    close(dW2, dW[8:24], 0, "bwd_w range")
    close(db2, db[8:24], 0, "dbias range")
    dX = o.bwd_x(idx, W, dY, G, F_s, BF16)
    close(o.bwd_x(idx, W, dY, G, F_s, BF16, 2, 5), dX[2:5], 0, "bwd_x range")


def pin_head(o):
    """Dense head: Yh = X Wh^T + bh, dWh = dYh^T X, dXh = dYh Wh (np.matmul, fp64)."""
    rng = np.random.default_rng(51)
    for dtype in (F32, BF16):
        B, F_s, H = 6, 21, 13
        X = rng.standard_normal((B, F_s)).astype(np.float32)
        Wh = rng.standard_normal((H, F_s)).astype(np.float32)
        dYh = rng.standard_normal((B, H)).astype(np.float32)
        bh = rng.standard_normal(H).astype(np.float32)
        if dtype == BF16:
            X, Wh, dYh = synth.bf16_bits(X), synth.bf16_bits(Wh), synth.bf16_bits(dYh)
        Xd, Whd, dYd = f64(X, dtype), f64(Wh, dtype), f64(dYh, dtype)
        close(o.head_fwd(X, Wh, bh, dtype), Xd @ Whd.T + bh, 1e-12, "head fwd")
        close(o.head_fwd(X, Wh, None, dtype, 3, 9), (Xd @ Whd.T)[:, 3:9], 1e-12, "head fwd range")
        close(o.head_bwd_w(X, dYh, dtype), dYd.T @ Xd, 1e-12, "head dW")
        close(o.head_bwd_w(X, dYh, dtype, 2, 7), (dYd.T @ Xd)[2:7], 1e-12, "head dW range")
        close(o.head_bwd_x(Wh, dYh, dtype), dYd @ Whd, 1e-12, "head dX")
        close(o.head_bwd_x(Wh, dYh, dtype, 1, 4), (dYd @ Whd)[1:4], 1e-12, "head dX range")


def pin_bce_grad(o):
    """The BCE gradient is the derivative of the Section 3.3 objective: central differences of
    sum(log(1 + e^z) - y z), closed forms at z = 0 and z = ln 3, and the target rule (pos entries
    outside the row's range are ignored, repeats count once)."""
    rng = np.random.default_rng(21)
    B, N = 5, 23
    Z = 3.0 * rng.standard_normal((B, N))
    Z[0, :4] = 0.0
    Z[1, 2] = np.log(3.0)
    Z[2, 5], Z[2, 6] = 40.0, -40.0
    pos = np.array([[0, 3, 3, -1], [2, 22, 23, -7], [5, 6, 5, 6], [-1, -1, -1, -1], [11, 0, 22, 1]], np.int32)
    T = np.zeros((B, N))
    for b in range(B):
        for c in pos[b]:
            if 0 <= c < N:
                T[b, c] = 1.0
    g = o.bce_grad(Z, pos)
    h = 1e-5
    for b in range(B):
        for n in range(N):
            Zp, Zm = Z.copy(), Z.copy()
            Zp[b, n] += h
            Zm[b, n] -= h
            fd = (_bce(Zp, T) - _bce(Zm, T)) / (2 * h)
            assert abs(fd - g[b, n]) <= 1e-7, f"BCE grad [{b},{n}]: {g[b, n]} vs central difference {fd}"
    assert np.array_equal(g[0, :4], 0.5 - T[0, :4]), "sigmoid(0) - y must be 0.5 - y exactly"
    assert abs(g[1, 2] - (0.75 - T[1, 2])) <= 1e-15, "sigmoid(ln 3) = 3/4"
    # the sampled form agrees with the same central differences at every point
    bs, ns = np.meshgrid(np.arange(B), np.arange(N), indexing="ij")
    ga = o.bce_grad_at(pos, N, bs.ravel(), ns.ravel(), Z.ravel()).reshape(B, N)
    assert np.abs(ga - g).max() <= 1e-15, "sampled BCE gradient differs from the dense one"
    zero = o.bce_grad(Z, np.zeros((B, 0), np.int32))
    assert np.abs(zero - 1.0 / (1.0 + np.exp(-Z))).max() <= 1e-15, "no positives: gradient is sigmoid(z)"


def pin_sgd_momentum(o):
    """The momentum step against closed forms that do not restate it: a constant gradient g from rest
    gives m_T = g (1 - mu^T) / (1 - mu) and moves W by lr g sum_t (1 - mu^t) / (1 - mu); weight
    decay alone shrinks W geometrically by (1 - lr wd) per step (mu = 0); and heavy-ball steps on
    the quadratic |W - W*|^2 / 2 (gradient W - W*) converge to W*."""
    rng = np.random.default_rng(31)
    n = 37
    W0 = rng.standard_normal(n)
    g = rng.standard_normal(n)
    lr, mu, T = 0.05, 0.9, 6
    W, m = W0.copy(), np.zeros(n)
    for _ in range(T):
        W, m = o.sgd_momentum(W, g, m, lr, mu, 0.0, F32)
    geo = lambda t: (1 - mu ** t) / (1 - mu)
    m_ref = g * geo(T)
    W_ref = W0.astype(np.float32).astype(np.float64) - lr * g * sum(geo(t) for t in range(1, T + 1))
    # W passes through fp32 storage between steps in this loop: compare within that rounding
    assert np.abs(m - m_ref).max() <= 1e-12 * max(1.0, np.abs(m_ref).max()), "momentum of a constant gradient"
    assert np.abs(W - W_ref).max() <= 1e-5 * max(1.0, np.abs(W_ref).max()), "weights under a constant gradient"
    Wd = W0.copy()
    for _ in range(T):
        Wd, _m = o.sgd_momentum(Wd, np.zeros(n), np.zeros(n), lr, 0.0, 0.3, F32)
    Wd_ref = W0.astype(np.float32).astype(np.float64) * (1 - lr * 0.3) ** T
    assert np.abs(Wd - Wd_ref).max() <= 1e-6, "weight decay alone is a geometric shrink"
    Wstar = rng.standard_normal(n)
    Wq, mq = np.zeros(n), np.zeros(n)
    for _ in range(400):
        Wq, mq = o.sgd_momentum(Wq, Wq.astype(np.float32).astype(np.float64) - Wstar, mq, 0.1, 0.8, 0.0, F32)
    assert np.abs(Wq - Wstar).max() <= 1e-5, "heavy-ball steps on a quadratic must converge to its minimum"


def pin_splitmix64(o):
    """The counter-based generator of the rewiring draws is SplitMix64 (Steele, Lea and Flood, 2014):
    its first three outputs for seed 0, as published with the reference implementation."""
    assert [o.splitmix64(0, i) for i in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def _scores_f32(W, G, F, dtype):
    """Per-(group, slot) sums of |w| over the group's labels, fp32, labels in order (independent)."""
    Wf = np.abs(synth.to_f64(W, dtype).astype(np.float32)).reshape(-1, G, F)
    s = np.zeros((Wf.shape[0], F), np.float32)
    for g in range(G):
        s += Wf[:, g, :]
    return s


def pin_rewire_hand(o):
    """Alg. 3 on a hand-checked layer: scores [[0.1, 5, 3], [2, 0.05, 7]], rho = 0.34 gives
    m = floor(6 * 0.34) = 2, so slot 0 of group 0 and slot 1 of group 1 are pruned; kept features
    keep their weights, the new features are outside the kept ones, zero init gives zero weights."""
    idx = np.array([[1, 4, 6], [0, 2, 7]], np.int32)
    W = np.array([[0.05, 2.0, 1.0], [0.05, 3.0, 2.0], [1.0, 0.02, 3.0], [1.0, 0.03, 4.0]], np.float32)
    idx2, W2, _, n, mask = o.rewire(idx, W, None, 2, 8, F32, 0.34, False, 7)
    assert n == 2
    assert np.array_equal(mask, np.array([[1, 0, 0], [0, 1, 0]], bool)), f"pruned slots {mask}"
    for k, kept in ((0, {4: (2.0, 3.0), 6: (1.0, 2.0)}), (1, {0: (1.0, 1.0), 7: (3.0, 4.0)})):
        row = list(idx2[k])
        assert row == sorted(set(row)) and len(row) == 3
        new = [f for f in row if f not in kept]
        assert len(new) == 1, f"group {k} must gain exactly one feature outside its kept ones: {row}"
        for f, ws in kept.items():
            p = row.index(f)
            assert (W2[2 * k, p], W2[2 * k + 1, p]) == ws, f"kept weight of feature {f} moved wrongly"
        p = row.index(new[0])
        assert W2[2 * k, p] == 0.0 and W2[2 * k + 1, p] == 0.0


def pin_rewire_ties_and_noop(o):
    """Equal scores (all-zero weights) prune the lowest flat indices first; rho = 0 changes nothing."""
    rng = np.random.default_rng(41)
    K, F, G, H = 5, 4, 2, 20
    idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
    _, _, _, n, mask = o.rewire(idx, np.zeros((K * G, F), np.float32), None, G, H, F32, 0.5, False, 1)
    assert n == 10 and np.array_equal(mask.reshape(-1), np.arange(K * F) < 10), "ties must go to the lower index"
    W = rng.standard_normal((K * G, F)).astype(np.float32)
    idx2, W2, _, n, mask = o.rewire(idx, W, None, G, H, F32, 0.0, True, 1)
    assert n == 0 and not mask.any() and np.array_equal(idx2, idx) and np.array_equal(W2, W)


def pin_rewire_invariants(o):
    """On random layers: exactly m slots pruned, none scoring above a kept one; rows stay strictly
    increasing; every kept (feature, weight column, velocity) survives; new features are outside the
    kept set, with weights within 1/sqrt(F) (random init) and zero velocity."""
    rng = np.random.default_rng(43)
    for dtype, init in ((BF16, True), (F32, False)):
        K, G, F, H, rho = 50, 4, 16, 64, 0.3
        idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
        W = (rng.standard_normal((K * G, F)) * rng.random((K * G, 1))).astype(np.float32)
        W = synth.bf16_bits(W) if dtype == BF16 else W
        m = rng.standard_normal((K * G, F))
        idx2, W2, m2, n, mask = o.rewire(idx, W, m, G, H, dtype, rho, init, 123)
        assert n == int(np.floor(K * F * rho)) and mask.sum() == n
        S = _scores_f32(W, G, F, dtype)
        assert S[mask].max() <= S[~mask].min(), "a pruned slot scores above a kept one"
        Wv, W2v = synth.to_f64(W, dtype), synth.to_f64(W2, dtype)
        for k in range(K):
            row = list(idx2[k])
            assert all(0 <= f < H for f in row) and all(a < b for a, b in zip(row, row[1:]))
            kept = {int(idx[k, j]): j for j in range(F) if not mask[k, j]}
            new = [p for p, f in enumerate(row) if f not in kept]
            assert len(new) == int(mask[k].sum())
            for f, j in kept.items():
                p = row.index(f)
                for g in range(G):
                    l = k * G + g
                    assert W2v[l, p] == Wv[l, j] and m2[l, p] == m[l, j], "kept slot lost its weight or velocity"
            for p in new:
                for g in range(G):
                    l = k * G + g
                    assert m2[l, p] == 0.0
                    assert (abs(W2v[l, p]) <= 1.0 / np.sqrt(F) * (1 + 2 ** -8)) if init else W2v[l, p] == 0.0


def pin_rewire_uniform(o):
    """A pruned slot's new feature is uniform over the features its group does not keep: with F = 2
    and one slot pruned, the new feature's rank among the H - 1 free features is uniform."""
    rng = np.random.default_rng(47)
    K, F, H = 4000, 2, 6
    idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
    W = rng.random((K, F)).astype(np.float32) + 0.5
    idx2, _, _, _, mask = o.rewire(idx, W, None, 1, H, F32, 0.5, False, 99)
    counts = np.zeros(H - 1)
    for k in np.nonzero(mask.sum(axis=1) == 1)[0]:
        kept = int(idx[k][~mask[k]][0])
        others = [int(f) for f in idx2[k] if f != kept]
        assert len(others) == 1 and kept in idx2[k], f"group {k}: {idx2[k]} must keep {kept} and add one feature"
        free = [f for f in range(H) if f != kept]
        counts[free.index(others[0])] += 1
    exp = counts.sum() / (H - 1)
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert counts.sum() > 1000 and chi2 < 25.0, f"new-feature ranks not uniform: {counts}, chi2 {chi2:.1f}"


def pin_rewire_reinit_distribution(o):
    """Alg. 3's random mode draws each reinitialised weight from Unif(-1/sqrt(F), 1/sqrt(F)): over
    many pruned slots the values stay inside that interval, take both signs, reach both ends, have
    mean 0 and variance 1/(3F) (the moments of that uniform law), and fill ten equal bins evenly."""
    rng = np.random.default_rng(59)
    K, G, F, H, rho = 400, 8, 16, 64, 0.5
    idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
    W = (rng.random((K * G, F)) + 1.0).astype(np.float32)   # kept weights lie in [1, 2): not draws
    idx2, W2, _, n, mask = o.rewire(idx, W, None, G, H, F32, rho, True, 2024)
    vals = []
    for k in range(K):
        kept = set(int(idx[k, j]) for j in range(F) if not mask[k, j])
        new = [p for p, f in enumerate(idx2[k]) if int(f) not in kept]
        vals.append(W2[k * G:(k + 1) * G][:, new].reshape(-1))
    v = np.concatenate(vals).astype(np.float64)
    a = 1.0 / np.sqrt(F)
    assert v.size == n * G and v.size > 20000
    assert np.all(np.abs(v) <= a), "a reinitialised weight lies outside [-1/sqrt(F), 1/sqrt(F)]"
    assert (v > 0).mean() > 0.45 and (v < 0).mean() > 0.45, "reinitialised weights must take both signs"
    assert v.max() > 0.99 * a and v.min() < -0.99 * a, "draws must reach both ends of the interval"
    sd_mean = np.sqrt(a * a / 3 / v.size)
    assert abs(v.mean()) < 5 * sd_mean, f"mean {v.mean():.3g} is not 0"
    assert abs(v.var() / (a * a / 3) - 1) < 0.05, f"variance {v.var():.4g} is not 1/(3F) = {a * a / 3:.4g}"
    counts = np.histogram(v, bins=10, range=(-a, a))[0]
    exp = v.size / 10
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 30.0, f"reinitialised weights not uniform over ten bins: {counts}, chi2 {chi2:.1f}"


def _cos_rows(E, s):
    """fp64 cosine of every row of E with vector s (NumPy; independent of the oracle)."""
    Ef = E.astype(np.float64)
    sf = np.asarray(s, np.float64)
    return (Ef @ sf) / (np.linalg.norm(Ef, axis=1) * np.linalg.norm(sf))


def _brute_group(o, E, G, beta, iters, seed):
    """Alg. 2 written out with NumPy cosines: spherical k-means whose centres are the normalised
    means of their members (ties to the lower centre; an empty cluster keeps its centre), then per
    cluster a seed plus its top-(G - 1) unassigned neighbours by cosine (ties to the lower label).
    Random choices follow the documented counter draws of the generator (pinned separately)."""
    E = np.asarray(E, np.int8)
    N, D = E.shape
    C = max(1, N // (beta * G))
    perm = list(range(N))
    for i in range(C):
        j = i + o.splitmix64(seed, i) % (N - i)
        perm[i], perm[j] = perm[j], perm[i]
    mu = np.stack([E[perm[c]].astype(np.float64) for c in range(C)])
    mu /= np.linalg.norm(mu, axis=1, keepdims=True)
    Ef = E.astype(np.float64)

    def assign():
        return np.argmax(Ef @ mu.T, axis=1)   # the first maximum: the lower centre

    for _ in range(iters):
        cl = assign()
        for c in range(C):
            s = Ef[cl == c].sum(axis=0)
            if (cl == c).any() and np.linalg.norm(s) > 0:
                mu[c] = s / np.linalg.norm(s)
    cl = assign()
    order, gsize = [], []
    for c in range(C):
        un = [l for l in range(N) if cl[l] == c]
        t = 0
        while un:
            s = un[o.splitmix64(seed, N + c * N + t) % len(un)]
            t += 1
            rest = [l for l in un if l != s]
            cs = _cos_rows(E[rest], E[s]) if rest else np.zeros(0)
            ranked = sorted(range(len(rest)), key=lambda i: (-cs[i], rest[i]))
            grp = sorted([s] + [rest[i] for i in ranked[:G - 1]])
            order += grp
            gsize.append(len(grp))
            un = sorted(set(un) - set(grp))
    return np.array(order), np.array(gsize), cl


def pin_group_bruteforce(o):
    """Alg. 2 on small random int8 embeddings of uneven norms (so that a dot product and a cosine
    rank differently) against its brute-force statement with NumPy cosines: identical clusters,
    groups and group order, for several seeds and iteration counts, with exact duplicate rows."""
    rng = np.random.default_rng(61)
    for N, D, G, beta in ((40, 8, 4, 20), (240, 16, 4, 10), (300, 8, 8, 6)):
        E = (rng.integers(-127, 128, (N, D)) * (0.1 + 0.9 * rng.random((N, 1)))).astype(np.int8)
        E[np.abs(E).sum(axis=1) == 0, 0] = 1   # cosines need non-zero rows
        E[5] = E[17]                        # an exact tie of cosines, broken by the lower label
        for iters, seed in ((0, 3), (1, 0), (4, 11)):
            order, gs, cl = o.group_labels(E, G, beta, iters, seed)
            order_b, gs_b, cl_b = _brute_group(o, E, G, beta, iters, seed)
            assert np.array_equal(cl, cl_b), f"N={N} iters={iters}: clusters differ from spherical k-means"
            assert np.array_equal(gs, gs_b) and np.array_equal(order, order_b), \
                f"N={N} iters={iters} seed={seed}: groups differ from the greedy cosine stage"


def pin_group_seed_in_group(o):
    """The seed always belongs to its own group (Section 3.1: a seed and its top-(G - 1) neighbours),
    also for near-duplicate labels a, b whose int8 rounding makes a.b exceed b.b: with labels
    {a, b, a} and G = 2, a seed b gives the group {b, the lower a}, a seed a gives {a, a}."""
    rng = np.random.default_rng(67)
    while True:
        u = rng.standard_normal(16)
        a = np.rint(127 * u / np.linalg.norm(u)).astype(np.int64)
        w = u + rng.standard_normal(16) * 0.01
        b = np.rint(127 * w / np.linalg.norm(w)).astype(np.int64)
        if a @ b > b @ b and not np.array_equal(a, b):
            break
    E = np.stack([a, b, a]).astype(np.int8)
    seen = set()
    for seed in range(12):
        order, gs, _ = o.group_labels(E, 2, 8, 0, seed)
        first_seed = [0, 1, 2][o.splitmix64(seed, 3) % 3]
        want = [0, 1] if first_seed == 1 else [0, 2]
        assert list(gs) == [2, 1] and list(order[:2]) == want, f"seed {seed} (label {first_seed}): {order}"
        seen.add(first_seed)
    assert 1 in seen, "no draw picked the seed b"


def _unit_int8(X):
    X = np.asarray(X, np.float64)
    return np.rint(127 * X / np.linalg.norm(X, axis=1, keepdims=True)).astype(np.int8)


def pin_group_greedy(o):
    """Alg. 2's greedy stage on one coarse cluster (beta G >= N): three planted directions of four
    labels each (labels interleaved) come back as exactly those three groups, whatever the seed."""
    rng = np.random.default_rng(51)
    N, D = 12, 8
    X = np.zeros((N, D))
    for l in range(N):
        X[l, l % 3] = 10.0
        X[l, 3:] = rng.standard_normal(D - 3)
    E = _unit_int8(X)
    want = {frozenset(l for l in range(N) if l % 3 == g) for g in range(3)}
    for seed in (0, 1, 2, 12345):
        order, gs, cl = o.group_labels(E, 4, 3, 3, seed)
        assert list(gs) == [4, 4, 4] and not cl.any()
        groups = [order[4 * i: 4 * i + 4] for i in range(3)]
        assert all(list(g) == sorted(g) for g in groups)
        assert {frozenset(int(x) for x in g) for g in groups} == want, f"seed {seed}: {groups}"


def pin_group_planted(o):
    """On embeddings with eight planted clusters of 256, the coarse k-means recovers the clusters
    (each k-means cluster dominated by one planted cluster), at least 90% of the groups are pure,
    and the output is a partition into groups of G (the last of a cluster may be short)."""
    rng = np.random.default_rng(53)
    N, D, P, G, beta = 2048, 64, 8, 16, 16
    mu = rng.standard_normal((P, D))
    planted = rng.permutation(np.repeat(np.arange(P), N // P))
    E = _unit_int8(mu[planted] / np.linalg.norm(mu[planted], axis=1, keepdims=True) * 4 + rng.standard_normal((N, D)) * 0.15)
    order, gs, cl = o.group_labels(E, G, beta, 8, 77)
    assert sorted(order.tolist()) == list(range(N)), "groups must partition the labels"
    C = N // (beta * G)
    assert cl.min() >= 0 and cl.max() < C
    dominated = 0
    for c in range(C):
        members = planted[cl == c]
        if members.size and np.bincount(members, minlength=P).max() >= 0.8 * members.size:
            dominated += 1
    assert dominated >= C - 2, f"only {dominated} of {C} k-means clusters follow the planted ones"
    starts = np.concatenate([[0], np.cumsum(gs)])
    pure = 0
    for i in range(gs.size):
        g = order[starts[i]:starts[i + 1]]
        assert len(set(cl[g])) == 1, "a group spans two coarse clusters"
        pure += len(set(planted[g])) == 1
    assert pure >= 0.9 * gs.size, f"only {pure} of {gs.size} groups are pure"
    for c in range(C):
        n_c = int((cl == c).sum())
        assert sum(1 for i in range(gs.size) if cl[order[starts[i]]] == c) == -(-n_c // G), "groups per cluster"
    assert gs.max() <= G


ALL_PINS = [pin_fig2_gs, pin_fig2_ffi, pin_bruteforce, pin_duplicate_indices, pin_dense_special_case,
            pin_group_equals_expanded_ffi, pin_finite_differences, pin_adjoint_identity, pin_one_hot,
            pin_group_permutation, pin_label_ranges, pin_head, pin_bce_grad,
            pin_sgd_momentum, pin_splitmix64, pin_rewire_hand, pin_rewire_ties_and_noop, pin_rewire_invariants,
            pin_rewire_uniform, pin_rewire_reinit_distribution, pin_group_greedy, pin_group_planted,
            pin_group_bruteforce, pin_group_seed_in_group]
