"""Shared helpers of the GPU tests: device transfer, running the layer through the C ABI, and the
error metric.  The error metric follows the tolerance of the build target: per output tensor,
max_i |gpu_i - oracle_i| / max_i |oracle_i| (infinity-norm relative error) against the fp64 oracle;
1e-5 for fp32 layers, 2e-2 for bf16 storage with fp32 accumulation."""
from __future__ import annotations

import sys

import numpy as np

import synth

TOL = {synth.DT_F32: 1e-5, synth.DT_BF16: 2e-2}
F32 = synth.DT_F32


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel_err(a, r) -> float:
    a = np.asarray(a, np.float64)
    r = np.asarray(r, np.float64)
    if r.size == 0:
        return 0.0
    den = float(np.abs(r).max())
    return float(np.abs(a - r).max()) / (den if den > 0 else 1.0)


def to_dev(a, dev="cuda"):
    import torch
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


def host_f32(t, dtype) -> np.ndarray:
    """Device tensor in the layer's storage dtype -> fp32 numpy (exact)."""
    a = t.detach().cpu().numpy()
    if dtype == synth.DT_BF16:
        return synth.bf16_to_f32(a.view(np.uint16))
    return a.astype(np.float32)


def out_tensor(shape, dtype, dev="cuda"):
    import torch
    return torch.empty(shape, dtype=torch.int16 if dtype == synth.DT_BF16 else torch.float32, device=dev)


class Layer:
    """The tail layer's device buffers plus the three ABI calls."""

    def __init__(self, hs, wl, X, idx, W, bias, dY):
        import torch
        self.hs, self.wl = hs, wl
        self.desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, wl.dtype)
        self.X, self.idx, self.W = to_dev(X), to_dev(idx), to_dev(W)
        self.bias = to_dev(bias)
        self.dY = to_dev(dY)
        self.Y = out_tensor((wl.B, wl.L), wl.dtype)
        self.dW = torch.empty((wl.L, wl.F_in), dtype=torch.float32, device="cuda")
        self.dbias = torch.empty((wl.L,), dtype=torch.float32, device="cuda")
        self.dX = torch.empty((wl.B, wl.F_s), dtype=torch.float32, device="cuda")
        self.ws_w = hs.workspace(hs.haste_workspace_bytes(self.desc, hs.HASTE_OP_BWD_W))
        self.ws_x = hs.workspace(hs.haste_workspace_bytes(self.desc, hs.HASTE_OP_BWD_X))

    def fwd(self):
        self.hs.haste_fwd(self.desc, self.X, self.idx, self.W, self.bias, self.Y)

    def bwd_w(self, beta=0, dbias=True):
        self.hs.haste_bwd_w(self.desc, self.X, self.idx, self.dY, self.dW, self.dbias if dbias else None, beta,
                            self.ws_w)

    def bwd_x(self, beta=0):
        self.hs.haste_bwd_x(self.desc, self.idx, self.W, self.dY, self.dX, beta, self.ws_x)


def make_inputs(wl, orc=None, logits_from_oracle=False):
    X = synth.draw_X(wl)
    W = synth.draw_W(wl)
    idx = synth.draw_idx(wl)
    bias = synth.draw_bias(wl)
    if wl.dy_normal:
        dY = synth.draw_dY(wl)
    else:
        logits = orc.fwd(X, idx, W, bias, wl.G, wl.dtype) if logits_from_oracle else None
        dY = synth.draw_dY(wl, logits=logits)
    return X, idx, W, bias, dY


# ---- the loss-gradient calls: positives lists and the oracle's composition ----------------
def rand_pos(rng, B, L, P):
    """[B, P] positives with the awkward entries: repeats, -1 padding, ids past L and below -1,
    and ids on 512-label span edges and at both ends of the layer."""
    if P == 0:
        return np.zeros((B, 0), np.int32)
    pos = rng.integers(0, L, size=(B, P)).astype(np.int32)
    edges = [0, L - 1, min(511, L - 1), min(512, L - 1), L // 2]
    for b in range(B):
        r = rng.random()
        if r < 0.2:
            pos[b, -1] = -1
        elif r < 0.3:
            pos[b, -1] = L + int(rng.integers(0, 100))
        elif r < 0.4:
            pos[b, -1] = -int(rng.integers(2, 100))
        elif r < 0.6 and P > 1:
            pos[b, -1] = pos[b, 0]       # a repeat counts once
        pos[b, 0] = edges[b % len(edges)] if b % 3 == 0 else pos[b, 0]
    return pos


def skewed_pos(rng, B, L, P, hot=512):
    """[B, P] positives with rows of very different lengths (-1 padded): up to half of a row in the
    first `hot` labels (one workgroup's span, so that its cells hold many entries), the rest
    anywhere, some repeats, ids out of range."""
    pos = np.full((B, P), -1, np.int32)
    for b in range(B):
        n = P if b % 3 == 0 else int(rng.integers(0, P + 1))
        nh = min(n // 2, hot)
        row = list(rng.choice(hot, nh, replace=False)) + list(rng.integers(0, L, n - nh))
        if n > 2 and b % 5 == 0:
            row[-1] = row[0]              # a repeat counts once
        if n > 3 and b % 7 == 0:
            row[-2] = L + 5               # outside the layer: ignored
        pos[b, :n] = row
    return pos


def targets(pos, B, L):
    T = np.zeros((B, L), bool)
    for b in range(B):
        for c in pos[b]:
            if 0 <= c < L:
                T[b, c] = True
    return T


def oracle_fwd_bce(orc, X, idx, W, bias, pos, G, F_in, dt):
    """fp64 composition: logits, BCE gradient, backward-weight (dY passed at fp32 precision)."""
    z = orc.fwd(X, idx, W, bias, G, dt)
    dY = orc.bce_grad(z, pos)
    Xf = synth.to_f64(X, dt).astype(np.float32)   # exact for bf16 and fp32 storage
    dW, db = orc.bwd_w(Xf, idx, dY.astype(np.float32), G, F_in, F32, with_dbias=True)
    return dY, dW, db
