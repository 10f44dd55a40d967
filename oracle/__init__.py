"""CPU oracle for the group-shared fixed fan-in output layer (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may import
this package.  The product path (the HIP library and its binding) never touches it.

The arithmetic lives in ``haste_oracle.c`` (plain C, fp64 accumulation, OpenMP over rows or
labels); this module only builds it with gcc and marshals NumPy arrays.  Definitions followed:
paper Section 3.1 (logit of a label on its group's support), Section 3.2 (backward-weight on the
support only; backward-feature as a reduction over groups) and Section 3.3 (dense head).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "haste_oracle.c")
LIB = os.path.join(HERE, "liboracle_haste.so")

DT_F32 = 0
DT_BF16 = 1


def build(src: str = SRC, out: str = LIB, extra: tuple = ()) -> str:
    """Compile the oracle with gcc (-O2, no fast-math: fp64 sums keep the written order)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """ctypes view of one compiled oracle library (the real one, or a planted-mistake build)."""

    def __init__(self, path: str = LIB):
        if not os.path.exists(path):
            build(out=path) if path == LIB else None
        self.lib = ctypes.CDLL(path)
        L = self.lib
        L.haste_oracle_num_threads.restype = ctypes.c_int
        sig_layer = [_I64] * 5 + [ctypes.c_int]
        L.haste_oracle_fwd.argtypes = sig_layer + [_P, _P, _P, _P, _I64, _I64, _P]
        L.haste_oracle_fwd_at.argtypes = sig_layer + [_P, _P, _P, _P, _I64, _P, _P, _P]
        L.haste_oracle_bwd_w.argtypes = sig_layer + [_P, _P, _P, _I64, _I64, _P, _P]
        L.haste_oracle_bwd_x.argtypes = sig_layer + [_P, _P, _P, _I64, _I64, _P]
        sig_head = [_I64, _I64, _I64, ctypes.c_int]
        L.haste_oracle_head_fwd.argtypes = sig_head + [_P, _P, _P, _I64, _I64, _P]
        L.haste_oracle_head_bwd_w.argtypes = sig_head + [_P, _P, _I64, _I64, _P]
        L.haste_oracle_head_bwd_x.argtypes = sig_head + [_P, _P, _I64, _I64, _P]
        L.haste_oracle_bce_grad.argtypes = [_I64, _I64, _P, _P, _I64, _P]
        L.haste_oracle_bce_grad_at.argtypes = [_I64, _I64, _P, _I64, _I64, _P, _P, _P, _P]
        _D = ctypes.c_double
        L.haste_oracle_sgd_momentum.argtypes = [_I64, ctypes.c_int, _P, _P, _P, _D, _D, _D, _P]
        L.haste_oracle_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.haste_oracle_splitmix64.restype = ctypes.c_uint64
        L.haste_oracle_rewire.argtypes = [_I64, _I64, _I64, _I64, ctypes.c_int, _P, _P, _P, _D, ctypes.c_int,
                                          ctypes.c_uint64, _P, _P]
        L.haste_oracle_rewire.restype = ctypes.c_int
        L.haste_oracle_group_labels.argtypes = [_I64, _I64, _P, _I64, _I64, _I64, ctypes.c_uint64, _P, _P, _P, _P]
        L.haste_oracle_group_labels.restype = ctypes.c_int
        for f in ("fwd", "fwd_at", "bwd_w", "bwd_x", "head_fwd", "head_bwd_w", "head_bwd_x", "bce_grad",
                  "bce_grad_at", "sgd_momentum"):
            getattr(L, "haste_oracle_" + f).restype = ctypes.c_int

    # ---- helpers --------------------------------------------------------------------------
    @staticmethod
    def _c(a, dtype=None):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        if dtype is not None:
            a = np.ascontiguousarray(a, dtype=dtype)
        return a

    @staticmethod
    def _store(a, dt):
        return np.ascontiguousarray(a, dtype=np.uint16 if dt == DT_BF16 else np.float32)

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise ValueError(f"oracle {what}: invalid arguments (rc={rc})")

    def num_threads(self) -> int:
        return int(self.lib.haste_oracle_num_threads())

    # ---- tail ------------------------------------------------------------------------------
    def fwd(self, X, idx, W, bias, G, dtype, l0=0, l1=None):
        """Y[B, l1-l0] (fp64) for labels [l0, l1)."""
        X, W = self._store(X, dtype), self._store(W, dtype)
        idx = self._c(idx, np.int32)
        bias = self._c(bias, np.float32)
        B, F_s = X.shape
        L, F_in = W.shape
        l1 = L if l1 is None else l1
        Y = np.empty((B, l1 - l0), dtype=np.float64)
        rc = self.lib.haste_oracle_fwd(B, F_s, L, G, F_in, dtype, _ptr(X), _ptr(idx), _ptr(W), _ptr(bias),
                                       l0, l1, _ptr(Y))
        self._check(rc, "fwd")
        return Y

    def fwd_at(self, X, idx, W, bias, G, dtype, bs, ls):
        X, W = self._store(X, dtype), self._store(W, dtype)
        idx = self._c(idx, np.int32)
        bias = self._c(bias, np.float32)
        bs = np.ascontiguousarray(bs, dtype=np.int64)
        ls = np.ascontiguousarray(ls, dtype=np.int64)
        B, F_s = X.shape
        L, F_in = W.shape
        out = np.empty(bs.size, dtype=np.float64)
        rc = self.lib.haste_oracle_fwd_at(B, F_s, L, G, F_in, dtype, _ptr(X), _ptr(idx), _ptr(W), _ptr(bias),
                                          bs.size, _ptr(bs), _ptr(ls), _ptr(out))
        self._check(rc, "fwd_at")
        return out

    def bwd_w(self, X, idx, dY, G, F_in, dtype, l0=0, l1=None, with_dbias=False):
        """(dW[l1-l0, F_in], dbias[l1-l0] or None) in fp64."""
        X, dY = self._store(X, dtype), self._store(dY, dtype)
        idx = self._c(idx, np.int32)
        B, F_s = X.shape
        L = dY.shape[1]
        l1 = L if l1 is None else l1
        dW = np.empty((l1 - l0, F_in), dtype=np.float64)
        db = np.empty(l1 - l0, dtype=np.float64) if with_dbias else None
        rc = self.lib.haste_oracle_bwd_w(B, F_s, L, G, F_in, dtype, _ptr(X), _ptr(idx), _ptr(dY), l0, l1,
                                         _ptr(dW), _ptr(db))
        self._check(rc, "bwd_w")
        return dW, db

    def bce_grad(self, Z, pos):
        """dY[B, N] = sigmoid(Z) - T (fp64); T[b, n] = 1 where n occurs in pos[b, :] (pos [B, P] int32)."""
        Z = np.ascontiguousarray(Z, dtype=np.float64)
        B, N = Z.shape
        pos = np.ascontiguousarray(pos, dtype=np.int32).reshape(B, -1)
        out = np.empty_like(Z)
        rc = self.lib.haste_oracle_bce_grad(B, N, _ptr(Z), _ptr(pos), pos.shape[1], _ptr(out))
        self._check(rc, "bce_grad")
        return out

    def bce_grad_at(self, pos, N, bs, ns, z):
        """The BCE gradient at points (bs[i], ns[i]) whose logits are z[i]."""
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        B = pos.shape[0]
        bs = np.ascontiguousarray(bs, dtype=np.int64)
        ns = np.ascontiguousarray(ns, dtype=np.int64)
        z = np.ascontiguousarray(z, dtype=np.float64)
        out = np.empty(bs.size, dtype=np.float64)
        rc = self.lib.haste_oracle_bce_grad_at(B, N, _ptr(pos), pos.shape[1] if pos.ndim == 2 else 0, bs.size,
                                               _ptr(bs), _ptr(ns), _ptr(z), _ptr(out))
        self._check(rc, "bce_grad_at")
        return out

    def sgd_momentum(self, W, grad, m, lr, momentum, weight_decay, dtype):
        """One momentum step: returns (W_next, m_next) in fp64; W in its storage dtype."""
        W = self._store(W, dtype)
        g = np.ascontiguousarray(grad, dtype=np.float64).reshape(-1)
        mm = np.array(m, dtype=np.float64).reshape(-1)
        out = np.empty(W.size, dtype=np.float64)
        rc = self.lib.haste_oracle_sgd_momentum(W.size, dtype, _ptr(W), _ptr(g), _ptr(mm), lr, momentum,
                                                weight_decay, _ptr(out))
        self._check(rc, "sgd_momentum")
        return out.reshape(W.shape), mm.reshape(W.shape)

    def splitmix64(self, seed: int, i: int) -> int:
        return int(self.lib.haste_oracle_splitmix64(seed, i))

    def rewire(self, idx, W, m, G, H, dtype, rho, init_random, seed):
        """Returns (idx', W' in storage dtype, m' (fp64) or None, n_pruned, mask[K, F] by old slot)."""
        idx = np.array(idx, dtype=np.int32, order="C")
        W = np.array(self._store(W, dtype), order="C")
        K, F = idx.shape
        mm = None if m is None else np.array(m, dtype=np.float64, order="C")
        mask = np.empty(K * F, dtype=np.uint8)
        n = ctypes.c_int64(0)
        rc = self.lib.haste_oracle_rewire(K, G, F, H, dtype, _ptr(idx), _ptr(W), _ptr(mm), rho, int(init_random),
                                          seed, ctypes.byref(n), _ptr(mask))
        self._check(rc, "rewire")
        return idx, W, mm, int(n.value), mask.reshape(K, F).astype(bool)

    def group_labels(self, E, G, beta, iters, seed):
        """Alg. 2 on int8 embeddings E [N, D]: (order [N], group sizes, cluster [N])."""
        E = np.ascontiguousarray(E, dtype=np.int8)
        N, D = E.shape
        order = np.empty(N, dtype=np.int32)
        gsize = np.empty(N, dtype=np.int32)
        cl = np.empty(N, dtype=np.int32)
        ng = ctypes.c_int64(0)
        rc = self.lib.haste_oracle_group_labels(N, D, _ptr(E), G, beta, iters, seed, _ptr(order), _ptr(gsize),
                                                ctypes.byref(ng), _ptr(cl))
        self._check(rc, "group_labels")
        return order, gsize[:ng.value].copy(), cl

    def bwd_x(self, idx, W, dY, G, F_s, dtype, b0=0, b1=None):
        """dX[b1-b0, F_s] in fp64 for rows [b0, b1)."""
        W, dY = self._store(W, dtype), self._store(dY, dtype)
        idx = self._c(idx, np.int32)
        L, F_in = W.shape
        B = dY.shape[0]
        b1 = B if b1 is None else b1
        dX = np.empty((b1 - b0, F_s), dtype=np.float64)
        rc = self.lib.haste_oracle_bwd_x(B, F_s, L, G, F_in, dtype, _ptr(idx), _ptr(W), _ptr(dY), b0, b1, _ptr(dX))
        self._check(rc, "bwd_x")
        return dX

    # ---- dense head -----------------------------------------------------------------------
    def head_fwd(self, X, Wh, bias_h, dtype, h0=0, h1=None):
        X, Wh = self._store(X, dtype), self._store(Wh, dtype)
        bias_h = self._c(bias_h, np.float32)
        B, F_s = X.shape
        H = Wh.shape[0]
        h1 = H if h1 is None else h1
        Y = np.empty((B, h1 - h0), dtype=np.float64)
        rc = self.lib.haste_oracle_head_fwd(B, F_s, H, dtype, _ptr(X), _ptr(Wh), _ptr(bias_h), h0, h1, _ptr(Y))
        self._check(rc, "head_fwd")
        return Y

    def head_bwd_w(self, X, dYh, dtype, h0=0, h1=None):
        X, dYh = self._store(X, dtype), self._store(dYh, dtype)
        B, F_s = X.shape
        H = dYh.shape[1]
        h1 = H if h1 is None else h1
        dWh = np.empty((h1 - h0, F_s), dtype=np.float64)
        rc = self.lib.haste_oracle_head_bwd_w(B, F_s, H, dtype, _ptr(X), _ptr(dYh), h0, h1, _ptr(dWh))
        self._check(rc, "head_bwd_w")
        return dWh

    def head_bwd_x(self, Wh, dYh, dtype, b0=0, b1=None):
        Wh, dYh = self._store(Wh, dtype), self._store(dYh, dtype)
        H, F_s = Wh.shape
        B = dYh.shape[0]
        b1 = B if b1 is None else b1
        dX = np.empty((b1 - b0, F_s), dtype=np.float64)
        rc = self.lib.haste_oracle_head_bwd_x(B, F_s, H, dtype, _ptr(Wh), _ptr(dYh), b0, b1, _ptr(dX))
        self._check(rc, "head_bwd_x")
        return dX


_default: Optional[Oracle] = None


def get() -> Oracle:
    """The oracle built from ``haste_oracle.c`` (built on first use if missing)."""
    global _default
    if _default is None:
        if not os.path.exists(LIB):
            build()
        _default = Oracle(LIB)
    return _default
