"""Python binding of libhaste.so: the MI355X (gfx950) group-shared fixed fan-in output layer.

The functions below carry the names of the C ABI in ``include/haste.h`` and only marshal
arguments: torch tensors provide device memory and the current HIP stream, every step of the
layer runs in the library's HIP kernels.  The library must be built (``build.build()``); importing
this package without it raises immediately, there is no fallback implementation.

Layer (paper Section 3.1): labels in contiguous groups of G share one sorted support
idx[k, 0..F_in-1] of input features; label l keeps its own weights W[l, 0..F_in-1].
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libhaste.so")

HASTE_DTYPE_F32 = 0
HASTE_DTYPE_BF16 = 1
(HASTE_OP_FWD, HASTE_OP_BWD_W, HASTE_OP_BWD_X, HASTE_OP_FWD_BCE, HASTE_OP_FWD_BCE_SGD, HASTE_OP_REWIRE,
 HASTE_OP_TAIL_STEP, HASTE_OP_TAIL_STEP_SGD) = range(8)
STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "workspace too small", 4: "HIP error"}


class HasteError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class haste_desc_t(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("F_s", ctypes.c_int64), ("L", ctypes.c_int64), ("G", ctypes.c_int64),
                ("F_in", ctypes.c_int64), ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class haste_sgd_t(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("reserved", ctypes.c_int32)]


class haste_group_opts_t(ctypes.Structure):
    _fields_ = [("G", ctypes.c_int64), ("beta", ctypes.c_int64), ("iters", ctypes.c_int64), ("seed", ctypes.c_uint64)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libhaste.so is not built ({LIB_PATH}); run paper_2606_01117_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(haste_desc_t)
    sigs = {
        "haste_fwd": [D, P, P, P, P, P, P, SZ, P],
        "haste_bwd_w": [D, P, P, P, P, P, ctypes.c_int, P, SZ, P],
        "haste_bwd_x": [D, P, P, P, P, ctypes.c_int, P, SZ, P],
        "haste_fwd_bce": [D, P, P, P, P, P, I32, P, P, P, ctypes.c_int, P, SZ, P],
        "haste_fwd_bce_static": [D, P, P, P, P, P, I32, P, P, P, ctypes.c_int, P],
        "haste_bce_grad": [I64, I64, I32, P, P, I32, P, P],
        "haste_fwd_bce_sgd": [D, P, P, P, P, P, I32, P, P, ctypes.POINTER(haste_sgd_t), P, P, P, SZ, P],
        "haste_sgd_momentum": [I64, I32, P, P, P, ctypes.POINTER(haste_sgd_t), P, P],
        "haste_rewire": [D, P, P, P, ctypes.c_double, I32, ctypes.c_uint64, P, P, SZ, P],
        "haste_group_labels": [I64, I64, P, ctypes.POINTER(haste_group_opts_t), P, P, P, P, P, SZ, P],
        "haste_head_fwd": [I64, I64, I64, I32, P, P, P, P, P],
        "haste_tail_step": [D, P, P, P, P, P, I32, P, P, P, ctypes.c_int, P, ctypes.c_int, P, SZ, P],
        "haste_tail_step_sgd": [D, P, P, P, P, P, I32, P, P, ctypes.POINTER(haste_sgd_t), P, P, P, ctypes.c_int, P, SZ,
                                P],
        "haste_head_fwd_bce": [I64, I64, I64, I32, P, P, P, P, I32, P, P],
        "haste_head_bwd": [I64, I64, I64, I32, P, P, P, P, P, ctypes.c_int, P, SZ, P],
        "haste_validate_idx": [D, P, P, P],
        "haste_debug_gather": [D, P, P, I64, I64, P, P],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.haste_workspace_bytes.argtypes = [D, ctypes.c_int]
    lib.haste_workspace_bytes.restype = SZ
    lib.haste_head_workspace_bytes.argtypes = [I64, I64, I64, I32]
    lib.haste_head_workspace_bytes.restype = SZ
    lib.haste_group_workspace_bytes.argtypes = [I64, I64, ctypes.POINTER(haste_group_opts_t)]
    lib.haste_group_workspace_bytes.restype = SZ
    lib.haste_fwd_bce_static_max_bytes.argtypes = []
    lib.haste_fwd_bce_static_max_bytes.restype = SZ
    for name in ("haste_status_str", "haste_last_error", "haste_version"):
        getattr(lib, name).restype = ctypes.c_char_p
    lib.haste_status_str.argtypes = [ctypes.c_int]
    return lib


lib = _load()

# every symbol the header declares
EXPORTS = ("haste_fwd", "haste_bwd_w", "haste_bwd_x", "haste_fwd_bce", "haste_fwd_bce_static",
           "haste_fwd_bce_static_max_bytes", "haste_fwd_bce_sgd", "haste_sgd_momentum",
           "haste_rewire", "haste_group_labels", "haste_group_workspace_bytes", "haste_bce_grad", "haste_head_fwd",
           "haste_head_fwd_bce", "haste_head_bwd", "haste_tail_step", "haste_tail_step_sgd", "haste_workspace_bytes", "haste_head_workspace_bytes", "haste_validate_idx", "haste_debug_gather", "haste_status_str",
           "haste_last_error", "haste_version")


def haste_version() -> str:
    return lib.haste_version().decode()


def haste_status_str(status: int) -> str:
    return lib.haste_status_str(status).decode()


def haste_last_error() -> str:
    return lib.haste_last_error().decode()


def _check(rc: int):
    if rc != 0:
        raise HasteError(rc, haste_last_error())


def make_desc(B: int, F_s: int, L: int, G: int, F_in: int, dtype: int) -> haste_desc_t:
    return haste_desc_t(B, F_s, L, G, F_in, dtype, 0)


# ---- marshalling helpers (torch only supplies memory and the stream) ------------------------
def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors passed to libhaste must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ws(ws):
    if ws is None:
        return None, 0
    if isinstance(ws, tuple):
        return ws
    return ws.data_ptr(), ws.numel() * ws.element_size()


def workspace(nbytes: int, device="cuda"):
    """A caller-owned device workspace of nbytes bytes (None when nothing is needed)."""
    if nbytes == 0:
        return None
    import torch
    return torch.empty(int(nbytes), dtype=torch.uint8, device=device)


# ---- the C ABI ----------------------------------------------------------------------------
def haste_workspace_bytes(desc: haste_desc_t, op: int) -> int:
    return int(lib.haste_workspace_bytes(ctypes.byref(desc), op))


def haste_head_workspace_bytes(B: int, F_s: int, H: int, dtype: int) -> int:
    return int(lib.haste_head_workspace_bytes(B, F_s, H, dtype))


def haste_fwd(desc, X, idx, W, bias, Y, ws=None, stream=None):
    p, n = _ws(ws)
    _check(lib.haste_fwd(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(Y), p, n, _stream(stream)))


def haste_bwd_w(desc, X, idx, dY, dW, dbias=None, beta=0, ws=None, stream=None):
    p, n = _ws(ws)
    _check(lib.haste_bwd_w(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(dY), _ptr(dW), _ptr(dbias), int(beta), p, n,
                           _stream(stream)))


def haste_bwd_x(desc, idx, W, dY, dX, beta=0, ws=None, stream=None):
    p, n = _ws(ws)
    _check(lib.haste_bwd_x(ctypes.byref(desc), _ptr(idx), _ptr(W), _ptr(dY), _ptr(dX), int(beta), p, n,
                           _stream(stream)))


def _npos(pos) -> int:
    return 0 if pos is None else int(pos.shape[1])


def haste_fwd_bce(desc, X, idx, W, bias, pos, dY, dW=None, dbias=None, beta=0, ws=None, stream=None):
    """pos: [B, P] int32 tensor of positive tail column ids (or None for no positives)."""
    p, n = _ws(ws)
    _check(lib.haste_fwd_bce(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(pos), _npos(pos),
                             _ptr(dY), _ptr(dW), _ptr(dbias), int(beta), p, n, _stream(stream)))


def haste_fwd_bce_static(desc, X, idx, W, bias, pos, dY, dW=None, dbias=None, beta=0, stream=None):
    """haste_fwd_bce with the library's own per-device scratch (no workspace, allocates nothing)."""
    _check(lib.haste_fwd_bce_static(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(pos),
                                    _npos(pos), _ptr(dY), _ptr(dW), _ptr(dbias), int(beta), _stream(stream)))


def haste_fwd_bce_static_max_bytes() -> int:
    return int(lib.haste_fwd_bce_static_max_bytes())


def haste_tail_step(desc, X, idx, W, bias, pos, dY, dW, dbias, beta, dX, beta_dx, ws=None, stream=None):
    """haste_fwd_bce followed by haste_bwd_x on its dY (pos: [B, P] int32 tensor or None)."""
    p, n = _ws(ws)
    _check(lib.haste_tail_step(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(pos), _npos(pos),
                               _ptr(dY), _ptr(dW), _ptr(dbias), int(beta), _ptr(dX), int(beta_dx), p, n,
                               _stream(stream)))


def haste_tail_step_sgd(desc, X, idx, W, bias, pos, dY, dbias, opt, m, W_next, dX, beta_dx, ws=None, stream=None):
    """haste_fwd_bce_sgd followed by haste_bwd_x on its dY with the step's W."""
    p, n = _ws(ws)
    _check(lib.haste_tail_step_sgd(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(pos), _npos(pos),
                                   _ptr(dY), _ptr(dbias), ctypes.byref(opt), _ptr(m), _ptr(W_next), _ptr(dX),
                                   int(beta_dx), p, n, _stream(stream)))


def sgd_opts(lr: float, momentum: float, weight_decay: float = 0.0) -> haste_sgd_t:
    return haste_sgd_t(lr, momentum, weight_decay, 0)


def haste_fwd_bce_sgd(desc, X, idx, W, bias, pos, dY, opt, m, W_next, dbias=None, ws=None, stream=None):
    p, n = _ws(ws)
    _check(lib.haste_fwd_bce_sgd(ctypes.byref(desc), _ptr(X), _ptr(idx), _ptr(W), _ptr(bias), _ptr(pos), _npos(pos),
                                 _ptr(dY), _ptr(dbias), ctypes.byref(opt), _ptr(m), _ptr(W_next), p, n,
                                 _stream(stream)))


def haste_sgd_momentum(n, dtype, W, grad, m, opt, W_next, stream=None):
    _check(lib.haste_sgd_momentum(int(n), dtype, _ptr(W), _ptr(grad), _ptr(m), ctypes.byref(opt), _ptr(W_next),
                                  _stream(stream)))


def haste_rewire(desc, idx, W, m, rho, init_random, seed, ws=None, stream=None) -> int:
    """Rewires in place; returns the number of pruned slots."""
    p, n = _ws(ws)
    npr = ctypes.c_int64(0)
    _check(lib.haste_rewire(ctypes.byref(desc), _ptr(idx), _ptr(W), _ptr(m), float(rho), int(init_random),
                            int(seed) & ((1 << 64) - 1), ctypes.byref(npr), p, n, _stream(stream)))
    return int(npr.value)


def group_opts(G: int, beta: int, iters: int, seed: int) -> haste_group_opts_t:
    return haste_group_opts_t(G, beta, iters, seed & ((1 << 64) - 1))


def haste_group_workspace_bytes(N, D, opts) -> int:
    return int(lib.haste_group_workspace_bytes(N, D, ctypes.byref(opts)))


def haste_group_labels(E, opts, order, gsize, n_groups, cluster=None, ws=None, stream=None):
    """E: [N, D] int8 device tensor; n_groups: a 1-element int64 device tensor."""
    p, n = _ws(ws)
    N, D = E.shape
    _check(lib.haste_group_labels(N, D, _ptr(E), ctypes.byref(opts), _ptr(order), _ptr(gsize), _ptr(n_groups),
                                  _ptr(cluster), p, n, _stream(stream)))


def haste_bce_grad(B, N, dtype, Y, pos, dY, stream=None):
    _check(lib.haste_bce_grad(B, N, dtype, _ptr(Y), _ptr(pos), _npos(pos), _ptr(dY), _stream(stream)))


def haste_head_fwd(B, F_s, H, dtype, X, W_head, bias_h, Y_h, stream=None):
    _check(lib.haste_head_fwd(B, F_s, H, dtype, _ptr(X), _ptr(W_head), _ptr(bias_h), _ptr(Y_h), _stream(stream)))


def haste_head_fwd_bce(B, F_s, H, dtype, X, W_head, bias_h, pos, dY_h, stream=None):
    _check(lib.haste_head_fwd_bce(B, F_s, H, dtype, _ptr(X), _ptr(W_head), _ptr(bias_h), _ptr(pos), _npos(pos),
                                  _ptr(dY_h), _stream(stream)))


def haste_head_bwd(B, F_s, H, dtype, X, W_head, dY_h, dW_h, dX, beta_dx=0, ws=None, stream=None):
    p, n = _ws(ws)
    _check(lib.haste_head_bwd(B, F_s, H, dtype, _ptr(X), _ptr(W_head), _ptr(dY_h), _ptr(dW_h), _ptr(dX),
                              int(beta_dx), p, n, _stream(stream)))


def haste_validate_idx(desc, idx, n_bad_rows, stream=None):
    _check(lib.haste_validate_idx(ctypes.byref(desc), _ptr(idx), _ptr(n_bad_rows), _stream(stream)))


def haste_debug_gather(desc, X, idx, k0, nk, out, stream=None):
    _check(lib.haste_debug_gather(ctypes.byref(desc), _ptr(X), _ptr(idx), int(k0), int(nk), _ptr(out),
                                  _stream(stream)))
