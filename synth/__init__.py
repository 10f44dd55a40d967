"""Seeded synthetic inputs for the group-shared fixed fan-in output layer.

This module only *draws* inputs.  It holds none of the layer's arithmetic
(no logits, no gradients of the layer): it is shared by the CPU oracle's
tests and by the GPU path's tests and benchmark, so that both consume the
identical bytes.

Recipe (one NumPy PCG64 child stream per buffer, seeded by
``SeedSequence([seed, workload_id, buffer_id(, chunk)])``):

* X ~ N(0, 1) (post-LayerNorm-like encoder features), W ~ N(0, 1/F_in),
  W_head ~ N(0, 1/F_s); drawn in fp32, rounded to bf16 with
  round-to-nearest-even for bf16 workloads.
* idx: for every group, F_in distinct features drawn uniformly without
  replacement from [0, F_s), then sorted (group-shared supports of
  Section 3.1, one index row per group).
* positives: per batch row, a fixed number of distinct label ids drawn from a
  truncated Zipf(s) law over ranks 1..N (N = head + tail labels), rank r is
  label id r-1; ids below H are head labels (the most frequent ones,
  Section 3.3), the rest are tail labels.  Tail label u is stored at output
  neuron ``inv_perm[u - H]`` where ``perm`` is a seeded permutation (labels
  assigned to groups by contiguous blocks of a random order).
* dY: the binary cross-entropy gradient sigmoid(z) - y of the objective in
  Section 3.3, rounded to bf16.  ``z`` is either supplied by the caller (for
  example logits from the oracle) or a stand-in drawn as N(0, 1), which is
  the marginal law of the layer's logits under this recipe
  (Var = F_in * 1 * 1/F_in).
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Optional

import numpy as np

# dtype codes shared with the C interfaces
DT_F32 = 0
DT_BF16 = 1

# buffer ids of the per-buffer seed streams
_BUF_X, _BUF_W, _BUF_IDX, _BUF_BIAS, _BUF_POS, _BUF_Z, _BUF_WH, _BUF_PERM, _BUF_ZH, _BUF_DY = range(10)


# --------------------------------------------------------------------------------------------
# bf16 encoding (storage format only)
# --------------------------------------------------------------------------------------------
def bf16_bits(a) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round-to-nearest-even.  Inputs must be finite."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_to_f32(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_f64(a, dtype: int) -> np.ndarray:
    """Decode a stored buffer (fp32 or bf16 bits) to fp64 exactly."""
    if dtype == DT_BF16:
        return bf16_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


# --------------------------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int            # workload id, part of every seed
    B: int
    F_s: int
    L: int              # tail labels
    G: int
    F_in: int
    H: int = 0          # dense-head labels computed (0 = no head)
    dtype: int = DT_BF16
    n_pos: int = 5      # positives per row
    zipf_s: float = 1.1
    zipf_H: Optional[int] = None   # head ids used for the Zipf ranks (defaults to H)
    permute: bool = False          # tail labels grouped by contiguous blocks of a seeded permutation
    bias: bool = False             # explicit zero bias vector (exercises the bias path)
    dy_normal: bool = False        # dY ~ N(0,1) instead of the BCE gradient

    @property
    def K(self) -> int:
        return self.L // self.G

    @property
    def head_ids(self) -> int:
        return self.H if self.zipf_H is None else self.zipf_H

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # tiny fp32 layer, no head, zero bias, dY ~ N(0,1), seed 0
    "tiny_f32": Workload("tiny_f32", 1, B=32, F_s=256, L=4096, G=8, F_in=32, dtype=DT_F32,
                         bias=True, dy_normal=True),
    # 131K-label bf16 tail, identity label order, 5 Zipf(1.1) positives
    "l131k_g16": Workload("l131k_g16", 2, B=128, F_s=768, L=131072, G=16, F_in=64),
    # 655K-label tail + 16K dense head (Amazon-670K-shaped)
    "l655k_g32_h16k": Workload("l655k_g32_h16k", 3, B=256, F_s=768, L=655360, G=32, F_in=128,
                               H=16384, permute=True),
    # group-size sweep on a fixed 655K-label layer (X, W, dY as above; one idx per G)
    "gsweep_g1": Workload("gsweep_g1", 4, B=256, F_s=768, L=655360, G=1, F_in=64, zipf_H=16384, permute=True),
    "gsweep_g4": Workload("gsweep_g4", 4, B=256, F_s=768, L=655360, G=4, F_in=64, zipf_H=16384, permute=True),
    "gsweep_g16": Workload("gsweep_g16", 4, B=256, F_s=768, L=655360, G=16, F_in=64, zipf_H=16384, permute=True),
    "gsweep_g64": Workload("gsweep_g64", 4, B=256, F_s=768, L=655360, G=64, F_in=64, zipf_H=16384, permute=True),
    # 2.95M-label tail + 65K dense head (Amazon-3M-shaped), 8 Zipf(1.05) positives
    "l2949k_g32_h65k": Workload("l2949k_g32_h65k", 5, B=512, F_s=768, L=2949120, G=32, F_in=64,
                                H=65536, n_pos=8, zipf_s=1.05, permute=True),
}


def _rng(seed: int, wl: Workload, buf: int, chunk: Optional[int] = None) -> np.random.Generator:
    key = [seed, wl.wid, buf] if chunk is None else [seed, wl.wid, buf, chunk]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def _store(a_f32: np.ndarray, dtype: int) -> np.ndarray:
    return bf16_bits(a_f32) if dtype == DT_BF16 else np.ascontiguousarray(a_f32, dtype=np.float32)


def draw_X(wl: Workload, seed: int = 0) -> np.ndarray:
    r = _rng(seed, wl, _BUF_X)
    return _store(r.standard_normal((wl.B, wl.F_s), dtype=np.float32), wl.dtype)


def draw_W(wl: Workload, seed: int = 0, chunk_rows: int = 1 << 20) -> np.ndarray:
    """W[L, F_in] ~ N(0, 1/F_in).  Row chunks use their own streams."""
    out = np.empty((wl.L, wl.F_in), dtype=np.uint16 if wl.dtype == DT_BF16 else np.float32)
    scale = np.float32(1.0 / np.sqrt(wl.F_in))
    for c, r0 in enumerate(range(0, wl.L, chunk_rows)):
        r1 = min(wl.L, r0 + chunk_rows)
        r = _rng(seed, wl, _BUF_W, c)
        out[r0:r1] = _store(r.standard_normal((r1 - r0, wl.F_in), dtype=np.float32) * scale, wl.dtype)
    return out


def draw_idx(wl: Workload, seed: int = 0, n_rows: Optional[int] = None, chunk_rows: int = 8192) -> np.ndarray:
    """idx[n_rows, F_in] int32: per row F_in distinct features from [0, F_s), sorted.

    n_rows defaults to K = L/G (group-shared); pass L for a per-label (G = 1) index.
    """
    n = wl.K if n_rows is None else n_rows
    out = np.empty((n, wl.F_in), dtype=np.int32)
    for c, r0 in enumerate(range(0, n, chunk_rows)):
        r1 = min(n, r0 + chunk_rows)
        # the group size is part of the key: every G of a sweep gets its own supports
        r = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wl.wid, _BUF_IDX, wl.G, c])))
        keys = r.random((r1 - r0, wl.F_s), dtype=np.float32)
        if wl.F_in < wl.F_s:
            pick = np.argpartition(keys, wl.F_in - 1, axis=1)[:, : wl.F_in]
        else:
            pick = np.broadcast_to(np.arange(wl.F_s), keys.shape)
        out[r0:r1] = np.sort(pick, axis=1).astype(np.int32)
    return out


def draw_bias(wl: Workload) -> Optional[np.ndarray]:
    return np.zeros(wl.L, dtype=np.float32) if wl.bias else None


def draw_perm(wl: Workload, seed: int = 0) -> np.ndarray:
    """perm[n] = tail label id stored at output neuron n (identity if not permuted)."""
    if not wl.permute:
        return np.arange(wl.L, dtype=np.int64)
    return _rng(seed, wl, _BUF_PERM).permutation(wl.L).astype(np.int64)


def draw_positives(wl: Workload, seed: int = 0) -> np.ndarray:
    """[B, n_pos] distinct global label ids per row, truncated Zipf(s) over ranks 1..N."""
    N = wl.head_ids + wl.L
    w = np.arange(1, N + 1, dtype=np.float64) ** (-wl.zipf_s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    r = _rng(seed, wl, _BUF_POS)
    out = np.empty((wl.B, wl.n_pos), dtype=np.int64)
    for b in range(wl.B):
        got: list = []
        while len(got) < wl.n_pos:
            u = r.random()
            lab = int(np.searchsorted(cdf, u, side="right"))
            lab = min(lab, N - 1)
            if lab not in got:
                got.append(lab)
        out[b] = got
    return out


def positive_neurons(wl: Workload, positives: np.ndarray, perm: np.ndarray):
    """Split positives into (tail (b, neuron) pairs, head (b, id) pairs)."""
    inv = np.empty_like(perm)
    inv[perm] = np.arange(perm.size, dtype=perm.dtype)
    tail, head = [], []
    for b in range(positives.shape[0]):
        for u in positives[b]:
            u = int(u)
            if u >= wl.head_ids:
                tail.append((b, int(inv[u - wl.head_ids])))
            elif u < wl.H:
                head.append((b, u))
    return (np.array(tail, dtype=np.int64).reshape(-1, 2), np.array(head, dtype=np.int64).reshape(-1, 2))


def pos_matrix(pairs: np.ndarray, B: int, P: Optional[int] = None) -> np.ndarray:
    """(b, column) pairs -> [B, P] int32 column lists per row, padded with -1 (P = longest row)."""
    rows: list = [[] for _ in range(B)]
    for b, n in np.asarray(pairs).reshape(-1, 2):
        rows[int(b)].append(int(n))
    if P is None:
        P = max((len(r) for r in rows), default=0)
    out = np.full((B, P), -1, dtype=np.int32)
    for b, r in enumerate(rows):
        out[b, :len(r)] = r[:P]
    return out


def bce_grad(wl: Workload, pos_pairs: np.ndarray, n_cols: int, seed: int = 0,
             logits: Optional[np.ndarray] = None, buf: int = _BUF_Z, chunk_rows: int = 8) -> np.ndarray:
    """dY[B, n_cols] = bf16(sigmoid(z) - y).  z = supplied logits or N(0,1) stand-ins."""
    out = np.empty((wl.B, n_cols), dtype=np.uint16)
    by_row: dict = {}
    for b, n in pos_pairs:
        by_row.setdefault(int(b), []).append(int(n))
    for c, r0 in enumerate(range(0, wl.B, chunk_rows)):
        r1 = min(wl.B, r0 + chunk_rows)
        if logits is None:
            z = _rng(seed, wl, buf, c).standard_normal((r1 - r0, n_cols), dtype=np.float32)
        else:
            z = np.asarray(logits[r0:r1], dtype=np.float64)
        s = (1.0 / (1.0 + np.exp(-z))).astype(np.float32)
        for b in range(r0, r1):
            for n in by_row.get(b, ()):
                s[b - r0, n] -= np.float32(1.0)
        out[r0:r1] = bf16_bits(s)
    return out


def draw_dY(wl: Workload, seed: int = 0, logits: Optional[np.ndarray] = None,
            positives: Optional[np.ndarray] = None, perm: Optional[np.ndarray] = None) -> np.ndarray:
    """Tail upstream gradient dY[B, L] in the workload's dtype."""
    if wl.dy_normal:
        return _store(_rng(seed, wl, _BUF_DY).standard_normal((wl.B, wl.L), dtype=np.float32), wl.dtype)
    if positives is None:
        positives = draw_positives(wl, seed)
    if perm is None:
        perm = draw_perm(wl, seed)
    tail, _ = positive_neurons(wl, positives, perm)
    return bce_grad(wl, tail, wl.L, seed, logits, _BUF_Z)


def draw_W_head(wl: Workload, seed: int = 0) -> np.ndarray:
    r = _rng(seed, wl, _BUF_WH)
    a = r.standard_normal((wl.H, wl.F_s), dtype=np.float32) * np.float32(1.0 / np.sqrt(wl.F_s))
    return _store(a, wl.dtype)


def draw_dY_head(wl: Workload, seed: int = 0, logits: Optional[np.ndarray] = None,
                 positives: Optional[np.ndarray] = None, perm: Optional[np.ndarray] = None) -> np.ndarray:
    if positives is None:
        positives = draw_positives(wl, seed)
    if perm is None:
        perm = draw_perm(wl, seed)
    _, head = positive_neurons(wl, positives, perm)
    return bce_grad(wl, head, wl.H, seed, logits, _BUF_ZH)


def small(name: str = "small", B: int = 8, F_s: int = 40, L: int = 48, G: int = 4, F_in: int = 6,
          H: int = 0, dtype: int = DT_F32, wid: int = 100, **kw) -> Workload:
    """An ad-hoc small workload (tests)."""
    return Workload(name, wid, B=B, F_s=F_s, L=L, G=G, F_in=F_in, H=H, dtype=dtype, **kw)
