"""GPU parity of haste_rewire (Alg. 3, through the C ABI) against the CPU oracle.

Rewiring is integer and selection work on top of fp32 scores that both sides accumulate in the
same order, and its draws come from the same counter-based generator, so the comparison is exact:
the supports, the weights (bit patterns in their storage dtype) and the velocities must match the
oracle's bit for bit.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import out_tensor, say, to_dev

pytestmark = pytest.mark.gpu
F32, BF16 = synth.DT_F32, synth.DT_BF16


@pytest.fixture(scope="module")
def hs():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2606_01117_amd as m
    return m


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


def _run(hs, K, G, F, H, dt, idx, W, m, rho, init, seed):
    import torch
    desc = hs.make_desc(0, H, K * G, G, F, dt)
    idxd, Wd = to_dev(idx), to_dev(W)
    md = to_dev(np.asarray(m, np.float32)) if m is not None else None
    n = hs.haste_rewire(desc, idxd, Wd, md, rho, init, seed,
                        hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_REWIRE)))
    torch.cuda.synchronize()
    Wo = Wd.cpu().numpy()
    Wo = Wo.view(np.uint16) if dt == BF16 else Wo
    return n, idxd.cpu().numpy(), Wo, (md.cpu().numpy() if md is not None else None)


CASES = [
    # name, K, G, F, H, dtype, rho, init_random, with velocity
    ("bf16_g32_f64", 512, 32, 64, 768, BF16, 0.1, 1, True),
    ("bf16_g16_f128_zero", 300, 16, 128, 768, BF16, 0.25, 0, False),
    ("f32_g8_f32", 700, 8, 32, 256, F32, 0.3, 1, True),
    ("bf16_g1_ffi", 2000, 1, 16, 100, BF16, 0.05, 1, False),
    ("bf16_h_eq_f_plus_1", 64, 4, 63, 64, BF16, 0.5, 1, True),
    ("bf16_many_blocks", 4096, 2, 64, 1024, BF16, 0.02, 1, False),
    # the widest support the regrowth takes (four slots per lane)
    ("bf16_g8_f256", 400, 8, 256, 768, BF16, 0.1, 1, True),
    # supports that end inside a 64-slot word: two words with most slots pruned (few free features
    # per draw), and four words over the largest feature bitmap (H = 1024)
    ("bf16_g4_f100_rho09", 300, 4, 100, 512, BF16, 0.9, 1, True),
    ("f32_g2_f200_h1024", 200, 2, 200, 1024, F32, 0.4, 1, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_rewire_exact(hs, orc, case):
    name, K, G, F, H, dt, rho, init, with_m = case
    say(f"[rewire] {name}: K={K} G={G} F={F} H={H} rho={rho} init={init}")
    rng = np.random.default_rng(K * F + G)
    idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
    W = (rng.standard_normal((K * G, F)) / np.sqrt(F)).astype(np.float32)
    W = synth.bf16_bits(W) if dt == BF16 else W
    m = rng.standard_normal((K * G, F)).astype(np.float32) if with_m else None
    seed = 0x1234_5678_9ABC_DEF0 ^ K
    n, idx_g, W_g, m_g = _run(hs, K, G, F, H, dt, idx, W, m, rho, init, seed)
    idx_o, W_o, m_o, n_o, _ = orc.rewire(idx, W, m, G, H, dt, rho, init, seed)
    say(f"    pruned {n} slots")
    assert n == n_o == int(np.floor(K * F * rho))
    assert np.array_equal(idx_g, idx_o), "supports differ from the oracle"
    assert np.array_equal(W_g, W_o), "weights differ from the oracle (bit patterns)"
    if with_m:
        assert np.array_equal(m_g, m_o.astype(np.float32)), "velocities differ from the oracle"


def test_rewire_ties_and_noop(hs, orc):
    K, G, F, H = 1000, 4, 32, 512
    rng = np.random.default_rng(5)
    idx = np.stack([np.sort(rng.choice(H, F, replace=False)) for _ in range(K)]).astype(np.int32)
    Wz = np.zeros((K * G, F), np.uint16)        # all scores equal: the lowest flat indices go first
    n, idx_g, W_g, _ = _run(hs, K, G, F, H, BF16, idx, Wz, None, 0.37, 1, 11)
    idx_o, W_o, _, _, mask = orc.rewire(idx, Wz, None, G, H, BF16, 0.37, 1, 11)
    assert np.array_equal(mask.reshape(-1), np.arange(K * F) < n)
    assert np.array_equal(idx_g, idx_o) and np.array_equal(W_g, W_o)
    W = synth.bf16_bits(rng.standard_normal((K * G, F)).astype(np.float32))
    n, idx_g, W_g, _ = _run(hs, K, G, F, H, BF16, idx, W, None, 0.0, 1, 11)
    assert n == 0 and np.array_equal(idx_g, idx) and np.array_equal(W_g, W)


def test_rewire_large(hs, orc):
    """The 2.95M-label layer's supports and weights, rewired as the benchmark does."""
    wl = synth.WORKLOADS["l2949k_g32_h65k"]
    say(f"[rewire workload] {wl.name}")
    idx, W = synth.draw_idx(wl), synth.draw_W(wl)
    n, idx_g, W_g, _ = _run(hs, wl.K, wl.G, wl.F_in, wl.F_s, wl.dtype, idx, W, None, 0.1, 1, 2024)
    idx_o, W_o, _, n_o, _ = orc.rewire(idx, W, None, wl.G, wl.F_s, wl.dtype, 0.1, 1, 2024)
    say(f"    pruned {n} slots")
    assert n == n_o
    assert np.array_equal(idx_g, idx_o), "supports differ from the oracle"
    assert np.array_equal(W_g, W_o), "weights differ from the oracle"
