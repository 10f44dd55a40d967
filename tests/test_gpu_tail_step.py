"""GPU checks of haste_tail_step (through the C ABI): the tail's training pass in one call must
equal haste_fwd_bce followed by haste_bwd_x bit for bit (dY, dW, dbias, dX), both where the forward
kernel hands the transposed weights to backward-feature (groups of 32 labels) and where the call
composes the two; those two calls are themselves checked against the fp64 oracle elsewhere."""
import numpy as np
import pytest

import synth
from gpu_helpers import out_tensor, rand_pos, say, to_dev

pytestmark = pytest.mark.gpu
F32, BF16 = synth.DT_F32, synth.DT_BF16


@pytest.fixture(scope="module")
def hs():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2606_01117_amd as m
    return m


def _both(hs, wl, X, idx, W, bias, pos, beta_dx):
    import torch
    B, L, F_in, F_s, dt = wl.B, wl.L, wl.F_in, wl.F_s, wl.dtype
    desc = hs.make_desc(B, F_s, L, wl.G, F_in, dt)
    Xd, idxd, Wd, bd = to_dev(X), to_dev(idx), to_dev(W), to_dev(bias)
    posd = to_dev(pos) if pos.shape[1] else None
    outs = []
    for fused in (True, False):
        dY = out_tensor((B, L), dt)
        dW = torch.empty((L, F_in), dtype=torch.float32, device="cuda")
        db = torch.empty((L,), dtype=torch.float32, device="cuda") if bias is not None else None
        dX = torch.full((B, F_s), 0.25, dtype=torch.float32, device="cuda")
        if fused:
            ws = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP))
            hs.haste_tail_step(desc, Xd, idxd, Wd, bd, posd, dY, dW, db, 0, dX, beta_dx, ws)
        else:
            hs.haste_fwd_bce(desc, Xd, idxd, Wd, bd, posd, dY, dW, db, 0,
                             hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE)))
            hs.haste_bwd_x(desc, idxd, Wd, dY, dX, beta_dx, hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_X)))
        torch.cuda.synchronize()
        outs.append((dY, dW, db, dX))
    (a, b) = outs
    assert bool((a[0].view(torch.int16) == b[0].view(torch.int16)).all()) if dt == BF16 else bool((a[0] == b[0]).all()), "dY"
    assert bool((a[1] == b[1]).all()), "dW"
    if bias is not None:
        assert bool((a[2] == b[2]).all()), "dbias"
    assert bool((a[3] == b[3]).all()), "dX"
    return a


CASES = [
    # name, B, F_s, L, G, F_in, dtype, P, bias, beta_dx
    ("g32_f64", 64, 768, 4096, 32, 64, BF16, 8, False, 0),
    ("g32_f64_bias_acc", 40, 768, 8192, 32, 64, BF16, 5, True, 1),
    ("g32_f32_ragged_b33", 33, 256, 2048, 32, 32, BF16, 3, False, 0),
    ("g32_f128", 70, 768, 4096, 32, 128, BF16, 8, True, 0),
    ("g32_small_fs", 96, 128, 4096, 32, 64, BF16, 4, False, 1),
    ("g32_f64_p150_bucketed", 64, 768, 8192, 32, 64, BF16, 150, True, 1),
    ("g32_fs896", 40, 896, 4096, 32, 64, BF16, 6, False, 0),   # X^T past the prefetch; bwd_x takes F_s <= 910
    ("composed_g16", 64, 768, 4096, 16, 64, BF16, 8, False, 0),
    ("composed_f32", 32, 256, 4096, 8, 32, F32, 5, True, 1),
    # small groups: the forward forms the gradient as it stores, then the dense backward-weight
    # (G = 1, 2) or the gather kernel (G = 4) and the scattered-tile backward-feature
    ("small_g1", 40, 768, 2050, 1, 64, BF16, 6, True, 1),
    ("small_g2_f128", 33, 512, 4096, 2, 128, BF16, 5, False, 0),
    ("small_g4", 64, 768, 4096, 4, 64, BF16, 8, True, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_tail_step_equals_the_two_calls(hs, case):
    name, B, F_s, L, G, F_in, dt, P, with_bias, beta_dx = case
    say(f"[tail_step] {name}: B={B} F_s={F_s} L={L} G={G} F_in={F_in} P={P} beta_dx={beta_dx}")
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=dt, wid=900 + CASES.index(case))
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    rng = np.random.default_rng(wl.wid)
    bias = rng.standard_normal(L).astype(np.float32) if with_bias else None
    _both(hs, wl, X, idx, W, bias, rand_pos(rng, B, L, P), beta_dx)


def test_tail_step_large(hs):
    """The 2.95M-label layer of the benchmark, its own positives."""
    wl = synth.WORKLOADS["l2949k_g32_h65k"]
    say(f"[tail_step workload] {wl.name}")
    rng = np.random.default_rng(5)
    _both(hs, wl, synth.draw_X(wl), synth.draw_idx(wl), synth.draw_W(wl), None, rand_pos(rng, wl.B, wl.L, 8), 0)


def test_tail_step_workspace_checked(hs):
    import torch
    d = hs.make_desc(64, 768, 4096, 32, 64, BF16)
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    need = hs.haste_workspace_bytes(d, hs.HASTE_OP_TAIL_STEP)
    assert need >= hs.haste_workspace_bytes(d, hs.HASTE_OP_BWD_X) + hs.haste_workspace_bytes(d, hs.HASTE_OP_FWD_BCE)
    with pytest.raises(hs.HasteError):
        hs.haste_tail_step(d, dummy, dummy, dummy, None, None, dummy, dummy, None, 0, dummy, 0,
                           hs.workspace(need - 256))


@pytest.mark.parametrize("case", [("g32_f64", 64, 768, 4096, 32, 64, 8, True), ("g32_f128", 70, 768, 4096, 32, 128, 5, False),
                                  ("g32_f64_p120_bucketed", 50, 512, 4096, 32, 64, 120, True),
                                  ("composed_g16", 48, 512, 4096, 16, 64, 4, False),
                                  ("composed_g1", 40, 768, 2050, 1, 64, 6, True),
                                  ("composed_g2", 33, 256, 1030, 2, 32, 3, False)], ids=lambda c: c[0])
def test_tail_step_sgd_equals_the_two_calls(hs, case):
    import torch
    name, B, F_s, L, G, F_in, P, with_bias = case
    say(f"[tail_step_sgd] {name}: B={B} F_s={F_s} L={L} G={G} F_in={F_in} P={P}")
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=BF16, wid=950 + F_in + G)
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    rng = np.random.default_rng(wl.wid)
    bias = rng.standard_normal(L).astype(np.float32) if with_bias else None
    m0 = rng.standard_normal((L, F_in)).astype(np.float32)
    pos = rand_pos(rng, B, L, P)
    desc = hs.make_desc(B, F_s, L, G, F_in, BF16)
    Xd, idxd, Wd, bd, posd = to_dev(X), to_dev(idx), to_dev(W), to_dev(bias), to_dev(pos)
    opt = hs.sgd_opts(0.05, 0.9, 1e-4)
    outs = []
    for fused in (True, False):
        dY = out_tensor((B, L), BF16)
        m = to_dev(m0)
        Wn = torch.empty_like(Wd)
        db = torch.empty((L,), dtype=torch.float32, device="cuda") if with_bias else None
        dX = torch.zeros((B, F_s), dtype=torch.float32, device="cuda")
        if fused:
            hs.haste_tail_step_sgd(desc, Xd, idxd, Wd, bd, posd, dY, db, opt, m, Wn, dX, 0,
                                   hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP_SGD)))
        else:
            hs.haste_fwd_bce_sgd(desc, Xd, idxd, Wd, bd, posd, dY, opt, m, Wn, db,
                                 hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE_SGD)))
            hs.haste_bwd_x(desc, idxd, Wd, dY, dX, 0, hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_X)))
        torch.cuda.synchronize()
        outs.append((dY.view(torch.int16), m, Wn.view(torch.int16), db, dX))
    a, b = outs
    for i, what in enumerate(("dY", "velocity", "W_next", "dbias", "dX")):
        if a[i] is not None:
            assert bool((a[i] == b[i]).all()), what
