"""GPU parity of the momentum-step entry points (through the C ABI) against the fp64 CPU oracle.

haste_sgd_momentum applies one step of SGD with momentum to any weight array; haste_fwd_bce_sgd
forms dY = sigmoid(z) - T and applies that step to W with the backward-weight product of dY,
without storing dW.  The oracle composes its forward, BCE gradient, backward-weight product and
momentum step in fp64.  Beyond the tolerance checks, the fused call must equal haste_fwd_bce
followed by haste_sgd_momentum bit for bit (same fp32 operations in the same order).
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import TOL, host_f32, oracle_fwd_bce, out_tensor, rand_pos, rel_err, say, skewed_pos, to_dev

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


def _sync():
    import torch
    torch.cuda.synchronize()


def _check(name, got, ref, tol):
    e = rel_err(got, ref)
    say(f"    {name:<10s} rel_inf_err={e:.3e} (tol {tol:.0e})")
    assert e <= tol, f"{name}: {e:.3e} > {tol:.0e}"


@pytest.mark.parametrize("n,dt,inplace,wd,zero_grad", [
    (4096, BF16, False, 0.0, False), (4099, BF16, True, 1e-3, False), (1000, F32, False, 0.01, False),
    (77, F32, True, 0.0, False), (4096, BF16, False, 5e-4, True)])
def test_sgd_momentum_elementwise(hs, orc, n, dt, inplace, wd, zero_grad):
    import torch
    say(f"[sgd] n={n} dtype={dt} inplace={inplace} wd={wd} zero_grad={zero_grad}")
    rng = np.random.default_rng(n + dt)
    W = rng.standard_normal(n).astype(np.float32)
    Ws = synth.bf16_bits(W) if dt == BF16 else W
    g = np.zeros(n, np.float32) if zero_grad else rng.standard_normal(n).astype(np.float32)
    m0 = (0.1 * rng.standard_normal(n)).astype(np.float32)
    opt = hs.sgd_opts(0.05, 0.9, wd)
    Wd, gd, md = to_dev(Ws), to_dev(g), to_dev(m0)
    out = Wd if inplace else out_tensor((n,), dt)
    hs.haste_sgd_momentum(n, dt, Wd, None if zero_grad else gd, md, opt, out)
    _sync()
    Wn_ref, m_ref = orc.sgd_momentum(Ws, g.astype(np.float64), m0.astype(np.float64), 0.05, 0.9, wd, dt)
    _check("m", md.cpu().numpy(), m_ref, TOL[F32])
    _check("W_next", host_f32(out, dt), Wn_ref, TOL[dt])


CASES = [
    # name, B, F_s, L, G, F_in, dtype, P, bias, dbias   (fused: bf16, G % 16 == 0, F_s <= 1024; P < 0:
    # skewed rows of up to -P positives, bucketed by the pre-pass)
    ("fused_g32_f64", 40, 256, 2048, 32, 64, BF16, 6, False, False),
    ("fused_g16_ragged_b33", 33, 768, 4096, 16, 64, BF16, 5, True, True),
    ("fused_g64_f128", 70, 768, 4096, 64, 128, BF16, 8, True, True),
    ("fused_g32_f32_b300", 300, 512, 8192, 32, 32, BF16, 8, False, True),
    ("fused_fs1024", 40, 1024, 2048, 32, 64, BF16, 4, False, False),
    ("fused_p150_skewed", 64, 768, 4096, 32, 64, BF16, -150, True, True),
    ("fused_p200_skewed_f128", 48, 512, 4096, 32, 128, BF16, -200, False, True),
    ("composed_g8", 70, 768, 3072, 8, 32, BF16, 5, True, True),
    # small groups: dW from the dense backward-weight (G = 1, 2) in the workspace, then the step
    ("composed_g1", 40, 768, 2050, 1, 64, BF16, 6, True, True),
    ("composed_g2_f128", 33, 512, 4096, 2, 128, BF16, 5, False, True),
    ("composed_f32_g8", 32, 256, 4096, 8, 32, F32, 5, False, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fwd_bce_sgd(hs, orc, case):
    import torch
    name, B, F_s, L, G, F_in, dt, P, with_bias, with_db = case
    say(f"[fwd_bce_sgd] {name}: B={B} F_s={F_s} L={L} G={G} F_in={F_in} dtype={dt} P={P}")
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=dt, wid=700 + CASES.index(case))
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    rng = np.random.default_rng(wl.wid)
    bias = rng.standard_normal(L).astype(np.float32) if with_bias else None
    pos = skewed_pos(rng, B, L, -P) if P < 0 else rand_pos(rng, B, L, P)
    m0 = (0.01 * rng.standard_normal((L, F_in))).astype(np.float32)
    lr, mu, wd = 0.1, 0.9, 1e-4
    desc = hs.make_desc(B, F_s, L, G, F_in, dt)
    Xd, idxd, Wd, bd, posd = to_dev(X), to_dev(idx), to_dev(W), to_dev(bias), to_dev(pos)
    dY = out_tensor((B, L), dt)
    m = to_dev(m0)
    Wn = out_tensor((L, F_in), dt)
    db = torch.empty((L,), dtype=torch.float32, device="cuda") if with_db else None
    opt = hs.sgd_opts(lr, mu, wd)
    hs.haste_fwd_bce_sgd(desc, Xd, idxd, Wd, bd, posd, dY, opt, m, Wn, db,
                         hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE_SGD)))
    _sync()
    dY_ref, dW_ref, db_ref = oracle_fwd_bce(orc, X, idx, W, bias, pos, G, F_in, dt)
    Wn_ref, m_ref = orc.sgd_momentum(W, dW_ref, m0.astype(np.float64), lr, mu, wd, dt)
    _check("dY", host_f32(dY, dt), dY_ref, TOL[dt])
    _check("m", m.cpu().numpy(), m_ref, TOL[dt])
    _check("W_next", host_f32(Wn, dt), Wn_ref, TOL[dt])
    if with_db:
        _check("dbias", db.cpu().numpy(), db_ref, TOL[dt])
    # the fused step equals haste_fwd_bce + haste_sgd_momentum, bit for bit
    dW2 = torch.empty((L, F_in), dtype=torch.float32, device="cuda")
    dY2 = out_tensor((B, L), dt)
    m2 = to_dev(m0)
    Wn2 = out_tensor((L, F_in), dt)
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, bd, posd, dY2, dW2, None, 0,
                     hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE)))
    hs.haste_sgd_momentum(L * F_in, dt, Wd, dW2, m2, opt, Wn2)
    _sync()
    assert bool((dY2 == dY).all()), "dY differs from haste_fwd_bce"
    assert bool((m2 == m).all()) and bool((Wn2 == Wn).all()), "fused step differs from haste_fwd_bce + haste_sgd_momentum"


def test_fwd_bce_sgd_edges(hs):
    import torch
    dt = BF16
    L, F_in = 4096, 64
    W = to_dev(synth.bf16_bits(np.random.default_rng(1).standard_normal((L, F_in)).astype(np.float32)))
    m = torch.full((L, F_in), 0.5, dtype=torch.float32, device="cuda")
    Wn = out_tensor((L, F_in), dt)
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    opt = hs.sgd_opts(0.1, 0.5, 0.0)
    # no rows: a zero gradient, so m = 0.5 * m and W_next = W - 0.1 m
    d0 = hs.make_desc(0, 768, L, 32, F_in, dt)
    hs.haste_fwd_bce_sgd(d0, dummy, dummy, W, None, None, dummy, opt, m, Wn, None,
                         hs.workspace(hs.haste_workspace_bytes(d0, hs.HASTE_OP_FWD_BCE_SGD)))
    _sync()
    assert float((m - 0.25).abs().max()) == 0.0
    Wf = W.view(torch.bfloat16).float()
    assert float((Wn.view(torch.bfloat16).float() - (Wf - 0.025).bfloat16().float()).abs().max()) == 0.0
    d = hs.make_desc(8, 768, L, 32, F_in, dt)
    ws = hs.workspace(hs.haste_workspace_bytes(d, hs.HASTE_OP_FWD_BCE_SGD))
    with pytest.raises(hs.HasteError):   # W_next overlapping W
        hs.haste_fwd_bce_sgd(d, dummy, dummy, W, None, None, dummy, opt, m, W, None, ws)
    with pytest.raises(hs.HasteError):   # momentum out of range
        hs.haste_fwd_bce_sgd(d, dummy, dummy, W, None, None, dummy, hs.sgd_opts(0.1, 1.0), m, Wn, None, ws)
    with pytest.raises(hs.HasteError):   # rows of more positives than the queried workspace provides for
        pos = torch.zeros((8, 2000), dtype=torch.int32, device="cuda")
        hs.haste_fwd_bce_sgd(d, dummy, dummy, W, None, pos, dummy, opt, m, Wn, None, ws)


def test_fwd_bce_sgd_large(hs, orc):
    """The 2.95M-label layer as the benchmark launches it: label ranges against the oracle and the
    whole m and W_next against haste_fwd_bce + haste_sgd_momentum."""
    import torch
    wl = synth.WORKLOADS["l2949k_g32_h65k"]
    dt = wl.dtype
    say(f"[fwd_bce_sgd workload] {wl.name}")
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    tail, _ = synth.positive_neurons(wl, synth.draw_positives(wl), synth.draw_perm(wl))
    pos = synth.pos_matrix(tail, wl.B)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, dt)
    Xd, idxd, Wd, posd = to_dev(X), to_dev(idx), to_dev(W), to_dev(pos)
    dY = out_tensor((wl.B, wl.L), dt)
    m = torch.zeros((wl.L, wl.F_in), dtype=torch.float32, device="cuda")
    Wn = out_tensor((wl.L, wl.F_in), dt)
    lr, mu, wd = 0.5, 0.9, 0.0
    opt = hs.sgd_opts(lr, mu, wd)
    hs.haste_fwd_bce_sgd(desc, Xd, idxd, Wd, None, posd, dY, opt, m, Wn, None,
                         hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE_SGD)))
    _sync()
    Xf = synth.to_f64(X, dt).astype(np.float32)
    n = 4096
    for r0 in sorted({0, (wl.L // 2) // wl.G * wl.G, wl.L - n}):
        r1 = r0 + n
        say(f"  labels [{r0}, {r1})")
        dY_ref = orc.bce_grad(orc.fwd(X, idx, W, None, wl.G, dt, r0, r1), pos - r0)
        dW_ref, _ = orc.bwd_w(Xf, idx[r0 // wl.G:r1 // wl.G], dY_ref.astype(np.float32), wl.G, wl.F_in, F32)
        Wn_ref, m_ref = orc.sgd_momentum(W[r0:r1], dW_ref, np.zeros_like(dW_ref), lr, mu, wd, dt)
        _check("m", m[r0:r1].cpu().numpy(), m_ref, TOL[dt])
        _check("W_next", host_f32(Wn[r0:r1].contiguous(), dt), Wn_ref, TOL[dt])
    dW2 = torch.empty((wl.L, wl.F_in), dtype=torch.float32, device="cuda")
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, None, posd, dY, dW2, None, 0,
                     hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE)))
    m2 = torch.zeros_like(m)
    Wn2 = out_tensor((wl.L, wl.F_in), dt)
    hs.haste_sgd_momentum(wl.L * wl.F_in, dt, Wd, dW2, m2, opt, Wn2)
    _sync()
    assert bool((m2 == m).all()) and bool((Wn2 == Wn).all()), "fused step differs from the composed calls"
