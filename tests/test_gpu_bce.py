"""GPU parity of the BCE-gradient entry points (through the C ABI) against the fp64 CPU oracle.

haste_fwd_bce computes dY = sigmoid(z) - T from the layer's own logits z and, when asked, the
backward-weight product of that dY in the same pass; haste_bce_grad applies the same gradient to
stored logits.  The oracle composes its forward, its BCE gradient and its backward-weight product
in fp64.  Beyond the tolerance checks:
* the target rule is checked exactly: dY < 0 exactly where a positive sits (sigmoid never
  reaches 1 at these logits) and dY > 0 elsewhere;
* the fused dW/dbias equal haste_bwd_w applied to the returned dY, bit for bit.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import (TOL, host_f32, oracle_fwd_bce, out_tensor, rand_pos, rel_err, say, skewed_pos, targets,
                         to_dev)

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


def _check(name, got, ref, dtype):
    e = rel_err(got, ref)
    say(f"    {name:<10s} rel_inf_err={e:.3e} (tol {TOL[dtype]:.0e})")
    assert e <= TOL[dtype], f"{name}: {e:.3e} > {TOL[dtype]:.0e}"


CASES = [
    # name, B, F_s, L, G, F_in, dtype, P, bias   (fused: bf16, G % 16 == 0, F_s <= 1024; rows of more
    # than 64 positives are bucketed by a pre-pass)
    ("fused_g32_f64", 40, 256, 2048, 32, 64, BF16, 6, False),
    ("fused_g32_f64_bias", 64, 768, 4096, 32, 64, BF16, 8, True),
    ("fused_g16_ragged_b33", 33, 768, 4096, 16, 64, BF16, 5, False),
    ("fused_g64_f128", 70, 768, 4096, 64, 128, BF16, 8, True),
    ("fused_g48_f32", 97, 384, 48 * 40, 48, 32, BF16, 3, False),
    ("fused_b300_f32", 300, 768, 8192, 32, 32, BF16, 64, True),
    ("fused_b1", 1, 768, 1024, 32, 64, BF16, 2, False),
    ("fused_p0", 50, 512, 2048, 32, 64, BF16, 0, False),
    ("fused_p80_bucketed", 40, 256, 2048, 32, 64, BF16, 80, False),
    ("fused_p200_skewed", 96, 768, 8192, 32, 64, BF16, -200, True),
    ("fused_p130_skewed_f128", 70, 768, 4096, 64, 128, BF16, -130, False),
    ("fused_p90_skewed_g16_f32", 65, 512, 4096, 16, 32, BF16, -90, True),
    # 32 rows of 80 with half in one 512-label span: a cell of about 1280 entries, over one per thread
    ("fused_p80_full_cell", 32, 768, 4096, 32, 64, BF16, -80, False),
    ("fused_fs1024", 70, 1024, 4096, 32, 64, BF16, 8, True),
    ("fused_fs1024_f128_p100", 45, 1024, 2048, 32, 128, BF16, -100, False),
    # small groups: the forward kernel stores the gradient (rows of up to 256 positives, sorted
    # first), else the forward, the gradient pass and backward-weight
    ("composed_g8", 70, 768, 3072, 8, 32, BF16, 5, True),
    ("composed_g4", 64, 512, 1536, 4, 64, BF16, 5, False),
    ("composed_g1_ffi", 37, 768, 1024, 1, 64, BF16, 4, False),
    ("small_g4_p100_skewed", 64, 512, 2048, 4, 64, BF16, -100, True),
    ("small_g1_p40_l1030", 40, 256, 1030, 1, 32, BF16, 40, False),
    ("small_g2_p0", 33, 256, 1024, 2, 64, BF16, 0, True),
    ("small_g8_p256_skewed", 36, 768, 4096, 8, 64, BF16, -256, False),
    ("small_g2_p300_composed", 36, 256, 2048, 2, 64, BF16, 300, False),
    ("composed_f32_g8", 32, 256, 4096, 8, 32, F32, 5, True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fwd_bce(hs, orc, case):
    import torch
    name, B, F_s, L, G, F_in, dt, P, with_bias = case
    say(f"[fwd_bce] {name}: B={B} F_s={F_s} L={L} G={G} F_in={F_in} dtype={dt} P={P}")
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=dt, wid=600 + CASES.index(case))
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    rng = np.random.default_rng(wl.wid)
    bias = rng.standard_normal(L).astype(np.float32) if with_bias else None
    if P < 0:
        P = -P
        pos = skewed_pos(rng, B, L, P)
        if name == "fused_p80_full_cell":
            pos[:, :40] = np.stack([rng.choice(512, 40, replace=False) for _ in range(B)])
            pos[:, 40:] = rng.integers(512, L, (B, 40))
    else:
        pos = rand_pos(rng, B, L, P)
    desc = hs.make_desc(B, F_s, L, G, F_in, dt)
    Xd, idxd, Wd, bd = to_dev(X), to_dev(idx), to_dev(W), to_dev(bias)
    posd = to_dev(pos) if P else None
    dY = out_tensor((B, L), dt)
    dW = torch.empty((L, F_in), dtype=torch.float32, device="cuda")
    db = torch.empty((L,), dtype=torch.float32, device="cuda")
    ws = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE))
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, bd, posd, dY, dW, db, 0, ws)
    _sync()
    dY_ref, dW_ref, db_ref = oracle_fwd_bce(orc, X, idx, W, bias, pos, G, F_in, dt)
    got = host_f32(dY, dt)
    _check("dY", got, dY_ref, dt)
    _check("dW", dW.cpu().numpy(), dW_ref, dt)
    _check("dbias", db.cpu().numpy(), db_ref, dt)
    T = targets(pos, B, L)
    assert np.array_equal(got < 0, T) and np.all(got[~T] > 0), "targets are not applied exactly where pos names them"
    # the fused backward-weight product is haste_bwd_w on the returned dY, bit for bit
    dW2 = torch.empty_like(dW)
    db2 = torch.empty_like(db)
    hs.haste_bwd_w(desc, Xd, idxd, dY, dW2, db2, 0, hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_W)))
    _sync()
    assert bool((dW2 == dW).all()) and bool((db2 == db).all()), "fused dW differs from haste_bwd_w on its dY"
    if dt == BF16 and G in (1, 2, 4, 8):
        # small groups: the gradient the forward stores is the gradient pass's on its logits, bit for bit
        Y = out_tensor((B, L), dt)
        hs.haste_fwd(desc, Xd, idxd, Wd, bd, Y)
        dY3 = out_tensor((B, L), dt)
        hs.haste_bce_grad(B, L, dt, Y, posd, dY3)
        _sync()
        assert bool((dY3 == dY).all()), "the forward's gradient store differs from haste_bce_grad on its logits"
    # beta = 1 accumulates; without dW only dY is written
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, bd, posd, dY, dW, db, 1, ws)
    dY2 = out_tensor((B, L), dt)
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, bd, posd, dY2, None, None, 0, ws)
    _sync()
    assert bool((dW == 2 * dW2).all()) and bool((db == 2 * db2).all()), "beta = 1 must add the same sums"
    assert bool((dY2 == dY).all()), "dY without dW must equal dY with it"


@pytest.mark.parametrize("B,N,dt,inplace", [(33, 1000, BF16, False), (64, 4096, BF16, True), (7, 1003, BF16, True),
                                            (33, 1000, F32, False), (5, 77, F32, True)])
def test_bce_grad_elementwise(hs, orc, B, N, dt, inplace):
    say(f"[bce_grad] B={B} N={N} dtype={dt} inplace={inplace}")
    rng = np.random.default_rng(B * N)
    z = (2.5 * rng.standard_normal((B, N))).astype(np.float32)
    z[0, :3] = [0.0, 30.0, -30.0]
    zs = synth.bf16_bits(z) if dt == BF16 else z
    pos = rand_pos(rng, B, N, 6)
    Y = to_dev(zs)
    out = Y if inplace else out_tensor((B, N), dt)
    hs.haste_bce_grad(B, N, dt, Y, to_dev(pos), out)
    _sync()
    ref = orc.bce_grad(synth.to_f64(zs, dt), pos)
    got = host_f32(out, dt)
    _check("bce_grad", got, ref, dt)
    T = targets(pos, B, N)
    live = np.abs(synth.to_f64(zs, dt)) < 15          # sigmoid strictly inside (0, 1) in fp32
    assert np.array_equal((got < 0) & live, T & live), "targets are not applied exactly where pos names them"


def test_fwd_bce_empty_and_errors(hs):
    import torch
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    d0 = hs.make_desc(0, 768, 4096, 32, 64, BF16)
    dW = torch.full((4096, 64), 3.0, device="cuda")
    db = torch.full((4096,), 3.0, device="cuda")
    hs.haste_fwd_bce(d0, dummy, dummy, dummy, None, None, dummy, dW, db, 0)
    _sync()
    assert float(dW.abs().max()) == 0.0 and float(db.abs().max()) == 0.0
    d = hs.make_desc(8, 768, 4096, 32, 64, BF16)
    with pytest.raises(hs.HasteError):   # dbias without dW
        hs.haste_fwd_bce(d, dummy, dummy, dummy, None, None, dummy, None, db, 0)
    with pytest.raises(hs.HasteError):   # workspace missing
        hs.haste_fwd_bce(d, dummy, dummy, dummy, None, None, dummy, dW, None, 0)


LARGE = ["l2949k_g32_h65k", "l655k_g32_h16k", "gsweep_g16"]


@pytest.mark.parametrize("name", LARGE)
def test_fwd_bce_large_sampled(hs, orc, name):
    """The full-size layers, launched as the benchmark launches them: label ranges at the start,
    middle and end (every row), random points, the exact target rule over the whole dY, and the
    fused dW against haste_bwd_w on the same dY over the whole layer."""
    import torch
    wl = synth.WORKLOADS[name]
    dt = wl.dtype
    say(f"[fwd_bce workload] {wl.name}: B={wl.B} L={wl.L} G={wl.G} F_in={wl.F_in}")
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    positives = synth.draw_positives(wl)
    tail, _ = synth.positive_neurons(wl, positives, synth.draw_perm(wl))
    pos = synth.pos_matrix(tail, wl.B)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, dt)
    Xd, idxd, Wd, posd = to_dev(X), to_dev(idx), to_dev(W), to_dev(pos)
    dY = out_tensor((wl.B, wl.L), dt)
    dW = torch.empty((wl.L, wl.F_in), dtype=torch.float32, device="cuda")
    db = torch.empty((wl.L,), dtype=torch.float32, device="cuda")
    ws = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE))
    hs.haste_fwd_bce(desc, Xd, idxd, Wd, None, posd, dY, dW, db, 0, ws)
    _sync()
    Xf = synth.to_f64(X, dt).astype(np.float32)
    n = 4096
    for r0 in sorted({0, (wl.L // 2) // wl.G * wl.G, wl.L - n}):
        r1 = r0 + n
        say(f"  labels [{r0}, {r1})")
        z = orc.fwd(X, idx, W, None, wl.G, dt, r0, r1)
        dY_ref = orc.bce_grad(z, pos - r0)           # ids outside the range are ignored
        _check("dY", host_f32(dY[:, r0:r1].contiguous(), dt), dY_ref, dt)
        dW_ref, db_ref = orc.bwd_w(Xf, idx[r0 // wl.G:r1 // wl.G], dY_ref.astype(np.float32), wl.G, wl.F_in, F32,
                                   with_dbias=True)
        _check("dW", dW[r0:r1].cpu().numpy(), dW_ref, dt)
        _check("dbias", db[r0:r1].cpu().numpy(), db_ref, dt)
    rng = np.random.default_rng(11)
    bs = rng.integers(0, wl.B, 4096)
    ls = rng.integers(0, wl.L, 4096)
    bs = np.concatenate([bs, tail[:, 0]])            # every positive is a sample point too
    ls = np.concatenate([ls, tail[:, 1]])
    got = host_f32(dY[torch.from_numpy(bs).cuda(), torch.from_numpy(ls).cuda()].contiguous(), dt)
    ref = orc.bce_grad_at(pos, wl.L, bs, ls, orc.fwd_at(X, idx, W, None, wl.G, dt, bs, ls))
    _check("dY@rand", got, ref, dt)
    # exact target rule over the whole output: negative entries are exactly the positives
    neg = (dY.view(torch.bfloat16) < 0) if dt == BF16 else (dY < 0)
    n_pos = len({(int(b), int(c)) for b, c in tail})
    assert int(neg.sum()) == n_pos, f"{int(neg.sum())} negative entries, {n_pos} positives"
    assert bool(neg[torch.from_numpy(tail[:, 0]).cuda(), torch.from_numpy(tail[:, 1]).cuda()].all())
    dW2 = torch.empty_like(dW)
    hs.haste_bwd_w(desc, Xd, idxd, dY, dW2, None, 0, hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_W)))
    _sync()
    assert bool((dW2 == dW).all()), "fused dW differs from haste_bwd_w on its dY"


# ------------------------------------------------------------------------------------------
# dense head forward fused with the loss gradient
# ------------------------------------------------------------------------------------------
HEAD_BCE = [
    # B, F_s, H, dtype, P, bias   (the GEMM epilogue forms the gradient where the 256-tile kernel
    # runs: bf16, F_s and H multiples of 8; the other cases compose the forward and haste_bce_grad)
    (33, 200, 304, BF16, 6, True),
    (256, 768, 1024, BF16, 8, False),
    (300, 520, 2056, BF16, 64, True),
    (1, 64, 24, BF16, 3, False),
    (64, 256, 512, BF16, 0, True),
    (130, 768, 4100, BF16, 5, True),
    (33, 200, 300, F32, 6, True),
]


@pytest.mark.parametrize("case", HEAD_BCE, ids=[f"B{c[0]}_F{c[1]}_H{c[2]}_{'bf16' if c[3] else 'f32'}_P{c[4]}"
                                                for c in HEAD_BCE])
def test_head_fwd_bce(hs, orc, case):
    B, F_s, H, dt, P, with_bias = case
    say(f"[head_fwd_bce] B={B} F_s={F_s} H={H} dtype={dt} P={P}")
    wl = synth.small("head_bce", B=B, F_s=F_s, L=0, G=1, F_in=1, H=H, dtype=dt, wid=700 + HEAD_BCE.index(case))
    X, Wh = synth.draw_X(wl), synth.draw_W_head(wl)
    rng = np.random.default_rng(wl.wid)
    bh = rng.standard_normal(H).astype(np.float32) if with_bias else None
    pos = rand_pos(rng, B, H, P)
    dY = out_tensor((B, H), dt)
    hs.haste_head_fwd_bce(B, F_s, H, dt, to_dev(X), to_dev(Wh), to_dev(bh), to_dev(pos) if P else None, dY)
    _sync()
    got = host_f32(dY, dt)
    _check("head dY", got, orc.bce_grad(orc.head_fwd(X, Wh, bh, dt), pos), dt)
    T = targets(pos, B, H)
    assert np.array_equal(got < 0, T) and np.all(got[~T] > 0), "targets are not applied exactly where pos names them"


def test_head_fwd_bce_large_sampled(hs, orc):
    """The 65,536-label head of the 3M-label layer (B = 512), its own positives; column slices
    at both ends and across a tile edge against the oracle."""
    wl = synth.WORKLOADS["l2949k_g32_h65k"]
    say(f"[head_fwd_bce workload] {wl.name}")
    X, Wh = synth.draw_X(wl), synth.draw_W_head(wl)
    rng = np.random.default_rng(17)
    pos = rand_pos(rng, wl.B, wl.H, 8)
    pos[:, 0] = rng.integers(0, 300, wl.B)             # frequent labels first, as the head's are
    dY = out_tensor((wl.B, wl.H), wl.dtype)
    hs.haste_head_fwd_bce(wl.B, wl.F_s, wl.H, wl.dtype, to_dev(X), to_dev(Wh), None, to_dev(pos), dY)
    _sync()
    got = host_f32(dY, wl.dtype)
    T = targets(pos, wl.B, wl.H)
    assert np.array_equal(got < 0, T), "targets are not applied exactly where pos names them"
    for h0, h1 in [(0, 400), (32640, 33024), (wl.H - 300, wl.H)]:
        ref = orc.bce_grad(orc.head_fwd(X, Wh, None, wl.dtype, h0, h1), pos - h0)
        _check(f"[{h0},{h1})", got[:, h0:h1], ref, wl.dtype)


def test_head_fwd_bce_errors(hs):
    import torch
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    hs.haste_head_fwd_bce(0, 768, 1024, BF16, dummy, dummy, None, None, dummy)   # B = 0: nothing to do
    with pytest.raises(hs.HasteError):   # positives named but missing
        hs._check(hs.lib.haste_head_fwd_bce(4, 768, 1024, BF16, hs._ptr(dummy), hs._ptr(dummy), None, None, 3,
                                            hs._ptr(dummy), None))
