"""GPU parity of libhaste (through the C ABI) against the fp64 CPU oracle.

Small layers and the two small named workloads are compared element by element on every output
(the large named workloads, in full, are in test_gpu_fullsize.py); then the dense head on ragged
shapes, exact gathers and scatters, index validation, empty inputs and bitwise repeatability.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import TOL, Layer, host_f32, make_inputs, out_tensor, rel_err, say, to_dev

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


# ------------------------------------------------------------------------------------------
# small layers, every element
# ------------------------------------------------------------------------------------------
SMALL = [
    # name, B, F_s, L, G, F_in, dtype
    ("bf16_g32_f64", 40, 256, 2048, 32, 64, BF16),
    ("bf16_g16_ragged_b33", 33, 768, 4096, 16, 64, BF16),
    ("bf16_b1", 1, 768, 1024, 32, 32, BF16),
    ("bf16_g64_f128", 70, 768, 4096, 64, 128, BF16),
    ("bf16_g4", 64, 512, 1536, 4, 64, BF16),
    ("bf16_g8_f32", 70, 768, 3072, 8, 32, BF16),
    ("bf16_g96", 17, 256, 1920, 96, 32, BF16),
    ("bf16_g1_ffi", 37, 768, 1024, 1, 64, BF16),
    ("bf16_g3_f16", 20, 128, 600, 3, 16, BF16),
    ("bf16_b300_g32", 300, 768, 8192, 32, 64, BF16),
    ("bf16_b511_g32_f128", 511, 768, 2048, 32, 128, BF16),
    # a group of 72 = 32 + 32 + 8 labels: unit pairs that start on a partial tile
    ("bf16_g72_f32", 48, 384, 72 * 29, 72, 32, BF16),
    # 12-label groups (4-label stores) with a 128-slot support
    ("bf16_g12_f128", 45, 512, 12 * 37, 12, 128, BF16),
    # small groups (16 / G groups per matrix tile), ragged label counts and batch tails
    ("bf16_g2_f128", 50, 768, 2048, 2, 128, BF16),
    ("bf16_g4_f128_fs896", 70, 896, 4096, 4, 128, BF16),
    ("bf16_g1_f32_l1003", 33, 256, 1003, 1, 32, BF16),
    ("bf16_g8_f64_l2056", 100, 768, 2056, 8, 64, BF16),
    ("bf16_g2_f32_l1030", 40, 512, 1030, 2, 32, BF16),
    ("bf16_g4_b1", 1, 768, 1024, 4, 64, BF16),
    # backward-feature's small-group kernel: 32-label super-groups cut short at the end of the layer
    # (and rows ending inside a 16-byte piece), the narrow staging of the widest feature dimension
    ("bf16_g1_f128_l1062", 45, 512, 1062, 1, 128, BF16),
    ("bf16_g8_f128", 33, 768, 1024, 8, 128, BF16),
    ("bf16_g4_fs1024", 40, 1024, 2048, 4, 64, BF16),
    # the scattered-tile kernels: feature counts that are not whole tiles, 64-row workgroups with a
    # mostly empty row tile, 2-label row tails, a layer shorter than the segments it is cut into,
    # feature counts between the tile-count steps
    ("bf16_g2_fs104_l1030", 33, 104, 1030, 2, 32, BF16),
    ("bf16_g1_fs200_b31", 31, 200, 2050, 1, 64, BF16),
    ("bf16_g2_l130", 40, 256, 130, 2, 64, BF16),
    ("bf16_g8_fs520", 64, 520, 2048, 8, 64, BF16),
    # the dense backward-weight (G = 1, 2): more 64-label blocks than CUs (a second block for some
    # workgroups) ending in a 6-label block, a single row with 128-slot supports, and feature
    # counts short of the four waves' tiles with a padded K step
    ("bf16_g1_l19206", 40, 768, 64 * 300 + 6, 1, 64, BF16),
    ("bf16_g2_f128_b1", 1, 512, 384, 2, 128, BF16),
    ("bf16_g2_fs640_b96", 96, 640, 4096, 2, 64, BF16),
    # 256-slot supports (the VALU kernels)
    ("bf16_g32_f256", 40, 768, 2048, 32, 256, BF16),
    ("f32_g8", 32, 256, 4096, 8, 32, F32),
    ("f32_g1", 9, 100, 300, 1, 7, F32),
    ("f32_g32_f64", 50, 768, 2048, 32, 64, F32),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_small_layers(hs, orc, case):
    name, B, F_s, L, G, F_in, dt = case
    say(f"[small] {name}: B={B} F_s={F_s} L={L} G={G} F_in={F_in} dtype={dt}")
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=dt, wid=200 + SMALL.index(case),
                     dy_normal=True)
    X, idx, W, _, dY = make_inputs(wl)
    bias = np.random.default_rng(wl.wid).standard_normal(L).astype(np.float32)
    lay = Layer(hs, wl, X, idx, W, bias, dY)
    lay.fwd()
    lay.bwd_w()
    lay.bwd_x()
    _sync()
    _check("fwd", host_f32(lay.Y, dt), orc.fwd(X, idx, W, bias, G, dt), dt)
    dW_ref, db_ref = orc.bwd_w(X, idx, dY, G, F_in, dt, with_dbias=True)
    _check("bwd_w", lay.dW.cpu().numpy(), dW_ref, dt)
    _check("dbias", lay.dbias.cpu().numpy(), db_ref, dt)
    dX_ref = orc.bwd_x(idx, W, dY, G, F_s, dt)
    _check("bwd_x", lay.dX.cpu().numpy(), dX_ref, dt)
    # beta = 1 accumulates onto the previous results
    lay.bwd_w(beta=1)
    lay.bwd_x(beta=1)
    _sync()
    _check("bwd_w b1", lay.dW.cpu().numpy(), 2 * dW_ref, dt)
    _check("dbias b1", lay.dbias.cpu().numpy(), 2 * db_ref, dt)
    _check("bwd_x b1", lay.dX.cpu().numpy(), 2 * dX_ref, dt)


# ------------------------------------------------------------------------------------------
# the named workloads
# ------------------------------------------------------------------------------------------
def test_tiny_f32_full(hs, orc):
    wl = synth.WORKLOADS["tiny_f32"]
    say(f"[workload] {wl.name}")
    X, idx, W, bias, dY = make_inputs(wl)
    lay = Layer(hs, wl, X, idx, W, bias, dY)
    lay.fwd()
    lay.bwd_w()
    lay.bwd_x()
    _sync()
    _check("fwd", host_f32(lay.Y, F32), orc.fwd(X, idx, W, bias, wl.G, F32), F32)
    _check("bwd_w", lay.dW.cpu().numpy(), orc.bwd_w(X, idx, dY, wl.G, wl.F_in, F32)[0], F32)
    _check("bwd_x", lay.dX.cpu().numpy(), orc.bwd_x(idx, W, dY, wl.G, wl.F_s, F32), F32)


def test_l131k_full(hs, orc):
    wl = synth.WORKLOADS["l131k_g16"]
    say(f"[workload] {wl.name}: full tensors, dY from the oracle's logits")
    X, idx, W, bias, dY = make_inputs(wl, orc, logits_from_oracle=True)
    lay = Layer(hs, wl, X, idx, W, bias, dY)
    lay.fwd()
    lay.bwd_w()
    lay.bwd_x()
    _sync()
    _check("fwd", host_f32(lay.Y, BF16), orc.fwd(X, idx, W, bias, wl.G, BF16), BF16)
    _check("bwd_w", lay.dW.cpu().numpy(), orc.bwd_w(X, idx, dY, wl.G, wl.F_in, BF16)[0], BF16)
    _check("bwd_x", lay.dX.cpu().numpy(), orc.bwd_x(idx, W, dY, wl.G, wl.F_s, BF16), BF16)


# ------------------------------------------------------------------------------------------
# dense head alone, ragged shapes
# ------------------------------------------------------------------------------------------
HEAD = [(33, 200, 300, BF16), (256, 768, 1024, BF16), (1, 64, 17, BF16), (130, 768, 4100, BF16),
        (300, 520, 2056, BF16), (33, 200, 300, F32), (5, 96, 70, F32)]


@pytest.mark.parametrize("case", HEAD, ids=[f"B{c[0]}_F{c[1]}_H{c[2]}_{'bf16' if c[3] else 'f32'}" for c in HEAD])
def test_head(hs, orc, case):
    import torch
    B, F_s, H, dt = case
    say(f"[head] B={B} F_s={F_s} H={H} dtype={dt}")
    wl = synth.small("head", B=B, F_s=F_s, L=0, G=1, F_in=1, H=H, dtype=dt, wid=300 + HEAD.index(case))
    X, Wh = synth.draw_X(wl), synth.draw_W_head(wl)
    rng = np.random.default_rng(wl.wid)
    dYh = rng.standard_normal((B, H)).astype(np.float32)
    dYh = synth.bf16_bits(dYh) if dt == BF16 else dYh
    bh = rng.standard_normal(H).astype(np.float32)
    Xd, Whd, dYhd, bhd = to_dev(X), to_dev(Wh), to_dev(dYh), to_dev(bh)
    Yh = out_tensor((B, H), dt)
    dWh = torch.empty((H, F_s), dtype=torch.float32, device="cuda")
    dX = torch.full((B, F_s), 0.5, dtype=torch.float32, device="cuda")
    hs.haste_head_fwd(B, F_s, H, dt, Xd, Whd, bhd, Yh)
    hs.haste_head_bwd(B, F_s, H, dt, Xd, Whd, dYhd, dWh, dX, 1,
                      hs.workspace(hs.haste_head_workspace_bytes(B, F_s, H, dt)))
    _sync()
    _check("head fwd", host_f32(Yh, dt), orc.head_fwd(X, Wh, bh, dt), dt)
    _check("head dW", dWh.cpu().numpy(), orc.head_bwd_w(X, dYh, dt), dt)
    _check("head dX+0.5", dX.cpu().numpy(), orc.head_bwd_x(Wh, dYh, dt) + 0.5, dt)


# ------------------------------------------------------------------------------------------
# exact gathers and scatters, index handling, edge cases
# ------------------------------------------------------------------------------------------
ONE_BF16 = np.uint16(0x3F80)


@pytest.mark.parametrize("G,F_in,dt", [(32, 64, BF16), (16, 128, BF16), (1, 64, BF16), (8, 32, F32), (4, 64, BF16)])
def test_one_hot_bit_exact(hs, orc, G, F_in, dt):
    B, F_s, L = 70, 768, 64 * max(G, 4)
    say(f"[one-hot] G={G} F_in={F_in} dtype={dt}")
    wl = synth.small("onehot", B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=dt, wid=400 + G + F_in, dy_normal=True)
    X, idx, _, _, dY = make_inputs(wl)
    one = ONE_BF16 if dt == BF16 else np.float32(1)
    zeros = lambda shape: np.zeros(shape, dtype=np.uint16 if dt == BF16 else np.float32)
    g = np.arange(L) // G
    # forward with W = e_t0 returns the gathered features bit for bit
    t0 = F_in - 3
    W = zeros((L, F_in))
    W[:, t0] = one
    lay = Layer(hs, wl, X, idx, W, None, dY)
    lay.fwd()
    _sync()
    got = lay.Y.cpu().numpy().view(np.uint16 if dt == BF16 else np.float32)
    assert np.array_equal(got, X[:, idx[g, t0]]), "one-hot forward is not an exact gather"
    # backward-weight with dY = e_b0 returns X[b0, idx] exactly
    b0 = B - 2
    dYo = zeros((B, L))
    dYo[b0] = one
    lay.dY = to_dev(dYo)
    lay.bwd_w(dbias=False)
    _sync()
    assert np.array_equal(lay.dW.cpu().numpy(), synth.to_f64(X, dt)[b0][idx[g]].astype(np.float32))
    # backward-feature with a single unit weight moves one dY column to one feature
    l0 = L // 2 + 1
    W = zeros((L, F_in))
    W[l0, t0] = one
    lay.W = to_dev(W)
    lay.dY = to_dev(dY)
    lay.bwd_x()
    _sync()
    exp = np.zeros((B, F_s), np.float32)
    exp[:, idx[l0 // G, t0]] = synth.to_f64(dY, dt)[:, l0]
    assert np.array_equal(lay.dX.cpu().numpy(), exp), "one-hot backward-feature is not an exact scatter"


def test_untouched_features_zero(hs):
    wl = synth.small("untouched", B=64, F_s=768, L=4096, G=32, F_in=64, dtype=BF16, wid=500, dy_normal=True)
    X, idx, W, _, dY = make_inputs(wl)
    rng = np.random.default_rng(3)
    idx = np.stack([np.sort(rng.choice(384, wl.F_in, replace=False)) for _ in range(wl.K)]).astype(np.int32)
    lay = Layer(hs, wl, X, idx, W, None, dY)
    lay.dX.fill_(7.0)
    lay.bwd_x()
    _sync()
    dX = lay.dX.cpu().numpy()
    assert np.all(dX[:, 384:] == 0.0), "features outside every support must get exactly zero"


def test_debug_gather_exact(hs):
    import torch
    wl = synth.small("gather", B=50, F_s=768, L=2048, G=32, F_in=64, dtype=BF16, wid=501)
    X, idx = synth.draw_X(wl), synth.draw_idx(wl)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, BF16)
    out = torch.empty((7, wl.B, wl.F_in), dtype=torch.int16, device="cuda")
    hs.haste_debug_gather(desc, to_dev(X), to_dev(idx), 20, 7, out)
    _sync()
    exp = np.stack([X[:, idx[k]] for k in range(20, 27)])
    assert np.array_equal(out.cpu().numpy().view(np.uint16), exp)


def test_validate_idx(hs):
    import torch
    wl = synth.small("validate", B=4, F_s=768, L=4096, G=32, F_in=64, dtype=BF16, wid=502)
    idx = synth.draw_idx(wl)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, BF16)
    nbad = torch.empty(1, dtype=torch.int32, device="cuda")
    hs.haste_validate_idx(desc, to_dev(idx), nbad)
    _sync()
    assert int(nbad.item()) == 0
    bad = idx.copy()
    bad[3, 5] = bad[3, 4]          # duplicate
    bad[10, 0], bad[10, 1] = bad[10, 1], bad[10, 0]  # unsorted
    bad[77, -1] = 768              # out of range
    hs.haste_validate_idx(desc, to_dev(bad), nbad)
    _sync()
    assert int(nbad.item()) == 3


def test_empty_batch_and_labels(hs):
    import torch
    d0 = hs.make_desc(0, 768, 4096, 32, 64, BF16)
    dW = torch.full((4096, 64), 3.0, device="cuda")
    db = torch.full((4096,), 3.0, device="cuda")
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    hs.haste_bwd_w(d0, dummy, dummy, dummy, dW, db, 0)
    hs.haste_fwd(d0, dummy, dummy, dummy, None, dummy)
    dL = hs.make_desc(16, 768, 0, 32, 64, BF16)
    dX = torch.full((16, 768), 3.0, device="cuda")
    hs.haste_bwd_x(dL, dummy, dummy, dummy, dX, 0)
    _sync()
    assert float(dW.abs().max()) == 0.0 and float(db.abs().max()) == 0.0
    assert float(dX.abs().max()) == 0.0


@pytest.mark.parametrize("G", [32, 4])
def test_repeatable(hs, G):
    wl = synth.small("repeat", B=256, F_s=768, L=65536, G=G, F_in=64, dtype=BF16, wid=503, dy_normal=True)
    X, idx, W, _, dY = make_inputs(wl)
    lay = Layer(hs, wl, X, idx, W, None, dY)
    lay.fwd(); lay.bwd_w(); lay.bwd_x()
    _sync()
    Y1, dW1, dX1 = lay.Y.clone(), lay.dW.clone(), lay.dX.clone()
    lay.fwd(); lay.bwd_w(); lay.bwd_x()
    _sync()
    # every reduction runs in a fixed order (no atomics): all three outputs are bitwise repeatable
    assert bool((Y1 == lay.Y).all()) and bool((dW1 == lay.dW).all()), "fwd / bwd_w must be bitwise repeatable"
    assert bool((dX1 == lay.dX).all()), "bwd_x must be bitwise repeatable"
