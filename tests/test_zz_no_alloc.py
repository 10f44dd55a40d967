"""haste_fwd_bce_static (through the C ABI) against haste_fwd_bce with a caller workspace: the same
dY, dW and dbias bit for bit, on calls in a row whose later layers are smaller (the library's
per-device scratch keeps the earlier call's data), on the fused kernel and on the composed path."""
import numpy as np
import pytest

import synth
from gpu_helpers import out_tensor, rand_pos, say, to_dev

pytestmark = pytest.mark.gpu
BF16 = synth.DT_BF16


@pytest.fixture(scope="module")
def hs():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2606_01117_amd as m
    return m


CALLS = [
    # name, B, F_s, L, G, F_in, P, bias, beta
    ("fused_b300_g32", 300, 768, 8192, 32, 64, 8, True, 0),
    ("fused_smaller_b40_g16", 40, 256, 2048, 16, 32, 3, False, 1),
    ("composed_b33_g4", 33, 512, 1024, 4, 64, 5, True, 0),
    ("fused_bucketed_b64_p150", 64, 768, 4096, 32, 64, 150, False, 0),
]


def _run(hs, case, static):
    import torch
    name, B, F_s, L, G, F_in, P, with_bias, beta = case
    wl = synth.small(name, B=B, F_s=F_s, L=L, G=G, F_in=F_in, dtype=BF16, wid=1200 + CALLS.index(case))
    X, W, idx = synth.draw_X(wl), synth.draw_W(wl), synth.draw_idx(wl)
    rng = np.random.default_rng(wl.wid)
    bias = rng.standard_normal(L).astype(np.float32) if with_bias else None
    pos = rand_pos(rng, B, L, P)
    desc = hs.make_desc(B, F_s, L, G, F_in, BF16)
    dY = out_tensor((B, L), BF16)
    dW = torch.full((L, F_in), 0.5, dtype=torch.float32, device="cuda")
    db = torch.full((L,), 0.25, dtype=torch.float32, device="cuda") if with_bias else None
    args = (desc, to_dev(X), to_dev(idx), to_dev(W), to_dev(bias), to_dev(pos), dY, dW, db, beta)
    if static:
        hs.haste_fwd_bce_static(*args)
    else:
        hs.haste_fwd_bce(*args, ws=hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_FWD_BCE)))
    torch.cuda.synchronize()
    return dY.view(torch.int16), dW, db


def test_static_scratch_equals_workspace_calls(hs):
    import torch
    refs = [_run(hs, c, static=False) for c in CALLS]
    for c, ref in zip(CALLS, refs):
        say(f"[no-alloc] {c[0]}: B={c[1]} F_s={c[2]} L={c[3]} G={c[4]} F_in={c[5]} P={c[6]}")
        got = _run(hs, c, static=True)
        assert bool((got[0] == ref[0]).all()), f"{c[0]}: dY differs"
        assert bool((got[1] == ref[1]).all()), f"{c[0]}: dW differs"
        if ref[2] is not None:
            assert bool((got[2] == ref[2]).all()), f"{c[0]}: dbias differs"
    # a repeat of the first, larger layer after the smaller ones
    got = _run(hs, CALLS[0], static=True)
    assert all(bool((g == r).all()) for g, r in zip(got, refs[0]) if r is not None), "repeat of the first layer"
    assert torch.cuda.is_available()
