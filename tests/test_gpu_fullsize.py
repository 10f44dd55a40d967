"""Full-size GPU parity of the named large workloads (the 655K-label tail with its 16K head, the
group-size sweep on a 655K-label layer, the 2.95M-label tail with its 65K head) against the fp64
CPU oracle, through the C ABI.

* The separate calls (Section 3.2 forward, backward-weight and backward-feature, on a fixed dY):
  every dW row and every dbias entry (label chunks), every row of dX, the forward on label
  windows and random points, and the fp64 adjoint identity <dY, Y - b> = <dX, X> = <dW, W> on
  the GPU's own full-size outputs; then the dense head (Section 3.3) on slices and dX tail + head
  on every row.
* The tail's training pass in one call (haste_tail_step: the Section 3.3 BCE gradient formed from
  the step's own logits, dW and dX from it): every dY entry, dW row and dbias entry, and every row
  of dX, against the oracle's own chain (fp64 logits, fp64 BCE gradient, its backward products).

The adjoint identity holds exactly in exact arithmetic (the layer is bilinear).  Here Y is rounded
to bf16 (relative error at most 2^-9 per entry), so |<dY, Y> - <dY, Y_exact>| <= 2^-9 sum |dY Y|;
dX and dW are fp32 sums.  The three pairings must agree within 2^-8 sum |dY Y|.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import TOL, Layer, host_f32, make_inputs, out_tensor, rel_err, say, to_dev

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]
F32, BF16 = synth.DT_F32, synth.DT_BF16
LARGE = ["l655k_g32_h16k", "gsweep_g1", "gsweep_g4", "gsweep_g16", "gsweep_g64", "l2949k_g32_h65k"]
CHUNK = 1 << 16   # labels per oracle chunk (a multiple of every G here)


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


class _Worst:
    """Running infinity-norm relative error of one output over chunks: max |a - r| / max |r|."""

    def __init__(self, name, dtype):
        self.name, self.dtype, self.num, self.den = name, dtype, 0.0, 0.0

    def add(self, got, ref):
        got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
        if ref.size:
            self.num = max(self.num, float(np.abs(got - ref).max()))
            self.den = max(self.den, float(np.abs(ref).max()))

    def check(self):
        e = self.num / (self.den if self.den > 0 else 1.0)
        say(f"    {self.name:<14s} rel_inf_err={e:.3e} (tol {TOL[self.dtype]:.0e})")
        assert e <= TOL[self.dtype], f"{self.name}: {e:.3e} > {TOL[self.dtype]:.0e}"


def _check(name, got, ref, dtype):
    e = rel_err(got, ref)
    say(f"    {name:<14s} rel_inf_err={e:.3e} (tol {TOL[dtype]:.0e})")
    assert e <= TOL[dtype], f"{name}: {e:.3e} > {TOL[dtype]:.0e}"


def _chunks(L):
    return [(l0, min(L, l0 + CHUNK)) for l0 in range(0, L, CHUNK)]


@pytest.mark.parametrize("name", LARGE)
def test_large_separate_calls(hs, orc, name):
    import torch
    wl = synth.WORKLOADS[name]
    dt = wl.dtype
    say(f"[fullsize] {wl.name}: B={wl.B} L={wl.L} G={wl.G} F_in={wl.F_in} H={wl.H}: separate calls")
    X, idx, W, bias, dY = make_inputs(wl)
    lay = Layer(hs, wl, X, idx, W, bias, dY)
    lay.fwd()
    lay.bwd_w()
    lay.bwd_x()
    _sync()
    # every dW row and dbias entry, and the pairings <dY, Y - b> and <dW, W>, chunk by chunk
    e_dw, e_db = _Worst("bwd_w (all)", dt), _Worst("dbias (all)", dt)
    dyy = dyy_abs = ww = 0.0
    Wf = synth.to_f64(W, dt)
    for (l0, l1) in _chunks(wl.L):
        dW_ref, db_ref = orc.bwd_w(X, idx, dY, wl.G, wl.F_in, dt, l0, l1, with_dbias=True)
        dWg = lay.dW[l0:l1].cpu().numpy()
        e_dw.add(dWg, dW_ref)
        e_db.add(lay.dbias[l0:l1].cpu().numpy(), db_ref)
        Yc = host_f32(lay.Y[:, l0:l1].contiguous(), dt).astype(np.float64)
        if bias is not None:
            Yc -= bias[l0:l1]
        dYc = synth.to_f64(dY[:, l0:l1], dt)
        dyy += float(np.sum(dYc * Yc))
        dyy_abs += float(np.sum(np.abs(dYc * Yc)))
        ww += float(np.sum(dWg.astype(np.float64) * Wf[l0:l1]))
        if l0 // CHUNK % 8 == 0:
            say(f"  labels [{l0}, {l1})")
    e_dw.check()
    e_db.check()
    # every row of dX
    dX_tail = orc.bwd_x(idx, W, dY, wl.G, wl.F_s, dt)
    dXg = lay.dX.cpu().numpy()
    _check("bwd_x (all rows)", dXg, dX_tail, dt)
    xx = float(np.sum(dXg.astype(np.float64) * synth.to_f64(X, dt)))
    say(f"    adjoint <dY,Y-b>={dyy:.9e} <dX,X>={xx:.9e} <dW,W>={ww:.9e} (scale {dyy_abs:.3e})")
    tol = 2.0 ** -8 * dyy_abs
    assert abs(dyy - xx) <= tol and abs(dyy - ww) <= tol and abs(xx - ww) <= tol, "adjoint identity"
    # the forward on windows at both ends and the middle, and at random points
    n = min(4096, wl.L)
    for (r0, r1) in sorted({(0, n), (wl.L // 2 - n // 2, wl.L // 2 + n - n // 2), (wl.L - n, wl.L)}):
        _check(f"fwd [{r0},{r1})", host_f32(lay.Y[:, r0:r1].contiguous(), dt),
               orc.fwd(X, idx, W, bias, wl.G, dt, r0, r1), dt)
    rng = np.random.default_rng(7)
    bs, ls = rng.integers(0, wl.B, 4096), rng.integers(0, wl.L, 4096)
    got = host_f32(lay.Y[torch.from_numpy(bs).cuda(), torch.from_numpy(ls).cuda()].contiguous(), dt)
    _check("fwd@rand", got, orc.fwd_at(X, idx, W, bias, wl.G, dt, bs, ls), dt)
    if wl.H:
        Wh = synth.draw_W_head(wl)
        dYh = synth.draw_dY_head(wl)
        Whd, dYhd = to_dev(Wh), to_dev(dYh)
        Yh = out_tensor((wl.B, wl.H), dt)
        dWh = torch.empty((wl.H, wl.F_s), dtype=torch.float32, device="cuda")
        hs.haste_head_fwd(wl.B, wl.F_s, wl.H, dt, lay.X, Whd, None, Yh)
        ws = hs.workspace(hs.haste_head_workspace_bytes(wl.B, wl.F_s, wl.H, dt))
        hs.haste_head_bwd(wl.B, wl.F_s, wl.H, dt, lay.X, Whd, dYhd, dWh, lay.dX, 1, ws)
        _sync()
        _check("head fwd", host_f32(Yh, dt), orc.head_fwd(X, Wh, None, dt), dt)
        _check("head dW", dWh.cpu().numpy(), orc.head_bwd_w(X, dYh, dt), dt)
        _check("dX tail+head", lay.dX.cpu().numpy(), dX_tail + orc.head_bwd_x(Wh, dYh, dt), dt)


@pytest.mark.parametrize("name", LARGE)
def test_large_tail_step(hs, orc, name):
    """haste_tail_step on the workload's own positives, every output against the oracle's chain."""
    import torch
    wl = synth.WORKLOADS[name]
    dt = wl.dtype
    say(f"[fullsize] {wl.name}: B={wl.B} L={wl.L} G={wl.G} F_in={wl.F_in}: haste_tail_step")
    X, idx, W = synth.draw_X(wl), synth.draw_idx(wl), synth.draw_W(wl)
    tail_pairs, _ = synth.positive_neurons(wl, synth.draw_positives(wl), synth.draw_perm(wl))
    pos = synth.pos_matrix(tail_pairs, wl.B, wl.n_pos)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, dt)
    dY = out_tensor((wl.B, wl.L), dt)
    dW = torch.empty((wl.L, wl.F_in), dtype=torch.float32, device="cuda")
    db = torch.empty((wl.L,), dtype=torch.float32, device="cuda")
    dX = torch.empty((wl.B, wl.F_s), dtype=torch.float32, device="cuda")
    hs.haste_tail_step(desc, to_dev(X), to_dev(idx), to_dev(W), None, to_dev(pos), dY, dW, db, 0, dX, 0,
                       hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP)))
    _sync()
    Xf = synth.to_f64(X, dt).astype(np.float32)       # exact
    Wf = synth.to_f64(W, dt).astype(np.float32)       # exact
    e_dy, e_dw, e_db = _Worst("dY (all)", dt), _Worst("dW (all)", dt), _Worst("dbias (all)", dt)
    dX_ref = np.zeros((wl.B, wl.F_s))
    for (l0, l1) in _chunks(wl.L):
        k0, k1 = l0 // wl.G, l1 // wl.G
        z = orc.fwd(X, idx, W, None, wl.G, dt, l0, l1)
        pos_c = np.where((pos >= l0) & (pos < l1), pos - l0, -1).astype(np.int32)
        dY_o = orc.bce_grad(z, pos_c)
        e_dy.add(host_f32(dY[:, l0:l1].contiguous(), dt), dY_o)
        dY32 = dY_o.astype(np.float32)
        dW_o, db_o = orc.bwd_w(Xf, idx[k0:k1], dY32, wl.G, wl.F_in, F32, with_dbias=True)
        e_dw.add(dW[l0:l1].cpu().numpy(), dW_o)
        e_db.add(db[l0:l1].cpu().numpy(), db_o)
        dX_ref += orc.bwd_x(idx[k0:k1], Wf[l0:l1], dY32, wl.G, wl.F_s, F32)
        if l0 // CHUNK % 8 == 0:
            say(f"  labels [{l0}, {l1})")
    e_dy.check()
    e_dw.check()
    e_db.check()
    _check("dX (all rows)", dX.cpu().numpy(), dX_ref, dt)
