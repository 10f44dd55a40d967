"""Host-side checks of bench.py's bookkeeping (no GPU): the one-GPU guard, the algorithmic byte
counts the roofline divides by, and which profiled kernels each call is charged with."""
import os
import re
import subprocess
import sys

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_algorithmic_bytes_of_the_3m_layer():
    wl = synth.WORKLOADS["l2949k_g32_h65k"]
    B, F_s, L, G, F_in, H = wl.B, wl.F_s, wl.L, wl.G, wl.F_in, wl.H
    c = bench.call_cost(wl, n_pos=8)
    idx, W, Y, dW, dX, X = L // G * F_in * 4, L * F_in * 2, B * L * 2, L * F_in * 4, B * F_s * 4, B * F_s * 2
    # each operand moved once: the byte counts the roofline fractions divide by
    assert c["bwd_x"] == (idx + W + Y + dX, 2 * B * L * F_in)
    assert c["fwd"] == (X + idx + W + Y, 2 * B * L * F_in)
    assert c["fwd_bce"][0] == X + idx + W + B * 8 * 4 + Y + dW
    assert round(c["bwd_x"][0] / 1e9, 2) == 3.42 and round(c["fwd_bce"][0] / 1e9, 2) == 4.18
    assert c["head_fwd_bce"] == (c["head_fwd"][0] + B * 8 * 4, 2 * B * H * F_s)
    assert c["tail_step"][0] == c["fwd_bce"][0] + c["bwd_x"][0]


def test_profiled_kernels_are_charged_to_their_calls():
    def owners(kernel):
        return {c for c, pats in bench.CALL_KERNELS.items() if any(re.match(p, kernel) for p in pats)}
    assert owners("k_fwd_bce<64, false, 1, false>") == {"fwd_bce", "tail_step"}
    assert owners("k_fwd_bce<128, true, 2, true>") == {"fwd_bce_sgd", "tail_step_sgd"}
    assert owners("k_gemm4<128, true, true, 3>") == {"head_fwd_bce"}
    assert owners("k_gemm4<128, true, true, 0>") == {"head_fwd"}
    assert owners("k_gemm4<128, true, false, 2>") == {"head_bwd"}
    assert owners("k_bwd_x<64, 1>") == {"bwd_x", "tail_step", "tail_step_sgd"} and owners("k_transpose_w") == {"bwd_x"}
    assert "head_bwd" in owners("k_reduce_rmajor") and "bwd_x" in owners("k_reduce_fmajor")
