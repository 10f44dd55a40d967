"""Benchmark of the group-shared fixed fan-in output layer on one MI355X.

One step = one training pass of the layer on one batch of seeded synthetic input already resident
in HBM, with the upstream gradient formed from the step's own logits as the BCE gradient
sigmoid(z) - y of the Section 3.3 objective (the workload's definition of dY):
  the tail's pass in one call (haste_tail_step): forward + BCE gradient + backward-weight, fused,
  then backward-feature on the transposed weights the fused kernel wrote
  -> head forward + BCE gradient, fused (haste_head_fwd_bce)
  -> head backward (haste_head_bwd, adds its dX onto the tail's).
Timed beside it, on the same inputs:
  - the same training pass unfused: haste_fwd, haste_bce_grad, haste_bwd_w instead of haste_fwd_bce,
    and haste_head_fwd + haste_bce_grad instead of haste_head_fwd_bce;
  - the training pass plus one SGD-with-momentum step on W and W_h, fused (haste_fwd_bce_sgd, dW
    never stored) and unfused (haste_bwd_w + haste_sgd_momentum);
  - the five separate calls on a fixed dY (haste_fwd, haste_head_fwd, haste_bwd_w, haste_bwd_x,
    haste_head_bwd), i.e. without the loss gradient.
Default workload: the 2.95M-label tail (G = 32, F_in = 64) with a 65,536-label dense head, B = 512,
F_s = 768, bf16 storage with fp32 accumulation.

Prints ONE JSON line (rank 0): ms/step, per-call times from HIP events recorded on the stream the
calls are launched on, the roofline of the dominant kernel, the FLOPs-matched dense bottleneck
timed beside it, and the CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
PROFILES = os.path.join(ROOT, "profiles")
COPY_BYTES = 1 << 30            # plain device copy used to calibrate the HBM byte counters
FLUSH_BYTES = 512 << 20         # written before each timed step of a working set the MALL could hold
WARM_S = 0.2                    # untimed GPU work after host-side setup, before the first timed phase

# kernels launched by each call (patterns matched at the start of rocprofv3's kernel names; the
# fused kernel's third template argument is its output: 1 stores dW, 2 applies the momentum step)
CALL_KERNELS = {
    "fwd": ["k_fwd<"],
    "fwd_bce": ["k_transpose_x", r"k_fwd_bce<\d+, \w+, 1,"],
    "fwd_bce_sgd": ["k_transpose_x", r"k_fwd_bce<\d+, \w+, 2,"],
    "tail_step": ["k_transpose_x", r"k_fwd_bce<\d+, \w+, 1,", "k_bwd_x", "k_reduce_fmajor"],
    "tail_step_sgd": ["k_transpose_x", r"k_fwd_bce<\d+, \w+, 2,", "k_bwd_x", "k_reduce_fmajor"],
    "sgd": ["k_sgd_momentum"],
    "head_sgd": ["k_sgd_momentum"],
    "rewire": ["k_rw_"],
    "grouping": ["k_gl_"],
    "bce": ["k_bce_grad"],
    "head_bce": ["k_bce_grad"],
    "bwd_w": ["k_transpose_x", "k_bwd_w"],
    "bwd_x": ["k_transpose_w", "k_bwd_x", "k_reduce_fmajor"],
    # the head's GEMM kernels by operand layout and epilogue (three tile sizes: 256, 128, fallback)
    "head_fwd": [r"k_gemm4<\d+, true, true, 0>", "k_gemm2<true, true, 0>", "k_gemm_bf16<true, true, 0>"],
    # the large-tile kernel with the loss gradient in its epilogue (other shapes run head_fwd's kernels)
    "head_fwd_bce": [r"k_gemm4<\d+, true, true, 3>"],
    "head_bwd": [r"k_gemm4<\d+, false, false, 1>", r"k_gemm4<\d+, true, false, 2>", "k_gemm2<false, false, 1>",
                 "k_gemm2<true, false, 2>", "k_gemm_bf16<false, false, 1>", "k_gemm_bf16<true, false, 2>",
                 "k_reduce_rmajor"],
}


# calls whose kernel another call of a different size also launches: which dispatches are theirs
SHARED_KERNEL_PICK = {"bce": max, "head_bce": min, "sgd": max, "head_sgd": min}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="l2949k_g32_h65k")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-bottleneck", action="store_true")
    p.add_argument("--grouping", action="store_true", help="also time the label grouping of Alg. 2 (655K labels)")
    p.add_argument("--no-gsweep", action="store_true",
                   help="skip the group-size sweep (G = 1, 4, 16, 64 on the 655K-label layer, with its bottleneck)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="after the timed steps, run a plain %d-byte device copy (for counter calibration)" % COPY_BYTES)
    p.add_argument("--summarize-trace", metavar="DB",
                   help="write profiles/kernels_<workload>.md from a rocprofv3 --kernel-trace --stats database")
    p.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                   help="write profiles/traffic_<workload>.txt from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE databases")
    p.add_argument("--command", default="", help="the profiling command, recorded in the written summary")
    return p.parse_args()


def call_cost(wl, dt_bytes=2, n_pos=0):
    """Algorithmic bytes and FLOPs of each call (each operand moved once).  n_pos: positives per row."""
    B, F_s, L, F_in, H, K = wl.B, wl.F_s, wl.L, wl.F_in, wl.H, wl.K
    X = B * F_s * dt_bytes
    idx = K * F_in * 4
    W = L * F_in * dt_bytes
    Y = B * L * dt_bytes
    dW = L * F_in * 4
    dX = B * F_s * 4
    Wh, Yh, dWh = H * F_s * dt_bytes, B * H * dt_bytes, H * F_s * 4
    tail_flops = 2 * B * L * F_in
    head_flops = 2 * B * H * F_s
    pos = B * n_pos * 4
    c = {
        "fwd": (X + idx + W + Y, tail_flops),
        "fwd_bce": (X + idx + W + pos + Y + dW, 2 * tail_flops),   # writes dY (Y's size) and dW
        # reads W and the fp32 velocity, writes dY, the velocity and the next W
        "fwd_bce_sgd": (X + idx + 2 * W + pos + Y + 2 * dW, 2 * tail_flops),
        "sgd": (2 * W + 3 * dW, 0),
        "bce": (2 * Y + pos, 0),
        "bwd_w": (X + idx + Y + dW, tail_flops),
        "bwd_x": (idx + W + Y + dX, tail_flops),
    }
    c["tail_step"] = (c["fwd_bce"][0] + c["bwd_x"][0], c["fwd_bce"][1] + c["bwd_x"][1])   # both passes' operands
    c["tail_step_sgd"] = (c["fwd_bce_sgd"][0] + c["bwd_x"][0], c["fwd_bce_sgd"][1] + c["bwd_x"][1])
    if H:
        c["head_fwd"] = (X + Wh + Yh, head_flops)
        c["head_bce"] = (2 * Yh + pos, 0)
        c["head_fwd_bce"] = (X + Wh + pos + Yh, head_flops)   # writes dY_h (Y_h's size)
        c["head_sgd"] = (2 * Wh + 3 * dWh, 0)
        c["head_bwd"] = (X + Wh + Yh + dWh + 2 * dX, 2 * head_flops)
    return c


# source files of each call's kernels (the shared header is part of every call)
CALL_FILES = {
    "head_fwd": ["head.hip"], "head_fwd_bce": ["head.hip"], "head_bwd": ["head.hip", "util.hip"],
    "bce": ["util.hip"], "head_bce": ["util.hip"], "sgd": ["util.hip"], "head_sgd": ["util.hip"],
    "rewire": ["rewire.hip"], "grouping": ["group.hip"],
}


# a tail call runs, depending on the layer's shape, kernels of any of the tail files, and the
# fixed-order reductions of util.hip
TAIL_FILES = ["tail_mfma.hip", "tail_sg.hip", "tail_dense.hip", "tail_valu.hip", "util.hip"]


def kernel_source_hash(call=None):
    """Hash of the kernel sources: those of one call (default: the tail files), or all of them."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_01117_amd", "csrc")
    files = sorted(os.listdir(csrc)) if call is None else sorted(
        CALL_FILES.get(call, TAIL_FILES) + ["common.hpp"])
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def traffic_file(workload):
    return os.path.join(PROFILES, f"traffic_{workload}.txt")


def measured_traffic(workload, call):
    """HBM bytes per launch of a call's kernels from the committed rocprofv3 counter summary, if its
    counters were taken on the current kernel sources (null otherwise)."""
    try:
        with open(traffic_file(workload)) as fh:
            line = next(l for l in fh if l.startswith("{"))
        t = json.loads(line)
    except (OSError, ValueError, StopIteration):
        return None
    if t.get("call_source_hash", {}).get(call) != kernel_source_hash(call):
        return None
    return t.get("calls", {}).get(call)


def _short(name):
    n = name.replace("(anonymous namespace)::", "").replace("void ", "")
    return n.split("(")[0]


def _db_rows(db, query):
    import sqlite3
    con = sqlite3.connect(db)
    try:
        return con.execute(query).fetchall()
    finally:
        con.close()


def summarize_trace(db, workload, command):
    """Per-kernel launch counts and average durations from a rocprofv3 kernel-trace database."""
    rows = _db_rows(db, "select name, total_calls, total_duration, average, percentage from top_kernels")
    lines = [f"# Kernel times, workload {workload}", "",
             "rocprofv3 --kernel-trace --stats; durations in microseconds (average per launch).", "",
             f"Command: `{command}`", "", f"Kernel sources: {kernel_source_hash()}", "",
             "| kernel | launches | avg us | total us | % |", "|---|---|---|---|---|"]
    for name, n, tot, avg, pct in rows:
        lines.append(f"| `{_short(name)}` | {n} | {avg:.1f} | {tot:.1f} | {pct:.1f} |")
    path = os.path.join(PROFILES, f"kernels_{workload}.md")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(path)


def summarize_traffic(fetch_db, write_db, workload, command):
    """HBM bytes per kernel launch from FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by what
    the same counter reads for the plain COPY_BYTES device copy run in the same process."""
    def per_dispatch(db, counter):
        rows = _db_rows(db, f"select name, dispatch_id, sum(counter_value) from pmc_events "
                            f"where counter_name = '{counter}' group by name, dispatch_id")
        acc = {}
        for name, _, v in rows:
            acc.setdefault(_short(name), []).append(v * 1024.0)
        return acc
    fetch_d, write_d = per_dispatch(fetch_db, "FETCH_SIZE"), per_dispatch(write_db, "WRITE_SIZE")
    fetch = {k: sum(v) / len(v) for k, v in fetch_d.items()}
    write = {k: sum(v) / len(v) for k, v in write_d.items()}
    copy_keys = [k for k in fetch if "copy" in k.lower()]
    if not copy_keys:
        raise SystemExit("no copy kernel in the counter runs (run bench.py with --copy-calibration)")
    ck = max(copy_keys, key=lambda k: max(fetch_d[k]))
    # the calibration copies are the largest dispatches of the copy kernel (the same kernel also
    # moves the inputs from the host, in smaller pieces)
    f_fetch = COPY_BYTES / max(fetch_d[ck])
    f_write = COPY_BYTES / max(write_d[ck]) if write_d.get(ck) else None
    calls = {}
    for call, prefixes in CALL_KERNELS.items():
        ks = [k for k in fetch if any(re.match(p, k) for p in prefixes)]
        if not ks or f_write is None:
            continue
        # the tail's and the head's BCE gradient run one kernel: the tail's are its largest dispatches
        pick = SHARED_KERNEL_PICK.get(call)
        fv = (lambda k: pick(fetch_d[k])) if pick else (lambda k: fetch[k])
        wv = (lambda k: pick(write_d[k]) if k in write_d else 0.0) if pick else (lambda k: write.get(k, 0.0))
        calls[call] = round(sum(fv(k) * f_fetch + wv(k) * f_write for k in ks))
    rec = {"workload": workload, "kernel_source_hash": kernel_source_hash(),
           "call_source_hash": {c: kernel_source_hash(c) for c in calls}, "copy_kernel": ck,
           "fetch_factor": round(f_fetch, 4), "write_factor": round(f_write, 4), "calls": calls}
    lines = [f"HBM traffic per launch, workload {workload}",
             "rocprofv3 --pmc FETCH_SIZE, then --pmc WRITE_SIZE (KiB per dispatch), each scaled by the factor",
             f"that maps the same counter to the {COPY_BYTES} bytes a plain device copy ({ck}, its largest",
             "dispatches) reads or writes.",
             f"Command: {command}", "",
             "kernel | FETCH bytes (raw) | WRITE bytes (raw) | scaled HBM bytes"]
    for k in sorted(fetch, key=lambda k: -fetch[k]):
        sc = fetch[k] * f_fetch + write.get(k, 0.0) * f_write
        lines.append(f"{k} | {fetch[k]:.4g} | {write.get(k, 0.0):.4g} | {sc:.4g}")
    lines += ["", json.dumps(rec)]
    path = traffic_file(workload)
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(path)


def cpu_baseline(wl, X, idx, W, dY, Wh, dYh, pos_tail):
    """The fp64 oracle on a bounded sample of the same workload, scaled to ms per full step."""
    import oracle
    orc = oracle.get()
    dt = wl.dtype
    nl = min(wl.L, 32768)
    nb = min(wl.B, 4)
    nh = min(wl.H, 2048)
    parts = {}
    t = time.perf_counter(); z = orc.fwd(X, idx, W, None, wl.G, dt, 0, nl); parts["fwd"] = (time.perf_counter() - t) * wl.L / nl
    t = time.perf_counter(); orc.bce_grad(z, pos_tail); parts["bce"] = (time.perf_counter() - t) * wl.L / nl
    del z
    t = time.perf_counter(); orc.bwd_w(X, idx, dY, wl.G, wl.F_in, dt, 0, nl); parts["bwd_w"] = (time.perf_counter() - t) * wl.L / nl
    t = time.perf_counter(); orc.bwd_x(idx, W, dY, wl.G, wl.F_s, dt, 0, nb); parts["bwd_x"] = (time.perf_counter() - t) * wl.B / nb
    sample = f"tail fwd+BCE gradient+bwd_w on labels [0,{nl}), bwd_x on rows [0,{nb})"
    if wl.H:
        t = time.perf_counter(); orc.head_fwd(X, Wh, None, dt, 0, nh); parts["head_fwd"] = (time.perf_counter() - t) * wl.H / nh
        t = time.perf_counter(); orc.head_bwd_w(X, dYh, dt, 0, nh); tw = (time.perf_counter() - t) * wl.H / nh
        t = time.perf_counter(); orc.head_bwd_x(Wh, dYh, dt, 0, nb); parts["head_bwd"] = tw + (time.perf_counter() - t) * wl.B / nb
        sample += f"; head fwd+dW on heads [0,{nh}), head dX on rows [0,{nb})"
    ms = 1e3 * sum(parts.values())
    return {"value": round(ms, 1), "unit": "ms/step", "cores": orc.num_threads(), "kind": "oracle",
            "sample": sample + "; each part's time scaled by (full size / sampled size)",
            "per_call_ms": {k: round(1e3 * v, 1) for k, v in parts.items()}}


def warm_up(run_pass, min_passes):
    """Untimed passes before a timed phase: at least min_passes, and at least WARM_S seconds of them,
    so that the GPU's clocks have left the idle state that host-side setup (drawing inputs) leaves
    them in. With a few passes only, the first phase after such a pause ran about 12% slower in every
    kernel. Synchronises every four passes, so that the wall clock follows the GPU."""
    import torch
    t0, n = time.perf_counter(), 0
    while n < min_passes or time.perf_counter() - t0 < WARM_S:
        run_pass()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.workload, args.command)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, args.workload, args.command)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the layer's multi-GPU sharding "
              "is a design note, not a measured path.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_01117_amd as hs
    import synth

    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    X = synth.draw_X(wl)
    W = synth.draw_W(wl)
    idx = synth.draw_idx(wl)
    pos = synth.draw_positives(wl)
    perm = synth.draw_perm(wl)
    dY = synth.draw_dY(wl, positives=pos, perm=perm)
    Wh = synth.draw_W_head(wl) if wl.H else None
    dYh = synth.draw_dY_head(wl, positives=pos, perm=perm) if wl.H else None
    gen_s = time.perf_counter() - t0
    print(f"[bench] {wl.name}: inputs drawn in {gen_s:.1f}s", file=sys.stderr, flush=True)

    def up(a):
        if a is None:
            return None
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    is_bf = wl.dtype == synth.DT_BF16
    odt = torch.int16 if is_bf else torch.float32
    Xd, Wd, idxd, dYd = up(X), up(W), up(idx), up(dY)
    desc = hs.make_desc(wl.B, wl.F_s, wl.L, wl.G, wl.F_in, wl.dtype)
    Y = torch.empty((wl.B, wl.L), dtype=odt, device=dev)
    dW = torch.empty((wl.L, wl.F_in), dtype=torch.float32, device=dev)
    dX = torch.empty((wl.B, wl.F_s), dtype=torch.float32, device=dev)
    ws_w = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_W))
    ws_x = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_X))
    if wl.H:
        Whd, dYhd = up(Wh), up(dYh)
        Yh = torch.empty((wl.B, wl.H), dtype=odt, device=dev)
        dWh = torch.empty((wl.H, wl.F_s), dtype=torch.float32, device=dev)
        ws_h = hs.workspace(hs.haste_head_workspace_bytes(wl.B, wl.F_s, wl.H, wl.dtype))
    torch.cuda.synchronize()

    # positives as per-row column lists of the tail and of the head (-1 padded)
    tail_pairs, head_pairs = synth.positive_neurons(wl, pos, perm)
    n_pos = pos.shape[1]
    posd = up(synth.pos_matrix(tail_pairs, wl.B, n_pos))
    dYt = torch.empty((wl.B, wl.L), dtype=odt, device=dev)   # the training step's own dY
    ws_t = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP))
    if wl.H:
        posh = up(synth.pos_matrix(head_pairs, wl.B, n_pos))
        dYht = torch.empty((wl.B, wl.H), dtype=odt, device=dev)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def head_train(fused=True):
        if not wl.H:
            return []
        if fused:
            return [("head_fwd_bce", lambda: hs.haste_head_fwd_bce(wl.B, wl.F_s, wl.H, wl.dtype, Xd, Whd, None, posh,
                                                                   dYht))]
        return [("head_fwd", lambda: hs.haste_head_fwd(wl.B, wl.F_s, wl.H, wl.dtype, Xd, Whd, None, Yh)),
                ("head_bce", lambda: hs.haste_bce_grad(wl.B, wl.H, wl.dtype, Yh, posh, dYht))]

    def head_back(dyh):
        return [("head_bwd", lambda: hs.haste_head_bwd(wl.B, wl.F_s, wl.H, wl.dtype, Xd, Whd, dyh, dWh, dX, 1,
                                                       ws_h))] if wl.H else []

    fused = ([("tail_step", lambda: hs.haste_tail_step(desc, Xd, idxd, Wd, None, posd, dYt, dW, None, 0, dX, 0,
                                                        ws_t))] +
             head_train() + (head_back(dYht) if wl.H else []))
    unfused = ([("fwd", lambda: hs.haste_fwd(desc, Xd, idxd, Wd, None, Y)),
                ("bce", lambda: hs.haste_bce_grad(wl.B, wl.L, wl.dtype, Y, posd, dYt))] + head_train(False) +
               [("bwd_w", lambda: hs.haste_bwd_w(desc, Xd, idxd, dYt, dW, None, 0, ws_w)),
                ("bwd_x", lambda: hs.haste_bwd_x(desc, idxd, Wd, dYt, dX, 0, ws_x))] +
               (head_back(dYht) if wl.H else []))
    # the training pass with the optimizer (SGD with momentum on W and W_h): fused, the tail's step is
    # applied inside haste_fwd_bce_sgd and dW never reaches memory; unfused, dW is stored and stepped
    opt = hs.sgd_opts(0.01, 0.9, 0.0)
    mom = torch.zeros((wl.L, wl.F_in), dtype=torch.float32, device=dev)
    Wnext = torch.empty_like(Wd)
    if wl.H:
        mom_h = torch.zeros((wl.H, wl.F_s), dtype=torch.float32, device=dev)
        Whnext = torch.empty_like(Whd)
    head_step = ([("head_sgd", lambda: hs.haste_sgd_momentum(wl.H * wl.F_s, wl.dtype, Whd, dWh, mom_h, opt,
                                                             Whnext))] if wl.H else [])
    ws_ts = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP_SGD))
    fused_opt = ([("tail_step_sgd", lambda: hs.haste_tail_step_sgd(desc, Xd, idxd, Wd, None, posd, dYt, None, opt, mom,
                                                                   Wnext, dX, 0, ws_ts))] +
                 head_train() + (head_back(dYht) if wl.H else []) + head_step)
    unfused_opt = unfused + [("sgd", lambda: hs.haste_sgd_momentum(wl.L * wl.F_in, wl.dtype, Wd, dW, mom, opt,
                                                                   Wnext))] + head_step
    separate = [("fwd", lambda: hs.haste_fwd(desc, Xd, idxd, Wd, None, Y))]
    if wl.H:
        separate.append(("head_fwd", lambda: hs.haste_head_fwd(wl.B, wl.F_s, wl.H, wl.dtype, Xd, Whd, None, Yh)))
    separate.append(("bwd_w", lambda: hs.haste_bwd_w(desc, Xd, idxd, dYd, dW, None, 0, ws_w)))
    separate.append(("bwd_x", lambda: hs.haste_bwd_x(desc, idxd, Wd, dYd, dX, 0, ws_x)))
    separate += head_back(dYhd) if wl.H else []

    # a working set that fits the 256 MB MALL would be timed warm: flush it before every timed step
    # by writing a 512 MB buffer (outside the events that time the step)
    mall_flush = call_cost(wl, 2 if is_bf else 4, 0)["fwd"][0] + wl.B * wl.L * (2 if is_bf else 4) < (512 << 20)
    flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev) if mall_flush else None

    def timed(calls):
        """K steps after W warm-up steps; events between the calls on the launch stream."""
        for _ in range(args.warmup):
            for _, fn in calls:
                fn()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for s in range(args.steps):
            if flush_buf is not None:
                flush_buf.fill_(float(s))
            evs[s][0].record(stream)
            for i, (_, fn) in enumerate(calls):
                fn()
                evs[s][i + 1].record(stream)
        torch.cuda.synchronize()
        wall = (time.perf_counter() - w0) * 1e3 / args.steps
        per = {name: 0.0 for name, _ in calls}
        step = 0.0
        for s in range(args.steps):
            step += evs[s][0].elapsed_time(evs[s][-1])
            for i, (name, _) in enumerate(calls):
                per[name] += evs[s][i].elapsed_time(evs[s][i + 1])
        return step / args.steps, {k: v / args.steps for k, v in per.items()}, wall

    cost = call_cost(wl, 2 if is_bf else 4, n_pos)

    def detail(per):
        d = {}
        for name, ms in per.items():
            b, f = cost[name]
            d[name] = {"ms": round(ms, 4), "GBps": round(b / ms / 1e6, 1), "TFLOPs": round(f / ms / 1e9, 1),
                       "alg_bytes": b, "flops": f}
        return d

    warm_up(lambda: [fn() for _, fn in separate], 0)   # once, after the host-side input setup
    sep_ms, sep_per, _ = timed(separate)
    unf_ms, unf_per, _ = timed(unfused)
    step_ms, per_call, wall_ms = timed(fused)
    fo_ms, fo_per, _ = timed(fused_opt)
    uo_ms, uo_per, _ = timed(unfused_opt)

    step_bytes = sum(cost[k][0] for k in per_call)
    step_flops = sum(cost[k][1] for k in per_call)
    dom = max(per_call, key=per_call.get)
    db, df = cost[dom]
    achieved = db / per_call[dom] / 1e6
    roof = {"call": dom, "kernels": CALL_KERNELS[dom], "bound": "hbm", "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": measured_traffic(wl.name, dom), "alg_bytes_per_launch": db,
            "avg_launch_ms": round(per_call[dom], 4)}

    out = {
        "metric": "fwd+bwd ms/step (bf16, 3M-label tail); HBM GB/s and MFMA % of peak",
        "value": round(step_ms, 4), "unit": "ms/step", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if is_bf else "f32", "data": "synthetic (seeded; see synth/)",
        "config": {"workload": wl.name, "B": wl.B, "F_s": wl.F_s, "L_tail": wl.L, "G": wl.G, "F_in": wl.F_in,
                   "H_head": wl.H, "positives_per_row": int(n_pos), "parallelism": "single GPU"},
        "step": "training pass: fused tail forward + BCE gradient + backward-weight, head forward + BCE "
                "gradient, tail backward-feature, head backward",
        "labels_samples_per_s": round(wl.B * (wl.L + wl.H) / (step_ms / 1e3), 1),
        "step_alg_bytes": step_bytes,
        "step_hbm_GBps": round(step_bytes / step_ms / 1e6, 1),
        "step_hbm_frac": round(step_bytes / step_ms / 1e6 / HBM_PEAK_GBPS, 4),
        "step_mfma_pct": round(100 * step_flops / (step_ms / 1e3) / (MFMA_BF16_PEAK_TFLOPS * 1e12), 2),
        "wall_ms_per_step": round(wall_ms, 4),
        "mall_flush": bool(mall_flush),
        "per_call": detail(per_call),
        "roofline": roof,
        "unfused_training_step": {"ms": round(unf_ms, 4), "per_call": detail(unf_per),
                                  "what": "haste_fwd + haste_bce_grad + haste_bwd_w in place of haste_fwd_bce, haste_head_fwd + haste_bce_grad in place of haste_head_fwd_bce"},
        "training_step_with_optimizer": {
            "fused_ms": round(fo_ms, 4), "unfused_ms": round(uo_ms, 4),
            "fused_per_call_ms": {k: round(v, 4) for k, v in fo_per.items()},
            "unfused_per_call_ms": {k: round(v, 4) for k, v in uo_per.items()},
            "what": "the training pass plus one SGD-with-momentum step on W and W_h: fused, the tail's step runs "
                    "inside haste_tail_step_sgd (dW never stored) and the head's loss gradient inside "
                    "haste_head_fwd_bce; unfused, the unfused training step + haste_sgd_momentum"},
        "separate_calls_step": {
            "ms": round(sep_ms, 4), "per_call": detail(sep_per),
            "step_alg_bytes": sum(cost[k][0] for k in sep_per),
            "step_hbm_frac": round(sum(cost[k][0] for k in sep_per) / sep_ms / 1e6 / HBM_PEAK_GBPS, 4),
            "what": "haste_fwd, haste_head_fwd, haste_bwd_w, haste_bwd_x, haste_head_bwd on a fixed dY (no loss gradient)"},
    }

    if not args.no_bottleneck and is_bf:
        out["dense_bottleneck"] = bottleneck(wl, Xd, Wd, dYd, args)
        out["tail_vs_bottleneck"] = round(sum(per_call[k] for k in ("tail_step", "fwd_bce", "bwd_x") if k in per_call) /
                                          out["dense_bottleneck"]["ms"], 3)
        out["separate_calls_step"]["tail_vs_bottleneck"] = round(
            sum(sep_per[k] for k in ("fwd", "bwd_w", "bwd_x")) / out["dense_bottleneck"]["ms"], 3)
    # rewiring (Alg. 3) at rho = 0.1 on copies of the supports and weights, timed alone (it runs
    # every few hundred steps, not in the step)
    if wl.dtype == synth.DT_BF16 or wl.dtype == synth.DT_F32:
        idx_r, W_r = idxd.clone(), Wd.clone()
        ws_r = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_REWIRE))
        n_r = 0
        for _ in range(2):
            idx_r.copy_(idxd)
            W_r.copy_(Wd)
            n_r = hs.haste_rewire(desc, idx_r, W_r, None, 0.1, 1, 7, ws_r)
        torch.cuda.synchronize()
        r_ms = 0.0
        for it in range(5):
            idx_r.copy_(idxd)
            W_r.copy_(Wd)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            hs.haste_rewire(desc, idx_r, W_r, None, 0.1, 1, 7 + it, ws_r)
            e1.record(stream)
            torch.cuda.synchronize()
            r_ms += e0.elapsed_time(e1) / 5
        out["rewire"] = {"ms": round(r_ms, 4), "rho": 0.1, "pruned_slots": n_r,
                         "what": "haste_rewire (Alg. 3) on the layer's supports and weights, random reinit"}
        del idx_r, W_r, ws_r
    # grouping (Alg. 2), done once before training: the tail's labels as 768-dimensional int8 unit
    # embeddings around planted directions (drawn on the device from a seeded generator), at the
    # tail size of the 655K-label layer, bucket factor 16
    if args.grouping:
        gN, gD, gG, gbeta, giters = 655360, 768, 32, 16, 10
        gen = torch.Generator(device=dev).manual_seed(17)
        mu = torch.randn((4096, gD), device=dev, generator=gen)
        lab = torch.randint(0, 4096, (gN,), device=dev, generator=gen)
        Xg = mu[lab] / mu[lab].norm(dim=1, keepdim=True) + 0.3 / gD ** 0.5 * torch.randn((gN, gD), device=dev,
                                                                                     generator=gen)
        Eg = torch.round(127 * Xg / Xg.norm(dim=1, keepdim=True)).to(torch.int8)
        del mu, lab, Xg
        gopts = hs.group_opts(gG, gbeta, giters, 5)
        g_order = torch.empty(gN, dtype=torch.int32, device=dev)
        g_size = torch.empty(gN, dtype=torch.int32, device=dev)
        g_n = torch.empty(1, dtype=torch.int64, device=dev)
        ws_g = hs.workspace(hs.haste_group_workspace_bytes(gN, gD, gopts))
        hs.haste_group_labels(Eg, gopts, g_order, g_size, g_n, None, ws_g)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        hs.haste_group_labels(Eg, gopts, g_order, g_size, g_n, None, ws_g)
        e1.record(stream)
        torch.cuda.synchronize()
        out["grouping"] = {"ms": round(e0.elapsed_time(e1), 3), "N": gN, "D": gD, "G": gG, "beta": gbeta,
                           "iters": giters, "groups": int(g_n.item()),
                           "what": "haste_group_labels (Alg. 2) on planted int8 unit embeddings"}
        del Eg, g_order, g_size, ws_g
    if not args.no_gsweep and wl.name == "l2949k_g32_h65k":
        print("[bench] group-size sweep", file=sys.stderr, flush=True)
        out["gsweep"] = gsweep(args, hs, synth, torch, np)
    if args.copy_calibration:
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, X, idx, W, dY, Wh, dYh, synth.pos_matrix(tail_pairs, wl.B, n_pos))
    print(json.dumps(out), flush=True)


def gsweep(args, hs, synth, torch, np):
    """The group-size sweep (Fig. 4's axis) on the 655K-label layer (B = 256, F_s = 768, F_in = 64):
    for G = 1 (standard fixed fan-in), 4, 16 and 64 the training pass of the tail (haste_tail_step)
    and the separate calls on a fixed dY, with the FLOPs-matched dense bottleneck timed beside them.
    X, W and dY are shared by every G; each G has its own supports."""
    dev = torch.device("cuda:0")
    base = synth.WORKLOADS["gsweep_g16"]
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if a.dtype == np.uint16 else
                                    np.ascontiguousarray(a)).to(dev)
    Xd, Wd = up(synth.draw_X(base)), up(synth.draw_W(base))
    pos = synth.draw_positives(base)
    perm = synth.draw_perm(base)
    dYd = up(synth.draw_dY(base, positives=pos, perm=perm))
    tail_pairs, _ = synth.positive_neurons(base, pos, perm)
    posd = up(synth.pos_matrix(tail_pairs, base.B, pos.shape[1]))
    B, F_s, L, F_in = base.B, base.F_s, base.L, base.F_in
    Y = torch.empty((B, L), dtype=torch.int16, device=dev)
    dYt = torch.empty((B, L), dtype=torch.int16, device=dev)
    dW = torch.empty((L, F_in), dtype=torch.float32, device=dev)
    dX = torch.empty((B, F_s), dtype=torch.float32, device=dev)
    st = torch.cuda.current_stream()

    def time_it(fns, n):
        """Mean ms per pass of the calls in order, and of each call (events between the calls), over n
        passes after the warm-up passes. The calls of a pass run back to back, as in a step, so no
        call is timed with its working set left in the caches by a repeat of itself."""
        warm_up(lambda: [f() for f in fns], max(1, args.warmup))
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)] for _ in range(n)]
        for r in range(n):
            evs[r][0].record(st)
            for i, f in enumerate(fns):
                f()
                evs[r][i + 1].record(st)
        torch.cuda.synchronize()
        per = [sum(evs[r][i].elapsed_time(evs[r][i + 1]) for r in range(n)) / n for i in range(len(fns))]
        return sum(evs[r][0].elapsed_time(evs[r][-1]) for r in range(n)) / n, per

    n = max(3, min(args.steps, 10))
    res = {}
    for G in (1, 4, 16, 64):
        wl = synth.WORKLOADS[f"gsweep_g{G}"]
        idxd = up(synth.draw_idx(wl))
        desc = hs.make_desc(B, F_s, L, G, F_in, hs.HASTE_DTYPE_BF16)
        ws_t = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_TAIL_STEP))
        ws_w = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_W))
        ws_x = hs.workspace(hs.haste_workspace_bytes(desc, hs.HASTE_OP_BWD_X))
        step, _ = time_it([lambda: hs.haste_tail_step(desc, Xd, idxd, Wd, None, posd, dYt, dW, None, 0, dX, 0, ws_t)], n)
        sep, (f, w, x) = time_it([lambda: hs.haste_fwd(desc, Xd, idxd, Wd, None, Y),
                                  lambda: hs.haste_bwd_w(desc, Xd, idxd, dYd, dW, None, 0, ws_w),
                                  lambda: hs.haste_bwd_x(desc, idxd, Wd, dYd, dX, 0, ws_x)], n)
        res[f"G{G}"] = {"tail_step_ms": round(step, 4), "fwd_ms": round(f, 4), "bwd_w_ms": round(w, 4),
                        "bwd_x_ms": round(x, 4), "separate_ms": round(sep, 4)}
        del idxd, ws_t, ws_w, ws_x
    bn = bottleneck(base, Xd, Wd, dYd, args)
    res["dense_bottleneck_ms"] = bn["ms"]
    for G in (1, 4, 16, 64):
        res[f"G{G}"]["separate_vs_bottleneck"] = round(res[f"G{G}"]["separate_ms"] / bn["ms"], 3)
    res["what"] = ("655K-label layer, B=256, F_s=768, F_in=64, bf16: haste_tail_step (forward + BCE gradient + "
                   "backward-weight + backward-feature) and the separate fwd / bwd_w / bwd_x calls on a fixed dY "
                   "per group size (G=1 is standard fixed fan-in), the separate calls timed back to back per pass "
                   "like the dense bottleneck, [256,64]x[64,655360] fwd + dW + dX with torch.matmul")
    return res


def bottleneck(wl, Xd, Wd, dYd, args):
    """FLOPs-matched dense bottleneck: a dense layer of width F_in over all L labels, fwd + dW + dX
    via torch.matmul (hipBLASLt), bf16 in and out, every operand contiguous."""
    import torch
    bf = lambda t: t.view(torch.bfloat16)
    Xr = bf(Xd)[:, : wl.F_in].contiguous()            # [B, F_in]
    Wt = bf(Wd).t().contiguous()                       # [F_in, L]
    Wn = bf(Wd)                                        # [L, F_in]
    dY = bf(dYd)                                       # [B, L]
    dYt = dY.t().contiguous()                          # [L, B]
    ops = [lambda: torch.matmul(Xr, Wt), lambda: torch.matmul(dYt, Xr), lambda: torch.matmul(dY, Wn)]
    warm_up(lambda: [f() for f in ops], args.warmup)
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(args.steps):
        for f in ops:
            f()
    e1.record(st)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    del Wt, dYt
    return {"ms": round(ms, 4), "what": "[B,F_in]x[F_in,L] fwd + dW + dX, torch.matmul bf16 (dW, dX in bf16)"}


if __name__ == "__main__":
    main()
