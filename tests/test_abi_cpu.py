"""Host-side checks of the C ABI: the library loads, exports every declared entry point, and
rejects invalid arguments before anything is launched (no GPU needed: no call here reaches a
kernel launch)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "haste.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(haste_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def hs():
    from paper_2606_01117_amd import LIB_PATH
    if not os.path.exists(LIB_PATH):
        from paper_2606_01117_amd import build
        build.build()
    import paper_2606_01117_amd as m
    return m


def test_header_declares_the_five_layer_calls():
    names = _declared()
    for n in ("haste_fwd", "haste_bwd_w", "haste_bwd_x", "haste_head_fwd", "haste_head_bwd"):
        assert n in names


def test_library_exports_every_declared_symbol(hs):
    names = _declared()
    out = subprocess.run(["nm", "-D", "--defined-only", hs.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (haste_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, f"declared but not exported: {missing}"
    for n in names:
        assert hasattr(hs.lib, n)
    assert set(hs.EXPORTS) == set(names)


def test_version_and_status_strings(hs):
    assert "gfx950" in hs.haste_version()
    assert hs.haste_status_str(0) == "ok"
    assert hs.haste_status_str(3) == "workspace too small"


FAKE = 1 << 20  # an aligned non-null address; validation fails before it could be dereferenced


def _desc(hs, **kw):
    d = dict(B=8, F_s=64, L=32, G=4, F_in=8, dtype=hs.HASTE_DTYPE_BF16)
    d.update(kw)
    return hs.make_desc(**d)


@pytest.mark.parametrize("kw,what", [
    (dict(L=30, G=4), "multiple of G"),
    (dict(F_in=0), "F_in"),
    (dict(F_in=65), "F_in"),
    (dict(G=0), "G must"),
    (dict(dtype=7), "dtype"),
    (dict(B=-1), "B and L"),
])
def test_invalid_descriptors_rejected(hs, kw, what):
    d = _desc(hs, **kw)
    rc = hs.lib.haste_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, None, 0, None)
    assert rc == 1
    assert what in hs.haste_last_error()
    assert hs.haste_workspace_bytes(d, hs.HASTE_OP_BWD_X) == 0


def test_null_and_misaligned_pointers_rejected(hs):
    d = _desc(hs)
    assert hs.lib.haste_fwd(ctypes.byref(d), None, FAKE, FAKE, None, FAKE, None, 0, None) == 1
    assert "X is NULL" in hs.haste_last_error()
    assert hs.lib.haste_fwd(ctypes.byref(d), FAKE + 2, FAKE, FAKE, None, FAKE, None, 0, None) == 1
    assert "aligned" in hs.haste_last_error()
    assert hs.lib.haste_bwd_w(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, 2, None, 0, None) == 1
    assert "beta" in hs.haste_last_error()


def test_unsupported_width_reported(hs):
    d = _desc(hs, F_s=4096, F_in=64)
    assert hs.lib.haste_fwd(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, None, 0, None) == 2


def test_workspace_too_small_rejected(hs):
    d = hs.make_desc(128, 768, 4096, 32, 64, hs.HASTE_DTYPE_BF16)
    need_x = hs.haste_workspace_bytes(d, hs.HASTE_OP_BWD_X)
    need_w = hs.haste_workspace_bytes(d, hs.HASTE_OP_BWD_W)
    assert need_x > 0 and need_w > 0
    assert hs.haste_workspace_bytes(d, hs.HASTE_OP_FWD) == 0
    assert hs.lib.haste_bwd_x(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, 0, FAKE, need_x - 1, None) == 3
    assert str(need_x) in hs.haste_last_error()
    assert hs.lib.haste_bwd_w(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, 0, None, 0, None) == 3
    assert hs.lib.haste_head_bwd(64, 768, 1024, 1, FAKE, FAKE, FAKE, FAKE, FAKE, 0, None, 0, None) == 3
    assert hs.haste_head_workspace_bytes(64, 768, 1024, 1) > 0


def test_workspace_sizes_scale_with_shape(hs):
    # backward-feature: fp32 [F_s x batch-tile] partials per label segment and tile; the bf16
    # path also keeps a group-transposed copy of W (L x F_in bf16, G padded to 8)
    small = hs.haste_workspace_bytes(hs.make_desc(32, 256, 4096, 8, 32, hs.HASTE_DTYPE_F32), hs.HASTE_OP_BWD_X)
    big = hs.haste_workspace_bytes(hs.make_desc(512, 768, 2949120, 32, 64, hs.HASTE_DTYPE_BF16), hs.HASTE_OP_BWD_X)
    wt = 2949120 * 64 * 2
    assert 0 < small < 256 << 20
    assert wt < big < wt + (256 << 20)


def test_debug_gather_range_checked(hs):
    d = _desc(hs)
    assert hs.lib.haste_debug_gather(ctypes.byref(d), FAKE, FAKE, 7, 2, FAKE, None) == 1
    assert "group range" in hs.haste_last_error()


def test_loss_optimizer_rewire_group_arguments_checked(hs):
    """The entry points added beside the layer calls reject bad arguments before any launch."""
    d = hs.make_desc(128, 768, 4096, 32, 64, hs.HASTE_DTYPE_BF16)
    # loss gradient: negative P, dbias without dW, missing workspace
    assert hs.lib.haste_fwd_bce(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, -1, FAKE, FAKE, None, 0, FAKE,
                                1 << 30, None) == 1
    assert hs.lib.haste_fwd_bce(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, 0, FAKE, None, FAKE, 0, FAKE,
                                1 << 30, None) == 1
    assert "dbias needs dW" in hs.haste_last_error()
    assert hs.lib.haste_fwd_bce(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, 0, FAKE, FAKE, None, 0, None, 0,
                                None) == 3
    assert hs.lib.haste_bce_grad(4, 8, 9, FAKE, None, 0, FAKE, None) == 1
    # head forward with the loss gradient: negative P, positives named but missing, unaligned bias
    assert hs.lib.haste_head_fwd_bce(4, 768, 1024, 1, FAKE, FAKE, None, FAKE, -1, FAKE, None) == 1
    assert hs.lib.haste_head_fwd_bce(4, 768, 1024, 1, FAKE, FAKE, None, None, 3, FAKE, None) == 1
    assert "pos" in hs.haste_last_error()
    assert hs.lib.haste_head_fwd_bce(4, 768, 1024, 1, FAKE, FAKE, FAKE + 4, None, 0, FAKE, None) == 1
    assert hs.lib.haste_head_fwd_bce(0, 768, 1024, 1, None, None, None, None, 0, None, None) == 0
    # optimizer: momentum outside [0, 1), W_next overlapping W
    bad = hs.sgd_opts(0.1, 1.0)
    assert hs.lib.haste_sgd_momentum(16, 1, FAKE, FAKE, FAKE, ctypes.byref(bad), FAKE, None) == 1
    assert "momentum" in hs.haste_last_error()
    ok = hs.sgd_opts(0.1, 0.9)
    ws = hs.haste_workspace_bytes(d, hs.HASTE_OP_FWD_BCE_SGD)
    assert ws > 0
    assert hs.lib.haste_fwd_bce_sgd(ctypes.byref(d), FAKE, FAKE, FAKE, None, None, 0, FAKE, None, ctypes.byref(ok),
                                    FAKE, FAKE + 64, FAKE, ws, None) == 1
    assert "overlaps" in hs.haste_last_error()
    # rewiring: rho outside [0, 1), init mode, width
    ws_r = hs.haste_workspace_bytes(d, hs.HASTE_OP_REWIRE)
    assert ws_r > 0
    assert hs.lib.haste_rewire(ctypes.byref(d), FAKE, FAKE, None, 1.0, 1, 0, None, FAKE, ws_r, None) == 1
    assert hs.lib.haste_rewire(ctypes.byref(d), FAKE, FAKE, None, 0.1, 2, 0, None, FAKE, ws_r, None) == 1
    wide = hs.make_desc(8, 1024, 4096, 16, 512, hs.HASTE_DTYPE_BF16)
    assert hs.lib.haste_rewire(ctypes.byref(wide), FAKE, FAKE, None, 0.1, 1, 0, None, FAKE, 1 << 30, None) == 2
    # rho = 0 prunes nothing: no launch, no workspace needed
    n = ctypes.c_int64(-1)
    assert hs.lib.haste_rewire(ctypes.byref(d), FAKE, FAKE, None, 0.0, 1, 0, ctypes.byref(n), None, 0, None) == 0
    assert n.value == 0
    # grouping: dimensions must be a multiple of 16; G within 1 .. 256
    g = hs.group_opts(32, 16, 5, 1)
    assert hs.haste_group_workspace_bytes(1000, 100, g) == 0
    assert hs.lib.haste_group_labels(1000, 100, FAKE, ctypes.byref(g), FAKE, FAKE, FAKE, None, FAKE, 1 << 30,
                                     None) == 2
    assert hs.haste_group_workspace_bytes(1000, 128, hs.group_opts(300, 16, 5, 1)) == 0
    assert hs.haste_group_workspace_bytes(1000, 128, g) > 0


def test_fwd_bce_static_limits(hs):
    """The no-workspace variant refuses a layer whose scratch exceeds its per-device array, and
    reports invalid descriptors as haste_fwd_bce does, before any device call."""
    assert hs.haste_fwd_bce_static_max_bytes() == 8 << 20
    big = hs.make_desc(8192, 768, 4096, 32, 64, hs.HASTE_DTYPE_BF16)     # 2 * 768 * 8192 + 256 > 8 MiB
    assert hs.haste_workspace_bytes(big, hs.HASTE_OP_FWD_BCE) > 8 << 20
    rc = hs.lib.haste_fwd_bce_static(ctypes.byref(big), FAKE, FAKE, FAKE, None, None, 0, FAKE, FAKE, None, 0, None)
    assert rc == 2 and b"8388608" in hs.lib.haste_last_error()
    bad = _desc(hs, L=30)                                               # L % G != 0
    rc = hs.lib.haste_fwd_bce_static(ctypes.byref(bad), FAKE, FAKE, FAKE, None, None, 0, FAKE, FAKE, None, 0, None)
    assert rc == 1
