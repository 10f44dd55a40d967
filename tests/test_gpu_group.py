"""GPU parity of haste_group_labels (Alg. 2, through the C ABI) against the CPU oracle.

Both sides take every decision in fp64 from exact integers (a centre is its members' exact sum;
a label's score for a centre is e.s / |s|; a greedy similarity is the cosine of two int8 rows),
and the draws come from the same counter-based generator on both sides, so the clusters, the
groups and their order must match the oracle exactly.  The cases include rows of uneven norm
(where a dot product and a cosine rank differently), near-duplicate rows, and clusters large
enough that their sums need all four digit planes of the int8 products.  At the size of the 655K-label tail (too slow for the oracle) the
output is checked for what holds at any size: a partition into groups of G (the last of each
cluster may be short), each group inside one cluster.
"""
import numpy as np
import pytest

import oracle
from gpu_helpers import say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hs():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2606_01117_amd as m
    return m


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


def planted(N, D, P, rng, noise=0.3):
    """int8 unit embeddings around P random directions (labels in random order)."""
    mu = rng.standard_normal((P, D)).astype(np.float32)
    mu /= np.linalg.norm(mu, axis=1, keepdims=True)
    lab = rng.integers(0, P, N)
    out = np.empty((N, D), np.int8)
    for r0 in range(0, N, 65536):                        # in chunks: the tail-size case is 655K x 768
        r1 = min(N, r0 + 65536)
        X = mu[lab[r0:r1]] + np.float32(noise / np.sqrt(D)) * rng.standard_normal((r1 - r0, D), dtype=np.float32)
        out[r0:r1] = np.rint(127 * X / np.linalg.norm(X, axis=1, keepdims=True))
    return out


def _run(hs, E, G, beta, iters, seed):
    import torch
    N, D = E.shape
    opts = hs.group_opts(G, beta, iters, seed)
    order = torch.empty(N, dtype=torch.int32, device="cuda")
    gsize = torch.empty(N, dtype=torch.int32, device="cuda")
    ng = torch.empty(1, dtype=torch.int64, device="cuda")
    cl = torch.empty(N, dtype=torch.int32, device="cuda")
    Ed = to_dev(E)
    hs.haste_group_labels(Ed, opts, order, gsize, ng, cl, hs.workspace(hs.haste_group_workspace_bytes(N, D, opts)))
    torch.cuda.synchronize()
    n = int(ng.item())
    return order.cpu().numpy(), gsize.cpu().numpy()[:n], cl.cpu().numpy()


def uneven(N, D, rng):
    """int8 rows of uneven norm with exact and near duplicates (non-zero rows)."""
    E = (rng.integers(-127, 128, (N, D)) * (0.1 + 0.9 * rng.random((N, 1)))).astype(np.int8)
    E[np.abs(E).astype(np.int32).sum(axis=1) == 0, 0] = 1
    E[1::7] = E[0:-1:7]                                                  # exact duplicates
    E[3::11] = np.clip(E[2:-1:11].astype(np.int32) + rng.integers(-1, 2, E[2:-1:11].shape), -127, 127)
    return E


def two_axes(n, D, n_mid, rng):
    """Two clusters of n labels near the axes e_0 and e_1, plus n_mid labels between them: the
    clusters' sums reach 127 n (four digit planes from n = 66,052) and the labels in between are
    decided by the exact scores."""
    E = np.zeros((2 * n + n_mid, D), np.int64)
    E[:n, 0] = 127
    E[n:2 * n, 1] = 127
    E[:2 * n, 2:] = rng.integers(-3, 4, (2 * n, D - 2))
    t = rng.random(n_mid) * 0.2 + 0.4
    E[2 * n:, 0] = np.rint(127 * np.cos(t * np.pi / 2))
    E[2 * n:, 1] = np.rint(127 * np.sin(t * np.pi / 2))
    E[2 * n:, 2:] = rng.integers(-2, 3, (n_mid, D - 2))
    return E[rng.permutation(E.shape[0])].astype(np.int8)


CASES = [
    # name, N, D, planted clusters (0: isotropic, -1: uneven norms, -2: two axes), G, beta, iters
    ("planted_2048_d64", 2048, 64, 8, 16, 16, 8),
    ("random_5000_d128", 5000, 128, 0, 32, 4, 4),
    ("d48_tail_chunk", 3000, 48, 20, 16, 8, 5),
    ("one_cluster", 300, 32, 5, 8, 64, 3),
    ("planted_50k_d256", 50000, 256, 200, 32, 16, 5),
    ("uneven_norms_3000_d32", 3000, 32, -1, 8, 8, 4),
    ("two_axes_141k_d16", 141000, 16, -2, 256, 275, 2),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_group_exact(hs, orc, case):
    name, N, D, P, G, beta, iters = case
    say(f"[group] {name}: N={N} D={D} G={G} beta={beta} iters={iters}")
    rng = np.random.default_rng(N + D)
    if P == -1:
        E = uneven(N, D, rng)
    elif P == -2:
        E = two_axes(70000, D, N - 140000, rng)
    elif P:
        E = planted(N, D, P, rng)
    else:
        X = rng.standard_normal((N, D))
        E = np.rint(127 * X / np.linalg.norm(X, axis=1, keepdims=True)).astype(np.int8)
    seed = 0xC0FFEE + N
    order, gs, cl = _run(hs, E, G, beta, iters, seed)
    order_o, gs_o, cl_o = orc.group_labels(E, G, beta, iters, seed)
    say(f"    {gs.size} groups")
    assert np.array_equal(cl, cl_o), "cluster assignment differs from the oracle"
    assert np.array_equal(gs, gs_o), "group sizes differ from the oracle"
    assert np.array_equal(order, order_o), "groups differ from the oracle"


def test_group_tail_size(hs):
    """The 655K-label tail with 768-dimensional embeddings (the paper's bucket factor 16)."""
    N, D, G, beta = 655360, 768, 32, 16
    rng = np.random.default_rng(3)
    E = planted(N, D, 4096, rng)
    say(f"[group] tail size N={N} D={D}")
    order, gs, cl = _run(hs, E, G, beta, 5, 99)
    C = N // (beta * G)
    assert sorted(order.tolist()) == list(range(N)), "groups must partition the labels"
    assert cl.min() >= 0 and cl.max() < C
    starts = np.concatenate([[0], np.cumsum(gs)])
    gcl = cl[order[starts[:-1]]]
    for i in range(0, gs.size, 97):                      # a sample of groups: one cluster each
        assert np.all(cl[order[starts[i]:starts[i + 1]]] == gcl[i])
    counts = np.bincount(cl, minlength=C)
    assert gs.size == int(np.sum(-(-counts // G))), "groups per cluster"
    assert gs.max() <= G and np.sum(gs < G) <= C, "only the last group of a cluster may be short"
