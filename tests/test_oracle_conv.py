"""Pins of the oracle's short causal convolution and conv-state commit.

The GDN layer mixes each channel over the last K = 4 tokens with a depthwise
causal convolution and SiLU before the recurrent core; its conv state C (the
last K-1 committed inputs) is the second per-layer state next to S (§7).  Each
pin below is a library routine (torch's grouped conv1d and SiLU), a closed
form, an invariant, or exact rational brute force on tiny inputs; none re-types
the oracle's loops.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2607_16673_amd import inputs


def rng(seed):
    return np.random.default_rng(seed)


def root_path(parent, j):
    p = []
    while j != -1:
        p.append(j)
        j = int(parent[j])
    return p[::-1]


def library_conv_last(seq, w, bias, activation):
    """torch conv1d (depthwise, no padding) over seq [L][D] at its last position."""
    D, K = w.shape
    t = torch.from_numpy(np.ascontiguousarray(seq.T))[None]  # [1][D][L]
    wt = torch.from_numpy(np.ascontiguousarray(w))[:, None, :]  # [D][1][K]
    bt = torch.from_numpy(bias) if bias is not None else None
    y = F.conv1d(t, wt, bt, groups=D)[0, :, -1]
    return (F.silu(y) if activation else y).numpy()


def random_forest(r, n):
    return np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32)


@pytest.mark.parametrize("K", [1, 2, 3, 4])
@pytest.mark.parametrize("activation", [True, False])
def test_chain_equals_library_conv1d(K, activation):
    """A chain draft is an ordinary causal sequence behind the committed inputs:
    every output equals torch's grouped conv1d over [C; x] followed by SiLU."""
    r = rng(10 + K)
    B, n, D = 2, 7, 12
    x = r.standard_normal((B, n, D))
    C = r.standard_normal((B, K - 1, D))
    w = r.standard_normal((D, K))
    bias = r.standard_normal(D)
    par = np.tile(inputs.chain(n), (B, 1))
    y, st = oracle.conv_verify(C, x, w, bias, par, activation=activation)
    assert (st == 0).all()
    for b in range(B):
        seq = np.concatenate([C[b], x[b]])  # [K-1+n][D]
        t = torch.from_numpy(np.ascontiguousarray(seq.T))[None]
        ref = F.conv1d(t, torch.from_numpy(w)[:, None, :], torch.from_numpy(bias), groups=D)[0].T
        if activation:
            ref = F.silu(ref)
        np.testing.assert_allclose(y[b], ref.numpy(), rtol=1e-13, atol=1e-13)


def test_tree_node_equals_conv_over_its_root_path():
    """Every node sees only its own root path (tree mask, §4.2) behind C."""
    r = rng(20)
    B, n, D, K = 3, 20, 6, 4
    pars = [inputs.random_tree(r, n, 6, 3), random_forest(r, n), np.full(n, -1, np.int32)]
    par = np.stack(pars)
    x = r.standard_normal((B, n, D))
    C = r.standard_normal((B, K - 1, D))
    w = r.standard_normal((D, K))
    bias = r.standard_normal(D)
    y, st = oracle.conv_verify(C, x, w, bias, par)
    assert (st == 0).all()
    for b in range(B):
        for j in range(n):
            seq = np.concatenate([C[b], x[b, root_path(par[b], j)]])
            np.testing.assert_allclose(y[b, j], library_conv_last(seq, w, bias, True), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("K", [2, 4])
def test_one_hot_tap_selects_ancestor_or_committed_row(K):
    """With one tap at lag s (identity activation, no bias) node j outputs its
    s-th ancestor's input if depth(j) > s, else committed row C[K-2-(s-depth(j))]:
    the window's indexing, exactly."""
    r = rng(30 + K)
    B, n, D = 2, 24, 5
    par = np.stack([inputs.random_tree(r, n, 7, 3), random_forest(r, n)])
    x = r.standard_normal((B, n, D))
    C = r.standard_normal((B, K - 1, D))
    for s in range(K):
        w = np.zeros((D, K))
        w[:, K - 1 - s] = 1.0
        y, st = oracle.conv_verify(C, x, w, None, par, activation=False)
        assert (st == 0).all()
        for b in range(B):
            for j in range(n):
                p = root_path(par[b], j)
                d = len(p)
                want = x[b, p[d - 1 - s]] if s < d else C[b, K - 2 - (s - d)]
                np.testing.assert_array_equal(y[b, j], want)


def test_sibling_isolation():
    """Changing x_j changes exactly the outputs of the nodes within K-1
    generations below j (j included); every other output keeps its bits."""
    r = rng(40)
    B, n, D, K = 1, 24, 4, 4
    par = inputs.random_tree(r, n, 8, 3)[None]
    x = r.standard_normal((B, n, D))
    C = r.standard_normal((B, K - 1, D))
    w = r.standard_normal((D, K))
    y0, _ = oracle.conv_verify(C, x, w, None, par)
    for j in range(n):
        x2 = x.copy()
        x2[0, j] += 1.0
        y1, _ = oracle.conv_verify(C, x2, w, None, par)
        for m in range(n):
            p = root_path(par[0], m)
            affected = j in p and len(p) - 1 - p.index(j) <= K - 1
            assert (not np.array_equal(y0[0, m], y1[0, m])) == affected, (j, m)


def test_commit_closed_form_and_prefix_invariance():
    """Commit keeps the last K-1 rows of [C; x_a1 .. x_aA] (bit-exact copies).
    Verifying node j from the committed prefix of its own path, as a chain of
    the rest, reproduces its tree output bit for bit."""
    r = rng(50)
    B, n, D, K = 1, 18, 6, 4
    par = inputs.random_tree(r, n, 7, 3)[None]
    x = r.standard_normal((B, n, D))
    C = r.standard_normal((B, K - 1, D))
    w = r.standard_normal((D, K))
    bias = r.standard_normal(D)
    y, _ = oracle.conv_verify(C, x, w, bias, par)
    for j in range(n):
        p = root_path(par[0], j)
        for t in range(len(p) + 1):
            path = np.full((1, n), -1, np.int32)
            path[0, :t] = p[:t]
            C1, st = oracle.conv_commit(C, x, par, path, np.array([t], np.int32))
            assert st[0] == 0
            full = np.concatenate([C[0], x[0, p[:t]]])
            np.testing.assert_array_equal(C1[0], full[len(full) - (K - 1):])
            rest = p[t:]
            if not rest:
                continue
            xs = x[:, rest]
            yc, st = oracle.conv_verify(C1, xs, w, bias, inputs.chain(len(rest))[None])
            assert st[0] == 0
            np.testing.assert_array_equal(yc[0, -1], y[0, j])


def test_commit_rejects_non_root_paths_and_leaves_state():
    r = rng(60)
    n, D, K = 8, 3, 4
    par = np.array([[-1, 0, 1, 1, 3, -1, 5, 2]], np.int32)
    x = r.standard_normal((1, n, D))
    C = r.standard_normal((1, K - 1, D))
    for path, ln in [([1, 2], 2), ([0, 2, 1], 3), ([0, 1, 9], 3), ([0], 9), ([0], -1)]:
        p = np.full((1, n), -1, np.int32)
        p[0, :len(path)] = path
        C1, st = oracle.conv_commit(C, x, par, p, np.array([ln], np.int32))
        assert st[0] == oracle.ERR_PATH
        np.testing.assert_array_equal(C1, C)


def test_invalid_topology_is_reported():
    x = np.zeros((2, 4, 3))
    par = np.array([[-1, 0, 1, 2], [-1, 2, 0, 1]], np.int32)
    _, st = oracle.conv_verify(np.zeros((2, 3, 3)), x, np.ones((3, 4)), None, par)
    assert st[0] == 0 and st[1] == oracle.ERR_TOPOLOGY


def test_silu_is_torch_silu_and_zero_input_gives_silu_bias():
    r = rng(70)
    B, n, D, K = 2, 9, 7, 4
    par = np.stack([inputs.random_tree(r, n, 4, 3) for _ in range(B)])
    x = r.standard_normal((B, n, D)) * 3
    C = r.standard_normal((B, K - 1, D))
    w = r.standard_normal((D, K))
    bias = r.standard_normal(D)
    pre, _ = oracle.conv_verify(C, x, w, bias, par, activation=False)
    post, _ = oracle.conv_verify(C, x, w, bias, par, activation=True)
    np.testing.assert_allclose(post, F.silu(torch.from_numpy(pre)).numpy(), rtol=1e-14, atol=1e-15)
    z, _ = oracle.conv_verify(np.zeros_like(C), np.zeros_like(x), w, bias, par)
    np.testing.assert_allclose(z, np.broadcast_to(F.silu(torch.from_numpy(bias)).numpy(), z.shape),
                               rtol=1e-15, atol=0)


def test_exact_rational_brute_force_every_small_parent_array():
    """Every parent array with parent[j] in [-1, j) for n <= 5, dyadic inputs,
    exact Fraction arithmetic: pre-activation outputs and every root-path commit
    agree exactly (dyadic fp64 sums of a few terms are exact)."""
    r = rng(80)
    D, K = 2, 3
    for n in range(1, 6):
        x = r.integers(-8, 9, (1, n, D)) / 4.0
        C = r.integers(-8, 9, (1, K - 1, D)) / 4.0
        w = r.integers(-4, 5, (D, K)) / 2.0
        bias = r.integers(-4, 5, D) / 8.0
        for par in itertools.product(*[range(-1, j) for j in range(n)]):
            par = np.array(par, np.int32)[None]
            y, st = oracle.conv_verify(C, x, w, bias, par, activation=False)
            assert st[0] == 0
            for j in range(n):
                p = root_path(par[0], j)
                rows = [C[0, i] for i in range(K - 1)] + [x[0, a] for a in p]
                for c in range(D):
                    s = Fraction(bias[c])
                    for i in range(K):
                        s += Fraction(w[c, i]) * Fraction(rows[len(rows) - K + i][c])
                    assert Fraction(y[0, j, c]) == s
                path = np.full((1, n), -1, np.int32)
                path[0, :len(p)] = p
                C1, st = oracle.conv_commit(C, x, par, path, np.array([len(p)], np.int32))
                assert st[0] == 0
                for i in range(K - 1):
                    np.testing.assert_array_equal(C1[0, i], rows[len(rows) - (K - 1) + i])
