"""Draft pruning, packing and the tree-mask converter of the library (host
versions, on the CPU) against the oracle, bit for bit, plus argument errors.
The device versions are checked in tests/test_draft_gpu.py."""
import itertools

import numpy as np
import pytest

from oracle import prune as P
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs


def rng(seed):
    return np.random.default_rng(seed)


def forest(r, n):
    return np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32)


def oracle_rows(par, lp, tau, T):
    keep, q, st = P.prune(par, lp, tau, T)
    if st != P.OK:
        return st, None
    packed, idx = P.pack(par, keep)
    return st, (keep, q, packed, idx)


def check_host(par, lp, tau, T):
    st, ref = oracle_rows(par, lp, tau, T)
    got = B.sla_prune_host(par, lp, tau, T)
    if st != P.OK:
        assert got["status"] == {P.ERR_TOPOLOGY: B.SLA_ERR_TOPOLOGY, P.ERR_SCORE: B.SLA_ERR_SCORE}[st]
        return
    keep, q, packed, idx = ref
    m = len(keep)
    assert got["status"] == 0 and got["count"] == m
    np.testing.assert_array_equal(got["packed_parent"][:m], packed)
    np.testing.assert_array_equal(got["index_map"][:m], idx)
    assert (got["packed_parent"][m:] == -1).all() and (got["index_map"][m:] == -1).all()
    np.testing.assert_array_equal(got["scores"], q)


def test_host_prune_matches_oracle_random():
    r = rng(1)
    for _ in range(300):
        n = int(r.integers(1, 65))
        par = inputs.random_tree(r, n, 12, 4) if r.random() < 0.7 else forest(r, n)
        lp = np.log(r.uniform(0.01, 1.0, n)).astype(np.float32)
        if r.random() < 0.3:
            lp[r.integers(0, n, 4)] = 0.0
        tau = float(r.choice([0.0, r.uniform(0, 1), r.uniform(1, 8), 1e9]))
        T = int(r.choice([0, 1, int(r.integers(1, n + 1)), n]))
        check_host(par, lp, tau, T)


def test_host_prune_brute_force_small():
    r = rng(2)
    for n in range(1, 6):
        for par in itertools.product(*[range(-1, j) for j in range(n)]):
            par = np.array(par, np.int32)
            lp = -r.integers(0, 4, n).astype(np.float32) / 2
            for tau in [0.0, 0.5, 2.0]:
                for T in range(0, n + 1):
                    check_host(par, lp, tau, T)


def test_host_prune_large_candidate_sets_and_errors():
    r = rng(3)
    n = 300  # beyond one wavefront: the host version takes any n
    par = inputs.random_tree(r, n, 30, 4)
    lp = np.log(r.uniform(0.05, 1.0, n)).astype(np.float32)
    check_host(par, lp, 3.0, 0)
    check_host(par, lp, 3.0, 40)
    check_host(np.array([-1, 0, 0]), np.array([-0.1, 0.2, -0.3], np.float32), 1.0, 0)
    check_host(np.array([-1, 0, 0]), np.array([-0.1, np.nan, -0.3], np.float32), 1.0, 0)
    check_host(np.array([-1, 2, 0]), np.array([-0.1, -0.2, -0.3], np.float32), 1.0, 0)
    assert B.sla_prune_host([-1, 0], [-0.1, -0.1], -1.0)["status"] == B.SLA_ERR_SHAPE
    assert B.sla_prune_host([-1, 0], [-0.1, -0.1], float("nan"))["status"] == B.SLA_ERR_SHAPE


def mask_rows(par):
    n = len(par)
    rows = np.zeros(n, np.uint64)
    for i in range(n):
        for a in inputs.walk_to_root(par, i):
            rows[i] |= np.uint64(1) << np.uint64(a)
    return rows


def rows_to_bool(rows, n):
    return np.array([[(int(rows[i]) >> j) & 1 for j in range(n)] for i in range(n)], bool)


def test_host_tree_mask_converter_matches_oracle():
    r = rng(4)
    for _ in range(200):
        n = int(r.integers(1, 65))
        par = inputs.random_tree(r, n, 16, 5) if r.random() < 0.6 else forest(r, n)
        rows = mask_rows(par)
        st, got = B.sla_tree_mask_to_parent_host(rows)
        ref, ost = P.mask_to_parent(rows_to_bool(rows, n))
        assert st == 0 and ost == P.OK
        np.testing.assert_array_equal(got, ref)
        np.testing.assert_array_equal(got, par)
        # corrupt one bit: the oracle and the library agree on rejecting it
        if n > 1:
            bad = rows.copy()
            i, j = int(r.integers(0, n)), int(r.integers(0, n))
            bad[i] ^= np.uint64(1) << np.uint64(j)
            st2, got2 = B.sla_tree_mask_to_parent_host(bad)
            ref2, ost2 = P.mask_to_parent(rows_to_bool(bad, n))
            assert (st2 == 0) == (ost2 == P.OK)
            if st2 == 0:
                np.testing.assert_array_equal(got2, ref2)


def test_draft_argument_errors():
    L = B.lib()
    import ctypes
    fake = ctypes.c_void_p(1 << 20)
    assert L.sla_prune(None, fake, 1, 4, 1.0, 0, fake, fake, fake, None, None, None) == B.SLA_ERR_NULL
    assert L.sla_prune(fake, fake, 1, 65, 1.0, 0, fake, fake, fake, None, None, None) == B.SLA_ERR_SHAPE
    assert L.sla_prune(fake, fake, 0, 4, 1.0, 0, fake, fake, fake, None, None, None) == B.SLA_ERR_SHAPE
    assert L.sla_prune(fake, fake, 1, 4, -1.0, 0, fake, fake, fake, None, None, None) == B.SLA_ERR_SHAPE
    assert L.sla_tree_mask_to_parent(None, 1, 4, fake, None, None) == B.SLA_ERR_NULL
    assert L.sla_tree_mask_to_parent(fake, 1, 65, fake, None, None) == B.SLA_ERR_SHAPE
