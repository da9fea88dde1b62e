"""Pins of the oracle's draft pruning, packing and tree-mask converter
(§6.1 tree pruning, §7 proposal converter).

Each pin is a closed form (a chain keeps the prefix inside the margin; under a
budget the kept set is the score-ranked prefix), a defining property
(ancestor closure, the window threshold, the budget, maximality), an
independent computation (matrix reachability for the tree mask, numpy's
lexsort for the ranking), or brute force over every parent array of a few
nodes; none re-types the oracle's loops.
"""
import itertools

import numpy as np
import pytest

from oracle import prune as P
from paper_2607_16673_amd import inputs


def rng(seed):
    return np.random.default_rng(seed)


def forest(r, n):
    return np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32)


def reach_mask(parent):
    """Ancestor-or-self matrix by boolean matrix powers of the parent relation."""
    n = len(parent)
    A = np.zeros((n, n), bool)
    for j, p in enumerate(parent):
        if p >= 0:
            A[j, p] = True
    R = np.eye(n, dtype=bool)
    step = np.eye(n, dtype=bool)
    for _ in range(n):
        step = (step.astype(np.int64) @ A.astype(np.int64)) > 0
        R |= step
    return R


def ancestor_closed(parent, keep):
    ks = set(keep)
    return all(int(parent[v]) == -1 or int(parent[v]) in ks for v in keep)


def rollout_logp(r, n):
    """Log-probabilities of a draft rollout: log of softmax-like probabilities."""
    return np.log(r.uniform(0.02, 1.0, n)).astype(np.float32)


def test_scores_are_path_sums_in_fp32():
    """q(v) = sum of logp over P(v), root first, rounded in fp32 at every add;
    against numpy's fp32 cumulative sum along each explicit root path."""
    r = rng(1)
    for _ in range(20):
        n = int(r.integers(1, 40))
        par = inputs.random_tree(r, n, 8, 4) if r.random() < 0.7 else forest(r, n)
        lp = rollout_logp(r, n)
        q, st = P.scores(par, lp)
        assert st == P.OK
        for v in range(n):
            path = inputs.walk_to_root(par, v)
            assert q[v] == np.cumsum(lp[path], dtype=np.float32)[-1]


def test_chain_keeps_the_prefix_inside_the_margin():
    r = rng(2)
    for _ in range(30):
        n = int(r.integers(1, 30))
        lp = rollout_logp(r, n)
        tau = float(r.uniform(0, 4))
        keep, q, st = P.prune(inputs.chain(n), lp, tau, 0)
        c = np.cumsum(lp, dtype=np.float32)
        thr = np.float32(c[0] - np.float32(tau))
        assert keep == list(range(int(np.count_nonzero(c >= thr))))


def test_window_threshold_and_ancestor_closure_without_budget():
    r = rng(3)
    for _ in range(60):
        n = int(r.integers(1, 64))
        par = inputs.random_tree(r, n, 10, 4) if r.random() < 0.7 else forest(r, n)
        lp = rollout_logp(r, n)
        tau = float(r.uniform(0, 5))
        keep, q, st = P.prune(par, lp, tau, 0)
        thr = np.float32(np.max(q) - np.float32(tau))
        assert keep == [v for v in range(n) if q[v] >= thr]
        assert ancestor_closed(par, keep)  # monotone scores: closed by construction
        assert int(np.argmax(q)) in keep


def test_budget_keeps_the_score_ranked_prefix():
    """Under a budget the kept set is the first T of the window in (score desc,
    index asc) order, which is ancestor-closed; it is maximal and within T."""
    r = rng(4)
    for _ in range(80):
        n = int(r.integers(2, 64))
        par = inputs.random_tree(r, n, 10, 4) if r.random() < 0.7 else forest(r, n)
        lp = rollout_logp(r, n)
        if r.random() < 0.3:
            lp[r.integers(0, n, 3)] = 0.0  # ties along paths
        tau = float(r.uniform(0, 6))
        T = int(r.integers(1, n + 1))
        keep, q, st = P.prune(par, lp, tau, T)
        thr = np.float32(np.max(q) - np.float32(tau))
        window = np.array([v for v in range(n) if q[v] >= thr])
        order = window[np.lexsort((window, -q[window].astype(np.float64)))]
        assert keep == sorted(order[:T].tolist())
        assert len(keep) == min(T, len(window))
        assert ancestor_closed(par, keep)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_brute_force_every_small_parent_array(n):
    """Every parent array of n nodes, every budget: the kept set is the largest
    ancestor-closed subset of the window reachable by taking candidates in
    score order (checked against the explicit ranking), and packing maps every
    kept node's packed root path back to its original root path."""
    r = rng(10 + n)
    for par in itertools.product(*[range(-1, j) for j in range(n)]):
        par = np.array(par, np.int32)
        lp = -r.integers(0, 4, n).astype(np.float32) / 2  # dyadic, with ties
        for tau in [0.0, 0.5, 1.0, 10.0]:
            for T in range(0, n + 1):
                keep, q, st = P.prune(par, lp, tau, T)
                assert st == P.OK
                assert ancestor_closed(par, keep)
                if T:
                    assert len(keep) <= T
                if keep:
                    assert int(np.argmax(q)) in keep  # the best path always survives
                if tau == 0.0 and T == 0:
                    assert keep == [v for v in range(n) if q[v] == np.max(q)]
                packed, idx = P.pack(par, keep)
                assert list(idx) == keep
                assert all(-1 <= int(packed[i]) < i for i in range(len(packed)))  # topological
                for i, old in enumerate(keep):
                    pp = [int(idx[a]) for a in inputs.walk_to_root(packed, i)]
                    assert pp == inputs.walk_to_root(par, old)


def test_window_decision_is_taken_in_fp32():
    """q* - tau is rounded to fp32 before the comparison (the library's
    precision): with q* = -1 and tau = 1e-7 the fp32 threshold is the next fp32
    value below -1, so a node scoring exactly that is kept (it would not be
    against the exact threshold -1.0000001)."""
    below = np.nextafter(np.float32(-1.0), np.float32(-2.0))
    lp = np.array([-1.0, below - np.float32(-1.0)], np.float32)
    keep, q, st = P.prune(inputs.chain(2), lp, 1e-7, 0)
    assert q[1] == below and keep == [0, 1]
    assert float(q[1]) < -1.0 - 1e-7


def test_rejects_positive_or_nan_logprob_and_bad_topology():
    assert P.scores([-1, 0], [-0.5, 0.25])[1] == P.ERR_SCORE
    assert P.scores([-1, 0], [-0.5, float("nan")])[1] == P.ERR_SCORE
    assert P.scores([-1, 1], [-0.5, -0.5])[1] == P.ERR_TOPOLOGY
    assert P.prune([-1, 0], [0.1, -1.0], 1.0, 0)[2] == P.ERR_SCORE


def test_tree_mask_round_trip_against_reachability():
    r = rng(5)
    for _ in range(60):
        n = int(r.integers(1, 65))
        par = inputs.random_tree(r, n, 12, 5) if r.random() < 0.6 else forest(r, n)
        p2, st = P.mask_to_parent(reach_mask(par))
        assert st == P.OK
        np.testing.assert_array_equal(p2, par)


def test_tree_mask_rejects_non_tree_masks():
    good = reach_mask(np.array([-1, 0, 1, 0, 3], np.int32))
    bad = []
    m = good.copy(); m[2, 2] = False; bad.append(m)          # missing diagonal
    m = good.copy(); m[4, 1] = True; bad.append(m)           # two branches' ancestors
    m = good.copy(); m[2, 0] = False; bad.append(m)          # not closed under ancestry
    m = good.copy(); m[1, 3] = True; bad.append(m)           # ancestor after descendant
    for m in bad:
        assert P.mask_to_parent(m)[1] == P.ERR_TOPOLOGY
