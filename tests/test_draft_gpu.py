"""GPU: batched draft pruning/packing and the tree-mask converter (sla_prune,
sla_tree_mask_to_parent) against the oracle, bit for bit, through the C ABI.
Every decision is integer or an fp32 comparison taken in the same precision
on both sides, so the bar is exact equality."""
import numpy as np
import pytest
import torch

from oracle import prune as P
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def forest(r, n):
    return np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32)


@pytest.mark.parametrize("n", [1, 7, 16, 33, 64])
@pytest.mark.parametrize("tau,T", [(0.0, 0), (1.5, 0), (1e9, 0), (3.0, 5), (1e9, 12), (0.7, 1)])
def test_prune_matches_oracle(n, tau, T):
    r = np.random.default_rng(1000 + n)
    Bn = 96
    par = np.stack([inputs.random_tree(r, n, 12, 4) if b % 3 else forest(r, n) for b in range(Bn)])
    lp = np.log(r.uniform(0.01, 1.0, (Bn, n))).astype(np.float32)
    lp[::5, ::3] = 0.0  # ties along paths
    bad_rows = []
    if n > 2:
        par[7, n - 1] = n - 1  # not topological
        lp[11, 1] = 0.25       # a positive log-probability
        lp[12, 0] = np.nan
        bad_rows = [7, 11, 12]
    say("prune n=%d tau=%g T=%d" % (n, tau, T))
    out = B.sla_prune(torch.from_numpy(par).cuda(), torch.from_numpy(lp).cuda(), tau, T, with_scores=True)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    for b in range(Bn):
        keep, q, st = P.prune(par[b], lp[b], tau, T)
        if st != P.OK:
            assert b in bad_rows
            want = {P.ERR_TOPOLOGY: B.SLA_ERR_TOPOLOGY, P.ERR_SCORE: B.SLA_ERR_SCORE}[st]
            assert got["status"][b] == want and got["count"][b] == 0
            continue
        packed, idx = P.pack(par[b], keep)
        m = len(keep)
        assert got["status"][b] == 0 and got["count"][b] == m, b
        np.testing.assert_array_equal(got["packed_parent"][b, :m], packed)
        np.testing.assert_array_equal(got["index_map"][b, :m], idx)
        assert (got["packed_parent"][b, m:] == -1).all() and (got["index_map"][b, m:] == -1).all()
        np.testing.assert_array_equal(got["scores"][b], q)


def test_tree_mask_converter_matches_oracle():
    r = np.random.default_rng(2000)
    for n in [1, 5, 32, 64]:
        Bn = 64
        pars = [inputs.random_tree(r, n, 16, 5) if b % 2 else forest(r, n) for b in range(Bn)]
        rows = np.zeros((Bn, n), np.uint64)
        for b, par in enumerate(pars):
            for i in range(n):
                for a in inputs.walk_to_root(par, i):
                    rows[b, i] |= np.uint64(1) << np.uint64(a)
        if n > 1:
            rows[3, n - 1] ^= np.uint64(1) << np.uint64(0 if n - 1 else 0)  # flip a bit
            rows[5, 0] |= np.uint64(1) << np.uint64(n - 1)                   # ancestor after descendant
        say("mask converter n=%d" % n)
        par_d, st_d = B.sla_tree_mask_to_parent(torch.from_numpy(rows.view(np.int64)).cuda())
        torch.cuda.synchronize()
        par_g, st_g = par_d.cpu().numpy(), st_d.cpu().numpy()
        for b in range(Bn):
            m = np.array([[(int(rows[b, i]) >> j) & 1 for j in range(n)] for i in range(n)], bool)
            ref, ost = P.mask_to_parent(m)
            assert (st_g[b] == 0) == (ost == P.OK), b
            if ost == P.OK:
                np.testing.assert_array_equal(par_g[b], ref)
