"""GPU parity of the tree-verification study's routes with the fp64 oracle:
root-to-leaf replay (one chain verification per root-to-leaf path), the
serial, parallel and hybrid routes, on synthetic proposal trees (top-k
rollouts of the configured depth pruned to the node budget) at every
(top-k, depth, nodes) group of the paper's tree-shape table and its target
shape (batch 1, 8 heads, d_k = d_v = 256, bf16 activations).  Every node's
output of every route is compared with the oracle (bar 2e-3 normwise);
the hybrid route must equal the serial route bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import study

from gpu_util import rel_err

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("k,depth,n", study.TREE_SHAPES)
def test_study_routes_match_oracle(k, depth, n):
    rng = np.random.default_rng(1000 * k + depth)
    dev = torch.device("cuda")
    for ti in range(2):
        par = study.proposal_tree(rng, k, depth, n)
        assert B.sla_topology_host(par)["status"] == 0
        d = study.Draft(torch, dev, par, 8, 256, 256, seed=50 + ti)
        for route in study.ROUTES:
            d.launch(route)
        torch.cuda.synchronize()
        h = d.host
        ref, st = oracle.verify(d.state_np, h["q32"], h["k32"], h["v32"], h["alpha"], h["beta"], par[None])
        assert (st == 0).all()
        ref = ref[0]
        for route in study.ROUTES:
            e = rel_err(d.outputs(route), ref)
            say("study k=%d depth=%d n=%d tree %d (%d paths) %s: rel err %.3e"
                % (k, depth, n, ti, len(d.chains), route, e))
            assert e <= 2e-3
        assert torch.equal(d.out["serial"], d.out["hybrid"])
        assert torch.equal(d.fac["serial"].u, d.fac["hybrid"].u)
