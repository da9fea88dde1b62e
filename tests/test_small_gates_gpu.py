"""GPU parity at the near-reset edge of the gated state: strong-forgetting
gates (alpha, or GLA's per-key gates, ~ U(1e-3, 0.3) with some at 1e-6 and
1e-20), whose products along a root path leave the fp32 range within a few
nodes (the decay of §2.2's gated state and the tree-masked factorisation of
§4.2, whose decay ratios are products of the gates strictly between two
nodes of a root path).

Per case, two rounds through the C ABI: round 0 verified from the committed
state; round 1 with round 0's accepted path pending (fused commit-and-
verify).  Every output and committed state must be finite; sampled (b, h)
units are compared with the fp64 oracle (bar 2e-3 normwise with bf16
q/k/v, 1e-5 with fp32);
the serial and parallel routes are compared over every unit.  The shapes:
64-deep chains, the 64-node depth-8 trees at batch 256 (d_v 256), the
paper's target shape (8 heads, d_k = d_v = 256) as a chain of 4 and a
32-node tree, the 16-node trees at batch 64, and with fp32 q/k/v a 32-deep
chain and a 48-node tree."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import TOL, act_tensor, rel_err, sample_units

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


CHAIN64 = inputs.Config("chain64_strong", 60, 4, 4, 128, 128, 64, True, 64, 1, inputs.BF16, 1,
                        "batch 4, 4 heads, dk=dv=128, 64-deep chain")
PAPER_TREE32 = inputs.Config("paper_tree32_strong", 61, 1, 8, 256, 256, 32, False, 6, 4, inputs.BF16, 1,
                             "batch 1, 8 heads, dk=dv=256, 32-node tree (depth<=6, branch<=4)")
# fp32 activations (the fp32 matrix-core contraction on the parallel route)
CHAIN32_F32 = inputs.Config("chain32_strong_f32", 62, 4, 4, 128, 128, 32, True, 32, 1, inputs.F32, 1,
                            "batch 4, 4 heads, dk=dv=128, 32-deep chain, fp32 q/k/v")
TREE48_F32 = inputs.Config("tree48_strong_f32", 63, 8, 4, 128, 192, 48, False, 8, 4, inputs.F32, 1,
                           "batch 8, 4 heads, dk=128, dv=192, 48-node tree (depth<=8), fp32 q/k/v")
CFGS = {c.name: c for c in [CHAIN64, PAPER_TREE32, CHAIN32_F32, TREE48_F32]}


def _cfg(name):
    return CFGS[name] if name in CFGS else inputs.config(name)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None


class Draft:
    def __init__(self, cfg, fam, round_index):
        self.rnd = inputs.draw_round(cfg, round_index, layers=[0])
        self.alpha = inputs.draw_strong_gates(cfg, 0, round_index, family=fam)
        self.beta = self.rnd.beta[0] if fam == "gdn" else None
        self.q = act_tensor(self.rnd.q[0], cfg.dtype)
        self.k = act_tensor(self.rnd.k[0], cfg.dtype)
        self.v = act_tensor(self.rnd.v[0], cfg.dtype)
        self.a, self.b = _dev(self.alpha), _dev(self.beta)
        self.parent, self.path, self.length = _dev(self.rnd.parent), _dev(self.rnd.path), _dev(self.rnd.length)

    def unit(self, b, h):
        r = self.rnd
        a = self.alpha[b:b + 1, :, h:h + 1]
        bt = None if self.beta is None else self.beta[b:b + 1, :, h:h + 1]
        return r.q32[0][b:b + 1, :, h:h + 1], r.k32[0][b:b + 1, :, h:h + 1], r.v32[0][b:b + 1, :, h:h + 1], a, bt


def _run(cfg, fam, route, S0, d0, d1):
    """Two rounds; returns (committed state, round-1 outputs) on the host."""
    dt = torch.bfloat16 if cfg.dtype == inputs.BF16 else torch.float32
    Bn, n, H = cfg.batch, cfg.n_nodes, cfg.heads
    f0 = B.Factors.empty(Bn, n, H, cfg.d_k, cfg.d_v, dt, family=fam)
    f1 = B.Factors.empty(Bn, n, H, cfg.d_k, cfg.d_v, dt, family=fam)
    out0 = torch.empty(Bn, n, H, cfg.d_v, device="cuda")
    out1 = torch.empty(Bn, n, H, cfg.d_v, device="cuda")
    state = torch.from_numpy(S0).cuda()
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    topo = "chain" if cfg.chain else "tree"
    B.sla_verify(state, d0.q, d0.k, d0.v, d0.a, d0.b, d0.parent, out0, f0, topology=topo, route=route,
                 family=fam)
    B.sla_verify(state, d1.q, d1.k, d1.v, d1.a, d1.b, d1.parent, out1, f1, pending=(f0, d0.path, d0.length),
                 status=st, topology=topo, route=route, family=fam)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    return state.cpu().numpy(), out0.cpu().numpy(), out1.cpu().numpy()


CASES = [(name, fam) for name in ["chain64_strong", "large_batch_tree64", "paper_fused_shape",
                                  "paper_tree32_strong", "batched_tree_serving", "chain32_strong_f32",
                                  "tree48_strong_f32"]
         for fam in ["gdn", "decay", "gla"]]


@pytest.mark.parametrize("name,fam", CASES)
def test_strong_gates_both_routes(name, fam):
    cfg = _cfg(name)
    tol = TOL[cfg.dtype]
    d0, d1 = Draft(cfg, fam, 0), Draft(cfg, fam, 1)
    S0 = inputs.draw_state(cfg, 0)
    units = sample_units(cfg, 16 if cfg.n_nodes >= 64 and cfg.batch > 8 else 64, 11)
    # the oracle on the sampled units: round 0 outputs, the committed state,
    # then round 1 outputs from it
    ref_o0, ref_S1, ref_o1 = [], [], []
    for b, h in units:
        q, k, v, a, bt = d0.unit(b, h)
        o, st = oracle.verify(S0[b:b + 1, h:h + 1], q, k, v, a, bt, d0.rnd.parent[b:b + 1], family=fam)
        assert st[0] == 0
        ref_o0.append(o[0, :, 0])
        S1, st = oracle.commit(S0[b:b + 1, h:h + 1], k, v, a, bt, d0.rnd.parent[b:b + 1], d0.rnd.path[b:b + 1],
                               d0.rnd.length[b:b + 1], family=fam)
        assert st[0] == 0
        ref_S1.append(S1[0, 0])
        q, k, v, a, bt = d1.unit(b, h)
        o, st = oracle.verify(S1, q, k, v, a, bt, d1.rnd.parent[b:b + 1], family=fam)
        assert st[0] == 0
        ref_o1.append(o[0, :, 0])
    got = {}
    for route in ["serial", "parallel"]:
        if route == "parallel" and fam == "gla" and cfg.d_k == 256 and cfg.n_nodes > 32:
            continue
        say("strong gates %s %s route=%s" % (name, fam, route))
        S1, o0, o1 = _run(cfg, fam, route, S0, d0, d1)
        assert np.isfinite(S1).all() and np.isfinite(o0).all() and np.isfinite(o1).all()
        es = rel_err(np.stack([S1[b, h] for b, h in units]), np.stack(ref_S1))
        e0 = rel_err(np.stack([o0[b, :, h] for b, h in units]), np.stack(ref_o0))
        e1 = rel_err(np.stack([o1[b, :, h] for b, h in units]), np.stack(ref_o1))
        say("  state %.3e  out0 %.3e  out1 %.3e" % (es, e0, e1))
        assert max(es, e0, e1) <= tol
        got[route] = (S1, o0, o1)
    if len(got) == 2:
        for x, y in zip(got["serial"], got["parallel"]):
            assert rel_err(y, x) <= tol
