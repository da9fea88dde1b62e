"""GPU parity of the 1-node (decode-step) kernel that the automatic route
takes for drafts of one node, through the C ABI, against the fp64 oracle and
against the two general routes.

Cases: every layer family, bf16 and fp32 activations, d_k 64/128/256, d_v
ragged against the 64-column slabs, and pending paths of several rounds of
accepted decode steps: a previous draft of up to 12 chained nodes, so the
path can run past the 8 records staged in LDS.  Each case runs a fused round
(pending path applied in front) against a standalone commit followed by a
plain verification (states, outputs and records bitwise equal), checks the
committed state and the outputs against the oracle, and the outputs against
the serial route.  Bars: 1e-5 (fp32 activations) or 2e-3 (bf16).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import TOL, act_tensor, rel_err

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None


class Round:
    def __init__(self, cfg, fam, r):
        self.rnd = inputs.draw_round(cfg, r, layers=[0])
        self.alpha, self.beta = inputs.family_gates(cfg, self.rnd, 0, fam, layer=0, round_index=r)
        self.q, self.k, self.v = (act_tensor(x[0], cfg.dtype) for x in (self.rnd.q, self.rnd.k, self.rnd.v))
        self.a, self.b = _dev(self.alpha), _dev(self.beta)
        self.parent = _dev(self.rnd.parent)


def _factors(cfg, fam):
    dt = torch.bfloat16 if cfg.dtype == inputs.BF16 else torch.float32
    return B.Factors.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v, dt, family=fam)


def _verify(cfg, fam, rd, state, out, f, route="auto", pending=None, status=None):
    B.sla_verify(state, rd.q, rd.k, rd.v, rd.a, rd.b, rd.parent, out, f, pending=pending, status=status,
                 topology="chain", route=route, family=fam)


CASES = [(fam, dt, dk, dv)
         for fam in ["gdn", "deltanet", "decay", "gla"]
         for dt, dk, dv in [(inputs.BF16, 128, 256), (inputs.BF16, 64, 80), (inputs.F32, 256, 48),
                            (inputs.BF16, 256, 16), (inputs.F32, 64, 320)]]


@pytest.mark.parametrize("fam,dt,dk,dv", CASES, ids=["%s-%s-dk%d-dv%d" % c for c in CASES])
def test_one_node_fused_round(fam, dt, dk, dv):
    Bn, H, npend = 6, 3, 12
    say("decode %s %s dk=%d dv=%d" % (fam, dt, dk, dv))
    c_prev = inputs.Config("dp", 800 + dk + dv, Bn, H, dk, dv, npend, True, npend, 1, dt, 1)
    c_node = inputs.Config("dn", 900 + dk + dv, Bn, H, dk, dv, 1, True, 1, 1, dt, 1)
    prev, cur = Round(c_prev, fam, 0), Round(c_node, fam, 1)
    # accepted lengths 0..12 across sequences: past the 8 staged records too
    plen = np.array([12, 0, 3, 9, 1, 8], np.int32)
    ppath = np.full((Bn, npend), -1, np.int32)
    for b_ in range(Bn):
        ppath[b_, :plen[b_]] = np.arange(plen[b_])
    prev.rnd.path, prev.rnd.length = ppath, plen
    S0 = inputs.draw_state(c_prev, 0)
    # the previous round's records come from the general route (a 12-node chain)
    f_prev = _factors(c_prev, fam)
    tmp = torch.from_numpy(S0).cuda()
    _verify(c_prev, fam, prev, tmp, torch.empty(Bn, npend, H, dv, device="cuda"), f_prev)
    path, length = _dev(ppath), _dev(plen)

    fused = torch.from_numpy(S0).cuda()
    out_f, f_f = torch.empty(Bn, 1, H, dv, device="cuda"), _factors(c_node, fam)
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    _verify(c_node, fam, cur, fused, out_f, f_f, pending=(f_prev, path, length), status=st)
    sep = torch.from_numpy(S0).cuda()
    B.sla_commit(sep, f_prev, path, length, family=fam)
    out_s, f_s = torch.empty(Bn, 1, H, dv, device="cuda"), _factors(c_node, fam)
    _verify(c_node, fam, cur, sep, out_s, f_s)
    ser = sep.clone()
    out_r = torch.empty(Bn, 1, H, dv, device="cuda")
    _verify(c_node, fam, cur, ser, out_r, _factors(c_node, fam), route="serial")
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep) and torch.equal(out_f, out_s)
    assert torch.equal(f_f.u, f_s.u) and torch.equal(f_f.k, f_s.k) and torch.equal(f_f.alpha, f_s.alpha)
    # records of the node: the key and gate as given, the parent -1
    assert torch.equal(f_f.k, cur.k)
    gate = np.ones((Bn, 1, H), np.float32) if fam == "deltanet" else cur.alpha
    np.testing.assert_array_equal(f_f.alpha.cpu().numpy(), gate)
    assert (f_f.parent.cpu().numpy() == -1).all()

    tol = TOL[dt]
    refS, sst = oracle.commit(S0, prev.rnd.k32[0], prev.rnd.v32[0], prev.alpha, prev.beta, prev.rnd.parent,
                              ppath, plen, family=fam)
    assert (sst == 0).all()
    es = rel_err(fused.cpu().numpy(), refS)
    ref, ost = oracle.verify(refS, cur.rnd.q32[0], cur.rnd.k32[0], cur.rnd.v32[0], cur.alpha, cur.beta,
                             cur.rnd.parent, family=fam)
    assert (ost == 0).all()
    eo = rel_err(out_f.cpu().numpy(), ref)
    er = rel_err(out_f.cpu().numpy(), out_r.cpu().numpy())
    say("  state err %.2e output err %.2e vs serial %.2e" % (es, eo, er))
    assert es <= tol and eo <= tol and er <= tol


def test_one_node_refuses_bad_parent_and_path():
    """A node that is not a child of the committed state, or a pending path
    that is not a root path, is reported per sequence and leaves its state
    untouched; the other sequences proceed."""
    fam, dt, dk, dv = "gdn", inputs.BF16, 128, 64
    Bn, H, npend = 3, 2, 4
    c_prev = inputs.Config("rp", 950, Bn, H, dk, dv, npend, True, npend, 1, dt, 1)
    c_node = inputs.Config("rn", 951, Bn, H, dk, dv, 1, True, 1, 1, dt, 1)
    prev, cur = Round(c_prev, fam, 0), Round(c_node, fam, 1)
    S0 = inputs.draw_state(c_prev, 0)
    f_prev = _factors(c_prev, fam)
    _verify(c_prev, fam, prev, torch.from_numpy(S0).cuda(), torch.empty(Bn, npend, H, dv, device="cuda"), f_prev)
    ppath = np.array([[0, 1, -1, -1], [1, -1, -1, -1], [0, 1, 2, 3]], np.int32)  # row 1: not a root path
    plen = np.array([2, 1, 4], np.int32)
    par = cur.rnd.parent.copy()
    par[2, 0] = 0  # row 2: the node names itself as parent
    cur.parent = _dev(par)
    state = torch.from_numpy(S0).cuda()
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    _verify(c_node, fam, cur, state, torch.empty(Bn, 1, H, dv, device="cuda"), _factors(c_node, fam),
            pending=(f_prev, _dev(ppath), _dev(plen)), status=st)
    torch.cuda.synchronize()
    assert list(st.cpu().numpy()) == [0, B.SLA_ERR_PATH, B.SLA_ERR_TOPOLOGY]
    got = state.cpu().numpy()
    np.testing.assert_array_equal(got[1], S0[1])
    np.testing.assert_array_equal(got[2], S0[2])
    assert not np.array_equal(got[0], S0[0])
