"""Randomised cases through the C ABI: per case a random layer family
(GDN, DeltaNet, scalar decay, GLA), activation dtype, route (automatic,
parallel, serial, hybrid), batch, heads, d_k in {64, 128, 256}, d_v any
multiple of 16 up to 320, node counts across the 16/32/64-row blocks for
the draft and the pending round, and topology (random trees, forests,
chains given as chains, stars, or a mix per batch).  Two fused rounds must
equal verify + standalone commit + verify bit for bit; the committed state
and the second round's outputs are checked against the fp64 oracle on up to
four units.  A draft beyond a route's on-chip stage must be refused before
any launch (SLA_ERR_UNSUPPORTED).  Seeds are fixed and every case prints
its parameters before it runs."""
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


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None


def _parents(r, Bn, n, kind):
    rows = []
    for b in range(Bn):
        k = kind if kind != "mix" else ["tree", "forest", "chain", "star"][b % 4]
        if k == "chain":
            rows.append(inputs.chain(n))
        elif k == "star":
            rows.append(np.array([-1] + [0] * (n - 1), np.int32))
        elif k == "forest":
            rows.append(np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32))
        else:
            rows.append(inputs.random_tree(r, n, max(2, n), int(r.integers(1, 5))))
    return np.stack(rows).astype(np.int32)


def _case(i, seed):
    r = np.random.default_rng(seed)
    fam = str(r.choice(["gdn", "gdn", "deltanet", "decay", "gla"]))
    dt = inputs.BF16 if r.random() < 0.6 else inputs.F32
    route = str(r.choice(["auto", "auto", "parallel", "serial", "hybrid"]))
    dk = int(r.choice([64, 128, 256]))
    dv = int(16 * r.integers(1, 21))
    n0 = int(r.choice([1, 2, 3, 7, 16, 17, 31, 32, 33, 48, 63, 64]))
    n1 = int(r.choice([1, 2, 5, 15, 16, 31, 33, 47, 64]))
    Bn, H = int(r.integers(1, 6)), int(r.integers(1, 4))
    kind = str(r.choice(["tree", "forest", "chain", "mix"]))
    say("random case %d: %s %s route=%s B=%d H=%d dk=%d dv=%d n0=%d n1=%d %s"
        % (i, fam, dt, route, Bn, H, dk, dv, n0, n1, kind))
    chain = kind == "chain"
    cfgs = [inputs.Config("rc%d" % k, 900 + (seed % 50) * 2 + k, Bn, H, dk, dv, n, chain, n, 64, dt, 1)
            for k, n in ((0, n0), (1, n1))]
    rnds, gates = [], []
    for k, c in enumerate(cfgs):
        rd = inputs.draw_round(c, 0, layers=[0])
        rd.parent = _parents(r, Bn, c.n_nodes, kind)
        rnds.append(rd)
        gates.append(inputs.family_gates(c, rd, 0, fam, layer=0, round_index=k))
    path = np.full((Bn, n0), -1, np.int32)
    ln = np.zeros(Bn, np.int32)
    for b in range(Bn):
        if r.random() < 0.85:
            p = inputs.walk_to_root(rnds[0].parent[b], int(r.integers(0, n0)))
            path[b, :len(p)] = p
            ln[b] = len(p)
    S0 = inputs.draw_state(cfgs[0], 0)
    tdt = torch.bfloat16 if dt == inputs.BF16 else torch.float32

    def verify(state, k, f, out, pend=None, st=None):
        rd = rnds[k]
        a, b = gates[k]
        B.sla_verify(state, act_tensor(rd.q[0], dt), act_tensor(rd.k[0], dt), act_tensor(rd.v[0], dt), _dev(a),
                     _dev(b), _dev(rd.parent), out, f, pending=pend, status=st,
                     topology="chain" if chain else "tree", route=route, family=fam)

    def fac(k):
        return B.Factors.empty(Bn, cfgs[k].n_nodes, H, dk, dv, tdt, family=fam)

    def outs(k):
        return torch.empty(Bn, cfgs[k].n_nodes, H, dv, device="cuda")

    try:
        fused, f0, f1, o1 = _dev(S0), fac(0), fac(1), outs(1)
        verify(fused, 0, f0, outs(0))
        st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
        verify(fused, 1, f1, o1, pend=(f0, _dev(path), _dev(ln)), st=st)
        sep, g0, g1, p1 = _dev(S0), fac(0), fac(1), outs(1)
        verify(sep, 0, g0, outs(0))
        B.sla_commit(sep, g0, _dev(path), _dev(ln), family=fam)
        verify(sep, 1, g1, p1)
        torch.cuda.synchronize()
    except B.SlaError as e:
        # refused before any launch: beyond the route's on-chip stage, which
        # only happens at d_k = 256 (GLA on every route; fp32 on the parallel one)
        assert e.code == B.SLA_ERR_UNSUPPORTED and dk == 256 and (fam == "gla" or dt == inputs.F32)
        assert max(n0, n1) > 32
        say("  refused before launch")
        return
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep)
    assert torch.equal(o1, p1)
    units = [(b, h) for b in range(Bn) for h in range(H)]
    units = [units[j] for j in sorted(r.choice(len(units), min(4, len(units)), replace=False))]
    worst = 0.0
    for b, h in units:
        def sl(x):
            return None if x is None else x[b:b + 1, :, h:h + 1]
        (a0, b0), (a1, b1) = gates
        S1, s1 = oracle.commit(S0[b:b + 1, h:h + 1], sl(rnds[0].k32[0]), sl(rnds[0].v32[0]), sl(a0), sl(b0),
                               rnds[0].parent[b:b + 1], path[b:b + 1], ln[b:b + 1], family=fam)
        ref, s2 = oracle.verify(S1, sl(rnds[1].q32[0]), sl(rnds[1].k32[0]), sl(rnds[1].v32[0]), sl(a1), sl(b1),
                                rnds[1].parent[b:b + 1], family=fam)
        assert s1[0] == 0 and s2[0] == 0
        worst = max(worst, rel_err(fused[b, h].cpu().numpy(), S1[0, 0]),
                    rel_err(o1[b, :, h].cpu().numpy(), ref[0, :, 0]))
    say("  worst normwise error %.2e (bar %.0e)" % (worst, TOL[dt]))
    assert worst <= TOL[dt]


CHUNK = 40


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("chunk", range(10))
def test_random_cases(chunk):
    for i in range(chunk * CHUNK, (chunk + 1) * CHUNK):
        _case(i, 20000 + i)
