"""GPU checks of the chain-decomposed hybrid route (heavy-light chains, §4.3).

Every node's state is the committed state advanced by the factor records of
its root path, root first, on the serial and the hybrid routes alike; only
the schedule differs (one wave in DFS order against one wave per chain,
level by level).  So the two routes must agree bit for bit -- outputs,
factor records and committed states -- on any topology: a chain given as a
tree, stars, forests of many roots, caterpillars (a spine with a leaf on
every node, so every level holds many one-node chains), complete binary
trees, the deepest and widest 64-node drafts, and random trees.  A schedule
that started a chain before its boundary records existed would read stale
records and break the equality.  Also: the oracle on sampled units, the
device data errors, the factor records, and the automatic route's choices
(fp32 drafts on the parallel route, the hybrid fallback for drafts beyond
the parallel route's on-chip stage)."""
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


def _caterpillar(n):
    p = np.full(n, -1, np.int32)
    spine = list(range(0, n, 2))
    for i, s in enumerate(spine[1:], 1):
        p[s] = spine[i - 1]
    for j in range(1, n, 2):
        p[j] = j - 1
    return p


def _binary(n):
    return np.array([-1] + [(j - 1) // 2 for j in range(1, n)], np.int32)


def _topologies(n, r):
    tops = {
        "chain_as_tree": inputs.chain(n),
        "star": np.array([-1] + [0] * (n - 1), np.int32),
        "all_roots": np.full(n, -1, np.int32),
        "caterpillar": _caterpillar(n),
        "binary": _binary(n),
        "random": inputs.random_tree(r, n, max(2, min(n, 8)), 4),
        "forest": np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32),
    }
    return tops


def _problem(seed, Bn, H, dk, dv, n, parents, dtype, fam):
    cfg = inputs.Config("hy", 700 + seed % 97, Bn, H, dk, dv, n, False, n, 64, dtype, 1)
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    rnd.parent = np.stack(parents).astype(np.int32)
    r = np.random.default_rng(seed)
    rnd.path = np.full((Bn, n), -1, np.int32)
    rnd.length = np.zeros(Bn, np.int32)
    for b in range(Bn):
        p = inputs.walk_to_root(rnd.parent[b], int(r.integers(0, n)))
        rnd.path[b, :len(p)] = p
        rnd.length[b] = len(p)
    alpha, beta = inputs.family_gates(cfg, rnd, 0, fam, layer=0)
    return cfg, rnd, alpha, beta, inputs.draw_state(cfg, 0)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None


def _two_rounds(cfg, rnd0, a0, b0, rnd1, a1, b1, S0, fam, route):
    dt = torch.bfloat16 if cfg.dtype == inputs.BF16 else torch.float32
    Bn, n, H = cfg.batch, cfg.n_nodes, cfg.heads
    res = []
    state = torch.from_numpy(S0).cuda()
    f_prev = None
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    for rnd, a, b in [(rnd0, a0, b0), (rnd1, a1, b1)]:
        f = B.Factors.empty(Bn, n, H, cfg.d_k, cfg.d_v, dt, family=fam)
        out = torch.empty(Bn, n, H, cfg.d_v, device="cuda")
        pend = None if f_prev is None else (f_prev, _dev(rnd0.path), _dev(rnd0.length))
        B.sla_verify(state, act_tensor(rnd.q[0], cfg.dtype), act_tensor(rnd.k[0], cfg.dtype),
                     act_tensor(rnd.v[0], cfg.dtype), _dev(a), _dev(b), _dev(rnd.parent), out, f, pending=pend,
                     status=st, route=route, family=fam)
        res.append((out, f))
        f_prev = f
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    return state, res


CASES = [(dk, dv, n, dt, fam) for dk, dv, n in [(64, 48, 16), (128, 64, 33), (128, 128, 64), (256, 32, 24)]
         for dt in [inputs.BF16, inputs.F32] for fam in ["gdn", "deltanet", "decay", "gla"]]


@pytest.mark.parametrize("dk,dv,n,dt,fam", CASES)
def test_hybrid_bitwise_equals_serial(dk, dv, n, dt, fam):
    r = np.random.default_rng(dk * 1000 + n * 10 + len(fam))
    tops = _topologies(n, r)
    names = list(tops)
    parents0 = [tops[nm] for nm in names]
    parents1 = [tops[names[(i + 3) % len(names)]] for i in range(len(names))]
    Bn, H = len(names), 2
    cfg, r0, a0, b0, S0 = _problem(11 + n, Bn, H, dk, dv, n, parents0, dt, fam)
    _, r1, a1, b1, _ = _problem(12 + n, Bn, H, dk, dv, n, parents1, dt, fam)
    say("hybrid vs serial dk=%d dv=%d n=%d %s %s: %s" % (dk, dv, n, dt, fam, ",".join(names)))
    s_ser, res_ser = _two_rounds(cfg, r0, a0, b0, r1, a1, b1, S0, fam, "serial")
    s_hy, res_hy = _two_rounds(cfg, r0, a0, b0, r1, a1, b1, S0, fam, "hybrid")
    assert torch.equal(s_ser, s_hy)
    for (o_s, f_s), (o_h, f_h) in zip(res_ser, res_hy):
        assert torch.equal(o_s, o_h)
        assert torch.equal(f_s.u, f_h.u) and torch.equal(f_s.k, f_h.k)
        assert torch.equal(f_s.alpha, f_h.alpha) and torch.equal(f_s.parent, f_h.parent)
    # round 0 against the oracle on every unit (small shapes)
    ref, st = oracle.verify(S0, r0.q32[0], r0.k32[0], r0.v32[0], a0, b0, r0.parent, family=fam)
    assert (st == 0).all()
    err = rel_err(res_hy[0][0].cpu().numpy(), ref)
    say("  round 0 output rel err %.3e" % err)
    assert err <= TOL[dt]


def test_hybrid_device_errors_leave_state():
    """A bad parent array or pending path sets status and leaves the state."""
    n, Bn, H, dk, dv = 16, 3, 2, 128, 64
    r = np.random.default_rng(5)
    parents = [inputs.random_tree(r, n, 5, 3) for _ in range(Bn)]
    cfg, r0, a0, b0, S0 = _problem(31, Bn, H, dk, dv, n, parents, inputs.BF16, "gdn")
    bad = r0.parent.copy()
    bad[1, 5] = 9  # a parent after its child
    state = torch.from_numpy(S0).cuda()
    f = B.Factors.empty(Bn, n, H, dk, dv, torch.bfloat16)
    out = torch.empty(Bn, n, H, dv, device="cuda")
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    q, k, v = (act_tensor(x[0], cfg.dtype) for x in (r0.q, r0.k, r0.v))
    B.sla_verify(state, q, k, v, _dev(a0), _dev(b0), _dev(bad), out, f, status=st, route="hybrid")
    torch.cuda.synchronize()
    assert st.cpu().numpy().tolist() == [0, B.SLA_ERR_TOPOLOGY, 0]
    # pending path that is not a root path for sequence 2
    B.sla_verify(state, q, k, v, _dev(a0), _dev(b0), _dev(r0.parent), out, f, status=st, route="hybrid")
    path = r0.path.copy()
    path[2, :] = -1
    path[2, 0] = n - 1 if r0.parent[2, n - 1] != -1 else 1
    length = r0.length.copy()
    length[2] = 1
    f1 = B.Factors.empty(Bn, n, H, dk, dv, torch.bfloat16)
    S_before = state.clone()
    B.sla_verify(state, q, k, v, _dev(a0), _dev(b0), _dev(r0.parent), out, f1, status=st, route="hybrid",
                 pending=(f, _dev(path), _dev(length)))
    torch.cuda.synchronize()
    s = st.cpu().numpy()
    assert s[2] == B.SLA_ERR_PATH and s[0] == 0 and s[1] == 0
    assert torch.equal(state[2], S_before[2])


# The automatic route's choices, bit for bit against the explicit route it
# should take: drafts of two or more nodes go to the parallel route whatever
# their activation dtype; a draft the parallel route cannot stage on chip
# (more than 32 nodes at d_k = 256 with fp32 activations or GLA's gates)
# falls back to the hybrid, which pays for trees of more than 32 nodes.
ROUTING = [
    (128, 64, 16, inputs.F32, "gdn", "parallel"),
    (128, 64, 48, inputs.F32, "decay", "parallel"),
    (64, 80, 9, inputs.BF16, "deltanet", "parallel"),
    (256, 48, 48, inputs.F32, "gdn", "hybrid"),
    (256, 32, 40, inputs.BF16, "gla", "hybrid"),
    (256, 48, 64, inputs.F32, "deltanet", "hybrid"),
]


@pytest.mark.parametrize("dk,dv,n,dt,fam,expect", ROUTING,
                         ids=["dk%d_dv%d_n%d_%s_%s_%s" % c for c in ROUTING])
def test_automatic_route_choices(dk, dv, n, dt, fam, expect):
    r = np.random.default_rng(dk + 7 * n + len(fam))
    Bn, H = 4, 2
    parents0 = [inputs.random_tree(r, n, max(2, min(n, 8)), 4) for _ in range(Bn)]
    parents1 = [inputs.random_tree(r, n, max(2, min(n, 8)), 4) for _ in range(Bn)]
    cfg, r0, a0, b0, S0 = _problem(31 + n, Bn, H, dk, dv, n, parents0, dt, fam)
    _, r1, a1, b1, _ = _problem(32 + n, Bn, H, dk, dv, n, parents1, dt, fam)
    say("automatic route dk=%d dv=%d n=%d %s %s: expect %s" % (dk, dv, n, dt, fam, expect))
    s_auto, res_auto = _two_rounds(cfg, r0, a0, b0, r1, a1, b1, S0, fam, "auto")
    s_exp, res_exp = _two_rounds(cfg, r0, a0, b0, r1, a1, b1, S0, fam, expect)
    assert torch.equal(s_auto, s_exp)
    for (o_a, f_a), (o_e, f_e) in zip(res_auto, res_exp):
        assert torch.equal(o_a, o_e)
        assert torch.equal(f_a.u, f_e.u) and torch.equal(f_a.k, f_e.k)
    ref, st = oracle.verify(S0, r0.q32[0], r0.k32[0], r0.v32[0], a0, b0, r0.parent, family=fam)
    assert (st == 0).all()
    err = rel_err(res_auto[0][0].cpu().numpy(), ref)
    say("  round 0 output rel err %.3e" % err)
    assert err <= TOL[dt]
