"""GPU parity of the other layer families (DeltaNet, scalar decay without the
delta rule, GLA's per-key gates; the factor-record remark closing §5.1)
against the fp64 oracle, through the C ABI, on both verification routes.

Per case: round 0 verified from the committed state (outputs against the
oracle, factor records against their definition: the key and gate copies
exact, the stored value exactly v for the no-delta families); round 1 with
round 0's accepted path pending (fused) and, separately, a standalone commit
followed by a plain verification: states and outputs bitwise equal between
the two, the committed state and round 1's outputs against the oracle.
Bars: 1e-5 (all-fp32 inputs) or 2e-3 (bf16 q/k/v), normwise max relative.
"""
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


GLA_DK256_N50 = inputs.Config("gla_dk256_n50", 50, 2, 2, 256, 64, 50, False, 7, 4, inputs.BF16, 1,
                              "batch 2, 2 heads, dk=256, dv=64, 50-node tree (the largest GLA draft at dk=256)")
# d_k = 256 with fp32 activations: 30 nodes, inside the parallel route's
# fp32 stage (the fp32 matrix cores; GLA's fp32 Q~)
F32_DK256_N30 = inputs.Config("f32_dk256_n30", 52, 2, 3, 256, 80, 30, False, 7, 4, inputs.F32, 1,
                              "batch 2, 3 heads, dk=256, dv=80, 30-node tree, fp32 q/k/v")


def _cfg(name):
    return {c.name: c for c in (GLA_DK256_N50, F32_DK256_N30)}.get(name) or inputs.config(name)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if x is not None else None


class Draft:
    """One round's device tensors and exact host values for one family."""

    def __init__(self, cfg, fam, round_index):
        self.rnd = inputs.draw_round(cfg, round_index, layers=[0])
        self.alpha, self.beta = inputs.family_gates(cfg, self.rnd, 0, fam, layer=0, round_index=round_index)
        dt = cfg.dtype
        self.q = act_tensor(self.rnd.q[0], dt)
        self.k = act_tensor(self.rnd.k[0], dt)
        self.v = act_tensor(self.rnd.v[0], dt)
        self.a = _dev(self.alpha)
        self.b = _dev(self.beta)
        self.parent = _dev(self.rnd.parent)
        self.path = _dev(self.rnd.path)
        self.length = _dev(self.rnd.length)


def _factors(cfg, fam):
    dt = torch.bfloat16 if cfg.dtype == inputs.BF16 else torch.float32
    return B.Factors.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v, dt, family=fam)


def _verify(cfg, fam, route, state, d, out, f, pending=None):
    st = torch.full((cfg.batch,), 99, dtype=torch.int32, device="cuda")
    B.sla_verify(state, d.q, d.k, d.v, d.a, d.b, d.parent, out, f, pending=pending, status=st,
                 topology="chain" if cfg.chain else "tree", route=route, family=fam)
    return st


def _unit_slices(d, b, h):
    a = None if d.alpha is None else d.alpha[b:b + 1, :, h:h + 1]
    bt = None if d.beta is None else d.beta[b:b + 1, :, h:h + 1]
    r = d.rnd
    return (r.q32[0][b:b + 1, :, h:h + 1], r.k32[0][b:b + 1, :, h:h + 1], r.v32[0][b:b + 1, :, h:h + 1], a, bt)


def _oracle_out(S, d, units, fam):
    res = []
    for b, h in units:
        q, k, v, a, bt = _unit_slices(d, b, h)
        o, st = oracle.verify(S[(b, h)][None, None], q, k, v, a, bt, d.rnd.parent[b:b + 1], family=fam)
        assert st[0] == 0
        res.append(o[0, :, 0])
    return np.stack(res)


def _oracle_commit(S0, d, units, fam):
    res = {}
    for b, h in units:
        _, k, v, a, bt = _unit_slices(d, b, h)
        S, st = oracle.commit(S0[b:b + 1, h:h + 1], k, v, a, bt, d.rnd.parent[b:b + 1], d.rnd.path[b:b + 1],
                              d.rnd.length[b:b + 1], family=fam)
        assert st[0] == 0
        res[(b, h)] = S[0, 0]
    return res


CASES = [(name, fam, route)
         for name in ["tiny_chain_f32", "chain8_bf16", "tree32_bf16", "paper_fused_shape",
                      "batched_tree_serving", "large_batch_tree64"]
         for fam in ["deltanet", "decay", "gla"]
         for route in ["serial", "parallel"]]
# fp32 q/k/v on the parallel route (the fp32 matrix-core contraction)
CASES += [(name, fam, "parallel") for name in ["batched_tree_serving_f32", "large_batch_tree64_f32",
                                                F32_DK256_N30.name]
          for fam in ["deltanet", "decay", "gla"]]
CASES += [(F32_DK256_N30.name, "gla", "auto")]
# the largest GLA draft at d_k = 256 exceeds the parallel route's on-chip stage:
# the automatic route falls back to the serial one
CASES += [(GLA_DK256_N50.name, "gla", "serial"), (GLA_DK256_N50.name, "gla", "auto")]
# the chain-decomposed hybrid on the tree workloads (chains run as serial)
CASES += [(name, fam, "hybrid") for name in ["tree32_bf16", "batched_tree_serving", "large_batch_tree64"]
          for fam in ["deltanet", "decay", "gla"]] + [(GLA_DK256_N50.name, "gla", "hybrid")]


@pytest.mark.parametrize("name,fam,route", CASES)
def test_family_two_rounds(name, fam, route):
    cfg = _cfg(name)
    tol = TOL[cfg.dtype]
    nunits = 12 if cfg.n_nodes >= 64 else 32
    units = sample_units(cfg, nunits, 7)
    d0, d1 = Draft(cfg, fam, 0), Draft(cfg, fam, 1)
    S0 = inputs.draw_state(cfg, 0)
    Bn, n, H = cfg.batch, cfg.n_nodes, cfg.heads

    # round 0 from the committed state
    state = torch.from_numpy(S0).cuda()
    out0 = torch.empty(Bn, n, H, cfg.d_v, device="cuda")
    f0 = _factors(cfg, fam)
    say("family %s %s route=%s round 0" % (fam, name, route))
    st = _verify(cfg, fam, route, state, d0, out0, f0)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    np.testing.assert_array_equal(state.cpu().numpy(), S0)
    got = out0.cpu().numpy()
    err = rel_err(np.stack([got[b, :, h] for b, h in units]),
                  _oracle_out({u: S0[u[0], u[1]] for u in units}, d0, units, fam))
    say("  round 0 output rel err %.3e" % err)
    assert err <= tol
    # factor records
    assert torch.equal(f0.k, d0.k)
    np.testing.assert_array_equal(f0.parent.cpu().numpy(), d0.rnd.parent)
    gate = np.ones((Bn, n, H), np.float32) if fam == "deltanet" else d0.alpha
    np.testing.assert_array_equal(f0.alpha.cpu().numpy(), gate)
    if fam in ("decay", "gla"):
        np.testing.assert_array_equal(f0.u.cpu().numpy(), d0.rnd.v32[0])

    # round 1: fused (pending) against standalone commit + plain verify
    sf = torch.from_numpy(S0).cuda()
    ss = torch.from_numpy(S0).cuda()
    out_f = torch.empty_like(out0)
    out_s = torch.empty_like(out0)
    f1f, f1s = _factors(cfg, fam), _factors(cfg, fam)
    say("  round 1 fused")
    st = _verify(cfg, fam, route, sf, d1, out_f, f1f, pending=(f0, d0.path, d0.length))
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    say("  round 1 standalone commit + verify")
    cst = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    B.sla_commit(ss, f0, d0.path, d0.length, status=cst, family=fam)
    st = _verify(cfg, fam, route, ss, d1, out_s, f1s)
    torch.cuda.synchronize()
    assert (cst.cpu().numpy() == 0).all() and (st.cpu().numpy() == 0).all()
    assert torch.equal(sf, ss)
    assert torch.equal(out_f, out_s)
    assert torch.equal(f1f.u, f1s.u)

    refS = _oracle_commit(S0, d0, units, fam)
    gotS = sf.cpu().numpy()
    errS = rel_err(np.stack([gotS[b, h] for b, h in units]), np.stack([refS[u] for u in units]))
    say("  committed state rel err %.3e" % errS)
    assert errS <= tol
    got = out_f.cpu().numpy()
    err1 = rel_err(np.stack([got[b, :, h] for b, h in units]), _oracle_out(refS, d1, units, fam))
    say("  round 1 output rel err %.3e" % err1)
    assert err1 <= tol


def test_gla_parallel_route_refuses_drafts_beyond_its_stage():
    cfg = GLA_DK256_N50
    d = Draft(cfg, "gla", 0)
    state = torch.from_numpy(inputs.draw_state(cfg, 0)).cuda()
    out = torch.empty(cfg.batch, cfg.n_nodes, cfg.heads, cfg.d_v, device="cuda")
    with pytest.raises(B.SlaError) as e:
        _verify(cfg, "gla", "parallel", state, d, out, _factors(cfg, "gla"))
    assert e.value.code == B.SLA_ERR_UNSUPPORTED


def test_gla_draft_beyond_the_on_chip_stage_is_rejected():
    """GLA at d_k = 256 stages keys, queries and gates of every node on chip:
    51 nodes need more than 160 KiB, rejected on the host before any launch."""
    z = torch.zeros
    n = 51
    q = z(1, n, 1, 256, dtype=torch.bfloat16, device="cuda")
    v = z(1, n, 1, 16, dtype=torch.bfloat16, device="cuda")
    par = torch.arange(-1, n - 1, dtype=torch.int32, device="cuda")[None]
    f = B.Factors.empty(1, n, 1, 256, 16, torch.bfloat16, family="gla")
    with pytest.raises(B.SlaError) as e:
        B.sla_verify(z(1, 1, 256, 16, device="cuda"), q, q, v, z(1, n, 1, 256, device="cuda"), None, par,
                     z(1, n, 1, 16, device="cuda"), f, family="gla")
    assert e.value.code == B.SLA_ERR_UNSUPPORTED


# ------------------------------------------------------------ random shapes
def _sweep_cases(seed, count):
    r = np.random.default_rng(seed)
    out = []
    for i in range(count):
        out.append((i, ["deltanet", "decay", "gla"][i % 3], int(r.integers(1, 5)), int(r.integers(1, 4)),
                    int(r.choice([64, 128, 256])), int(r.choice([16, 48, 64, 80, 128, 144, 192])),
                    int(r.choice([1, 3, 16, 17, 32, 33, 50, 64])), int(r.choice([1, 2, 15, 31, 40, 64])),
                    int(r.integers(0, 1 << 30))))
    return out


SWEEP = _sweep_cases(11, 18)


def _random_parent(r, Bn, n):
    rows = []
    for b in range(Bn):
        if b % 2:
            rows.append(np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32))
        else:
            rows.append(inputs.random_tree(r, n, max(2, n // 2), 4))
    return np.stack(rows)


@pytest.mark.parametrize("case", SWEEP, ids=["s%d_%s_B%d_H%d_dk%d_dv%d_n%d-%d" % c[:8] for c in SWEEP])
@pytest.mark.parametrize("route", ["auto", "serial"])
def test_family_sweep_two_fused_rounds(case, route):
    """Random shapes (d_k 64/128/256, ragged d_v, node counts across the
    16/32/64 blocks, trees and forests, pending rounds of another size):
    two fused rounds against verify + standalone commit bitwise, and the
    committed state and second outputs against the oracle."""
    _family_sweep_case(case, route, inputs.BF16)


@pytest.mark.parametrize("case", SWEEP, ids=["s%d_%s_B%d_H%d_dk%d_dv%d_n%d-%d" % c[:8] for c in SWEEP])
def test_family_sweep_f32_parallel(case):
    """The same shapes with fp32 q/k/v on the parallel route (the fp32
    matrix cores; GLA's scores on the vector ALUs with Q~ kept in fp32), at
    the 1e-5 bar.  Drafts of more than 32 nodes at d_k = 256 do not fit the
    route's on-chip stage with fp32 activations and are refused there."""
    _family_sweep_case(case, "parallel", inputs.F32)


def _family_sweep_case(case, route, dt):
    i, fam, Bn, H, dk, dv, n0, n1, seed = case
    r = np.random.default_rng(seed)
    say("family sweep %d %s route %s dtype %s: B=%d H=%d dk=%d dv=%d n0=%d n1=%d"
        % (i, fam, route, dt, Bn, H, dk, dv, n0, n1))
    cfgs = [inputs.Config("fs%d" % k, 700 + 2 * i + k, Bn, H, dk, dv, n, False, n, 64, dt, 1)
            for k, n in ((0, n0), (1, n1))]
    drafts = []
    for k, cfg in enumerate(cfgs):
        d = Draft(cfg, fam, 0)
        d.rnd.parent = _random_parent(r, Bn, cfg.n_nodes)
        d.parent = _dev(d.rnd.parent)
        drafts.append(d)
    d0, d1 = drafts
    path = np.full((Bn, n0), -1, np.int32)
    ln = np.zeros(Bn, np.int32)
    for b in range(Bn):
        if r.random() < 0.85:
            p = inputs.walk_to_root(d0.rnd.parent[b], int(r.integers(0, n0)))
            path[b, :len(p)] = p
            ln[b] = len(p)
    d0.rnd.path, d0.rnd.length = path, ln
    d0.path, d0.length = _dev(path), _dev(ln)
    S0 = inputs.draw_state(cfgs[0], 0)
    # beyond the on-chip stage at d_k = 256: the parallel route holds 32 nodes
    # with GLA's gates or fp32 activations; the serial routes (and AUTO's
    # fallback to them) 50 nodes with GLA's gates
    if route == "parallel":
        limit = 32 if (fam == "gla" or dt == inputs.F32) else 64
    else:
        limit = 50 if fam == "gla" else 64
    too_big = dk == 256 and max(n0, n1) > limit
    f0, f1, g0, g1 = (_factors(c, fam) for c in (cfgs[0], cfgs[1], cfgs[0], cfgs[1]))
    out1, o1 = (torch.empty(Bn, n1, H, dv, device="cuda") for _ in range(2))
    fused = torch.from_numpy(S0).cuda()
    if too_big:
        with pytest.raises(B.SlaError) as e:
            _verify(cfgs[0] if n0 > limit else cfgs[1], fam, route, fused, d0 if n0 > limit else d1,
                    torch.empty(Bn, max(n0, n1), H, dv, device="cuda"), f0 if n0 > limit else f1)
        assert e.value.code == B.SLA_ERR_UNSUPPORTED
        return
    _verify(cfgs[0], fam, route, fused, d0, torch.empty(Bn, n0, H, dv, device="cuda"), f0)
    st = _verify(cfgs[1], fam, route, fused, d1, out1, f1, pending=(f0, d0.path, d0.length))
    sep = torch.from_numpy(S0).cuda()
    _verify(cfgs[0], fam, route, sep, d0, torch.empty(Bn, n0, H, dv, device="cuda"), g0)
    B.sla_commit(sep, g0, d0.path, d0.length, family=fam)
    _verify(cfgs[1], fam, route, sep, d1, o1, g1)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep)
    assert torch.equal(out1, o1)
    units = [(b, h) for b in range(Bn) for h in range(H)]
    if len(units) > 6:
        units = [units[j] for j in sorted(r.choice(len(units), 6, replace=False))]
    refS = _oracle_commit(S0, d0, units, fam)
    es = rel_err(np.stack([fused.cpu().numpy()[b, h] for b, h in units]), np.stack([refS[u] for u in units]))
    got = out1.cpu().numpy()
    eo = rel_err(np.stack([got[b, :, h] for b, h in units]), _oracle_out(refS, d1, units, fam))
    say("  state err %.2e output err %.2e" % (es, eo))
    assert es <= TOL[dt] and eo <= TOL[dt]
