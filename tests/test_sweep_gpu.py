"""Randomised sweep of shapes and routes through the C ABI against the fp64
oracle: batch, heads, d_k in {64, 128, 256}, d_v ragged against the 64- and
128-column tiles, node counts on both sides of the 16/32/64-row node blocks,
trees, forests and chains, and a pending path from a previous round of a
different size.  Every case runs two fused rounds and checks the committed
state and the second round's outputs (sampled units) within the bf16 bar,
the standalone-commit route bit for bit, and the conv kernel on the same
drafts.  Seeds are fixed; each case prints its shape before it runs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import (TOL, Layer, new_factors, new_out, oracle_commit_units, oracle_verify_units, parallel_supported,
                      rel_err)

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def _cases(seed, count):
    r = np.random.default_rng(seed)
    out = []
    for i in range(count):
        dk = int(r.choice([64, 128, 256]))
        dv = int(r.choice([16, 48, 64, 80, 128, 144, 192, 256, 320]))
        n1 = int(r.choice([1, 2, 7, 15, 16, 17, 31, 32, 33, 47, 63, 64]))
        n0 = int(r.choice([1, 5, 16, 24, 40, 64]))
        Bn = int(r.integers(1, 6))
        H = int(r.integers(1, 5))
        out.append((i, Bn, H, dk, dv, n0, n1, int(r.integers(0, 1 << 30))))
    return out


CASES = _cases(7, 24)


def _draft(cfg, r, kind):
    n = cfg.n_nodes
    if kind == "chain":
        return np.tile(inputs.chain(n), (cfg.batch, 1))
    rows = []
    for b in range(cfg.batch):
        if kind == "forest" or b % 3 == 2:
            rows.append(np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32))
        else:
            rows.append(inputs.random_tree(r, n, max(2, n // 2), 4))
    return np.stack(rows)


@pytest.mark.parametrize("case", CASES, ids=["c%d_B%d_H%d_dk%d_dv%d_n%d-%d" % c[:7] for c in CASES])
@pytest.mark.parametrize("route", ["auto", "serial", "hybrid"])
def test_sweep_two_fused_rounds(case, route):
    _sweep_case(case, route, inputs.BF16)


@pytest.mark.parametrize("case", CASES, ids=["c%d_B%d_H%d_dk%d_dv%d_n%d-%d" % c[:7] for c in CASES])
def test_sweep_two_fused_rounds_f32_parallel(case):
    """The same cases with fp32 q/k/v on the fp32 matrix-core contraction
    (1e-5 bar); a draft whose on-chip stage would not fit is refused."""
    _sweep_case(case, "parallel", inputs.F32)


def _sweep_case(case, route, dt):
    i, Bn, H, dk, dv, n0, n1, seed = case
    r = np.random.default_rng(seed)
    say("sweep case %d route %s dtype %s: B=%d H=%d dk=%d dv=%d n0=%d n1=%d"
        % (i, route, dt, Bn, H, dk, dv, n0, n1))
    if route == "parallel" and not all(parallel_supported(dk, dv, m, dt) for m in (n0, n1)):
        pytest.skip("the draft's on-chip stage does not fit the parallel route")
    c0 = inputs.Config("sw0", 300 + i, Bn, H, dk, dv, n0, False, n0, 64, dt, 1)
    c1 = inputs.Config("sw1", 400 + i, Bn, H, dk, dv, n1, False, n1, 64, dt, 1)
    r0 = inputs.draw_round(c0, 0, layers=[0])
    r1 = inputs.draw_round(c1, 0, layers=[0])
    r0.parent = _draft(c0, r, ["tree", "chain", "forest"][i % 3])
    r1.parent = _draft(c1, r, ["forest", "tree", "chain"][i % 3])
    # round 0's accepted paths: the root path of a random node, or empty
    r0.path = np.full((Bn, n0), -1, np.int32)
    r0.length = np.zeros(Bn, np.int32)
    for b in range(Bn):
        if r.random() < 0.85:
            p = inputs.walk_to_root(r0.parent[b], int(r.integers(0, n0)))
            r0.path[b, :len(p)] = p
            r0.length[b] = len(p)
    S0 = inputs.draw_state(c0, 0)
    L0, L1 = Layer(c0, r0, 0), Layer(c1, r1, 0)
    f0, f1, g0, g1 = new_factors(c0), new_factors(c1), new_factors(c0), new_factors(c1)
    out1, o1 = new_out(c1), new_out(c1)
    fused = torch.from_numpy(S0).cuda()
    B.sla_verify(fused, L0.q, L0.k, L0.v, L0.alpha, L0.beta, L0.parent, new_out(c0), f0, route=route)
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    B.sla_verify(fused, L1.q, L1.k, L1.v, L1.alpha, L1.beta, L1.parent, out1, f1,
                 pending=(f0, L0.path, L0.length), status=st, route=route)
    sep = torch.from_numpy(S0).cuda()
    B.sla_verify(sep, L0.q, L0.k, L0.v, L0.alpha, L0.beta, L0.parent, new_out(c0), g0, route=route)
    B.sla_commit(sep, g0, L0.path, L0.length)
    B.sla_verify(sep, L1.q, L1.k, L1.v, L1.alpha, L1.beta, L1.parent, o1, g1, route=route)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep)
    assert torch.equal(out1, o1)
    units = [(b, h) for b in range(Bn) for h in range(H)]
    if len(units) > 8:
        units = [units[j] for j in sorted(r.choice(len(units), 8, replace=False))]
    S1 = oracle_commit_units(S0, r0, 0, units)
    es = rel_err(np.stack([fused.cpu().numpy()[b, h] for b, h in units]), np.stack([S1[u] for u in units]))
    S1f = S0.astype(np.float64)
    for (b, h), s_ in S1.items():
        S1f[b, h] = s_
    ref = oracle_verify_units(S1f, r1, 0, units)
    got = out1.cpu().numpy()
    eo = rel_err(np.stack([got[b, :, h] for b, h in units]), np.stack([ref[u] for u in units]))
    say("sweep case %d route %s: state err %.2e output err %.2e" % (i, route, es, eo))
    assert es <= TOL[dt] and eo <= TOL[dt]


@pytest.mark.parametrize("case", CASES[:12], ids=["c%d" % c[0] for c in CASES[:12]])
def test_sweep_conv_on_the_same_drafts(case):
    i, Bn, H, dk, dv, n0, n1, seed = case
    r = np.random.default_rng(seed + 1)
    D = 8 * int(r.integers(1, 160))
    K = int(r.integers(1, 5))
    say("conv sweep case %d: B=%d D=%d K=%d n0=%d n1=%d" % (i, Bn, D, K, n0, n1))
    c0 = inputs.Config("cs0", 500 + i, Bn, 1, 64, 64, n0, False, n0, 64, inputs.BF16, 1)
    c1 = inputs.Config("cs1", 600 + i, Bn, 1, 64, 64, n1, False, n1, 64, inputs.BF16, 1)
    p0 = _draft(c0, r, "tree")
    p1 = _draft(c1, r, "forest")
    path = np.full((Bn, n0), -1, np.int32)
    ln = np.zeros(Bn, np.int32)
    for b in range(Bn):
        p = inputs.walk_to_root(p0[b], int(r.integers(0, n0)))
        path[b, :len(p)] = p
        ln[b] = len(p)
    x0s, x0 = inputs._to_dtype(r.standard_normal((Bn, n0, D)), inputs.BF16)
    x1s, x1 = inputs._to_dtype(r.standard_normal((Bn, n1, D)), inputs.BF16)
    w = r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)
    C = inputs._to_dtype(r.standard_normal((Bn, K - 1, D)), inputs.BF16)[1].astype(np.float32)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    X0, X1 = bf(x0s), bf(x1s)
    P0, P1 = torch.from_numpy(p0).cuda(), torch.from_numpy(p1).cuda()
    Cg = torch.from_numpy(C).cuda() if K > 1 else None
    wg = torch.from_numpy(w).cuda()
    y0, y1 = torch.empty_like(X0), torch.empty_like(X1)
    B.sla_conv_verify(Cg, X0, wg, P0, y0)
    B.sla_conv_verify(Cg, X1, wg, P1, y1, pending=(X0, P0, torch.from_numpy(path).cuda(), torch.from_numpy(ln).cuda()))
    torch.cuda.synchronize()
    C1, _ = oracle.conv_commit(C if K > 1 else np.zeros((Bn, 0, D)), x0, p0, path, ln)
    if K > 1:
        np.testing.assert_array_equal(Cg.cpu().numpy().astype(np.float64), C1)
    ref, _ = oracle.conv_verify(C1, x1, w, None, p1)
    got = inputs.bf16_to_f32(y1.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * np.max(np.abs(ref))
    assert (np.abs(got - ref) <= bound).all()
