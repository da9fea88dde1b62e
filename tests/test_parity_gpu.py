"""GPU parity of the HIP library against the fp64 oracle, through the C ABI.

Bars: topology tables, orders and commit indexing bit-exact; outputs and
committed states within normwise max relative error 1e-5 (all-fp32 inputs)
or 2e-3 (bf16 q/k/v, fp32 state and gates).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import (TOL, parallel_supported, Layer, act_tensor, new_factors, new_out, oracle_commit_units,
                      oracle_verify_units, rel_err, sample_units, verify)

pytestmark = pytest.mark.gpu

ROUTES = ["serial", "parallel", "hybrid"]


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


# ----------------------------------------------------------------- topology
def test_device_topology_bit_exact():
    r = np.random.default_rng(40)
    rows = []
    for n in [1, 2, 5, 16, 33, 64]:
        for _ in range(6):
            rows.append((n, inputs.random_tree(r, n, 64, 6)))
            rows.append((n, np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32)))
        rows.append((n, inputs.chain(n)))
        rows.append((n, np.full(n, -1, np.int32)))
    for n in sorted({n for n, _ in rows}):
        par = np.stack([p for m, p in rows if m == n])
        bad = par.copy()
        if n > 1:
            bad[0, n - 1] = n - 1  # self parent
            par = np.concatenate([par, bad[:1]])
        say("device topology n=%d rows=%d" % (n, len(par)))
        t = B.sla_topology(torch.from_numpy(par).cuda())
        torch.cuda.synchronize()
        for i, row in enumerate(par):
            o = oracle.topology(row)
            assert int(t["status"][i]) == o["status"]
            if o["status"] != 0:
                continue
            np.testing.assert_array_equal(t["depth"][i].cpu().numpy(), o["depth"])
            np.testing.assert_array_equal(t["anc"][i].cpu().numpy().view(np.uint64), o["anc"])
            np.testing.assert_array_equal(t["order"][i].cpu().numpy(), o["order"])
            np.testing.assert_array_equal(t["n_children"][i].cpu().numpy(), o["n_children"])


# ------------------------------------------------- one round, small configs
def _one_round(cfg, route, batch=None):
    rnd = inputs.draw_round(cfg, 0, layers=[0], batch=batch)
    S0 = inputs.draw_state(cfg, 0, batch=batch)
    L = Layer(cfg, rnd, 0)
    state = torch.from_numpy(S0).cuda()
    out = new_out(cfg, batch)
    f = new_factors(cfg, batch)
    Bn = S0.shape[0]
    status = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    say("verify %s route=%s B=%d" % (cfg.name, route, Bn))
    verify(state, L, out, f, status=status, route=route)
    torch.cuda.synchronize()
    assert (status.cpu().numpy() == 0).all()
    np.testing.assert_array_equal(state.cpu().numpy(), S0)  # no pending: state only read
    return rnd, S0, L, state, out, f


SMALL = ["tiny_chain_f32", "chain8_bf16", "tree32_bf16", "paper_fused_shape"]


@pytest.mark.parametrize("route", ROUTES)
@pytest.mark.parametrize("name", SMALL)
def test_verify_and_commit_small_configs(name, route):
    cfg = inputs.config(name)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0, L, state, out, f = _one_round(cfg, route)
    units = sample_units(cfg, 64, 1)
    ref = oracle_verify_units(S0, rnd, 0, units)
    got = out.cpu().numpy()
    err = rel_err(np.stack([got[b, :, h] for b, h in units]), np.stack([ref[u] for u in units]))
    say("%s %s output rel err %.3e" % (name, route, err))
    assert err <= TOL[cfg.dtype]
    # factor records: k, alpha and parent are exact copies
    np.testing.assert_array_equal(f.parent.cpu().numpy(), rnd.parent)
    np.testing.assert_array_equal(f.alpha.cpu().numpy(), rnd.alpha[0])
    assert torch.equal(f.k, L.k)
    # standalone commit of the accepted path
    st = torch.full((S0.shape[0],), 99, dtype=torch.int32, device="cuda")
    say("commit %s" % name)
    B.sla_commit(state, f, L.path, L.length, status=st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    refS = oracle_commit_units(S0, rnd, 0, units)
    gotS = state.cpu().numpy()
    errS = rel_err(np.stack([gotS[b, h] for b, h in units]), np.stack([refS[u] for u in units]))
    say("%s %s committed state rel err %.3e" % (name, route, errS))
    assert errS <= TOL[cfg.dtype]


def _parallel_ok(cfg):
    # a PARALLEL request on an unsupported shape is rejected host-side, before
    # any launch, with SLA_ERR_UNSUPPORTED
    return parallel_supported(cfg.d_k, cfg.d_v, cfg.n_nodes, cfg.dtype)


# ------------------------------------------- fused commit-and-verify (§5.2)
@pytest.mark.parametrize("route", ROUTES)
@pytest.mark.parametrize("name", ["tiny_chain_f32", "chain8_bf16", "tree32_bf16"])
def test_fused_round_matches_oracle_and_standalone_bitwise(name, route):
    _fused_round_check(inputs.config(name), route)


# Larger trees over several V-tiles: two tiles per workgroup (d_v 80 with a
# partial second tile, d_v 128), one per workgroup (d_v 192, three tiles);
# root paths within and beyond the depth that solves T in registers; and
# small trees at batch sizes where they pair V-tiles too.
LARGE = [
    inputs.Config("tree48_dv80", 95, 3, 3, 128, 80, 48, False, 6, 4, inputs.BF16, 1),
    inputs.Config("tree48_dv128", 96, 2, 4, 128, 128, 48, False, 12, 3, inputs.BF16, 1),
    inputs.Config("tree60_dv192", 97, 2, 2, 128, 192, 60, False, 8, 4, inputs.BF16, 1),
    inputs.Config("tree40_dv256_dk64", 98, 2, 2, 64, 256, 40, False, 10, 3, inputs.BF16, 1),
    # batches large enough that small trees take two V-tiles per workgroup
    # (13 and 27 nodes: ragged against the 16- and 32-row node blocks; paths
    # up to 12 deep, past the records staged on chip; d_v 256: two pairs)
    inputs.Config("pair_tree13", 112, 64, 16, 128, 128, 13, False, 5, 3, inputs.BF16, 1),
    inputs.Config("pair_tree27_deep", 113, 64, 16, 128, 128, 27, False, 12, 3, inputs.BF16, 1),
    inputs.Config("pair_tree16_dv256", 114, 32, 16, 128, 256, 16, False, 5, 3, inputs.BF16, 1),
    # paired tiles whose second tile's first d_k/2 state rows are staged in
    # LDS early: a ragged second tile (16 of its 64 columns inside d_v = 80),
    # and d_k 64 (a half-size stage)
    inputs.Config("pair_tree16_dv80", 116, 64, 32, 128, 80, 16, False, 5, 3, inputs.BF16, 1),
    inputs.Config("pair_tree11_dk64", 117, 64, 16, 64, 128, 11, False, 4, 3, inputs.BF16, 1),
    # 48-node trees at d_v 256: 128-column tiles, eight waves with the setup
    # work on wave 0; 1024 workgroups are one full round at two per CU on a
    # 256-CU part (state reads held back, committed rows written through)
    inputs.Config("tree48_dv256_round", 115, 64, 16, 128, 256, 48, False, 8, 4, inputs.BF16, 1),
    # fp32 q/k/v on the fp32 matrix-core contraction: paired tiles with the
    # early-staged state rows, d_k 64 and 256, eight-wave 128-column tiles,
    # and a 64-node tree (a 64-row node block)
    inputs.Config("pair_tree13_f32", 118, 64, 16, 128, 128, 13, False, 5, 3, inputs.F32, 1),
    inputs.Config("pair_tree11_dk64_f32", 119, 64, 16, 64, 128, 11, False, 4, 3, inputs.F32, 1),
    inputs.Config("tree30_dv80_dk256_f32", 120, 2, 3, 256, 80, 30, False, 10, 3, inputs.F32, 1),
    inputs.Config("tree48_dv256_round_f32", 121, 64, 16, 128, 256, 48, False, 8, 4, inputs.F32, 1),
    inputs.Config("tree64_dv144_f32", 122, 3, 2, 128, 144, 64, False, 12, 4, inputs.F32, 1),
]


@pytest.mark.parametrize("cfg", LARGE, ids=[c.name for c in LARGE])
def test_fused_rounds_large_trees_many_tiles(cfg):
    _fused_round_check(cfg, "parallel")


def _fused_round_check(cfg, route):
    name = cfg.name
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    r0 = inputs.draw_round(cfg, 0, layers=[0])
    r1 = inputs.draw_round(cfg, 1, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L0, L1 = Layer(cfg, r0, 0), Layer(cfg, r1, 0)
    f0, f1 = new_factors(cfg), new_factors(cfg)
    out0, out1 = new_out(cfg), new_out(cfg)
    # fused: verify round 0, then verify round 1 with round 0's accepted path pending
    fused = torch.from_numpy(S0).cuda()
    say("fused rounds %s %s" % (name, route))
    verify(fused, L0, out0, f0, route=route)
    st = torch.full((cfg.batch,), 99, dtype=torch.int32, device="cuda")
    verify(fused, L1, out1, f1, pending=(f0, L0.path, L0.length), status=st, route=route)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    # separate: verify round 0, standalone commit, verify round 1 from the committed state
    sep = torch.from_numpy(S0).cuda()
    g0, g1 = new_factors(cfg), new_factors(cfg)
    o0, o1 = new_out(cfg), new_out(cfg)
    verify(sep, L0, o0, g0, route=route)
    B.sla_commit(sep, g0, L0.path, L0.length)
    verify(sep, L1, o1, g1, route=route)
    torch.cuda.synchronize()
    assert torch.equal(fused, sep), "fused and standalone commit differ"
    assert torch.equal(out1, o1), "fused and separate verification outputs differ"
    assert torch.equal(f1.u, g1.u)
    # oracle: committed state and round-1 outputs
    units = sample_units(cfg, 64, 2)
    S1 = oracle_commit_units(S0, r0, 0, units)
    gotS = fused.cpu().numpy()
    errS = rel_err(np.stack([gotS[b, h] for b, h in units]), np.stack([S1[u] for u in units]))
    S1full = S0.astype(np.float64).copy()
    for (b, h), s in S1.items():
        S1full[b, h] = s
    ref = oracle_verify_units(S1full, r1, 0, units)
    got = out1.cpu().numpy()
    err = rel_err(np.stack([got[b, :, h] for b, h in units]), np.stack([ref[u] for u in units]))
    say("%s %s fused: state err %.3e output err %.3e" % (name, route, errS, err))
    assert errS <= TOL[cfg.dtype] and err <= TOL[cfg.dtype]


# ------------------------------------------------------------ edge cases
def _random_problem(seed, Bn, H, dk, dv, n, parents, dtype=inputs.BF16):
    r = np.random.default_rng(seed)
    q = r.standard_normal((Bn, n, H, dk))
    k = r.standard_normal((Bn, n, H, dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = r.standard_normal((Bn, n, H, dv))
    qs, q32 = inputs._to_dtype(q, dtype)
    ks, k32 = inputs._to_dtype(k, dtype)
    vs, v32 = inputs._to_dtype(v, dtype)
    alpha = (1 / (1 + np.exp(-r.uniform(2, 5, (Bn, n, H))))).astype(np.float32)
    beta = (1 / (1 + np.exp(-r.standard_normal((Bn, n, H))))).astype(np.float32)
    S0 = (r.standard_normal((Bn, H, dk, dv)) * 0.02).astype(np.float32)
    rnd = inputs.Round(parent=np.asarray(parents, np.int32), path=np.full((Bn, n), -1, np.int32),
                       length=np.zeros(Bn, np.int32), q=[qs], k=[ks], v=[vs], q32=[q32], k32=[k32],
                       v32=[v32], alpha=[alpha], beta=[beta])
    return rnd, S0


def _run_and_check(rnd, S0, cfg, route, topo="tree"):
    L = Layer(cfg, rnd, 0)
    state = torch.from_numpy(S0).cuda()
    out = new_out(cfg)
    f = new_factors(cfg)
    st = torch.full((cfg.batch,), 99, dtype=torch.int32, device="cuda")
    B.sla_verify(state, L.q, L.k, L.v, L.alpha, L.beta, L.parent, out, f, status=st,
                 topology=topo, route=route)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    units = [(b, h) for b in range(cfg.batch) for h in range(cfg.heads)]
    ref = oracle_verify_units(S0, rnd, 0, units)
    got = out.cpu().numpy()
    err = rel_err(np.stack([got[b, :, h] for b, h in units]), np.stack([ref[u] for u in units]))
    return err, out, f, state


@pytest.mark.parametrize("route", ROUTES)
def test_ragged_shapes_many_tiles(route):
    """d_v not a multiple of the 64-column tile, odd n, odd batch/heads, forests."""
    Bn, H, dk, dv, n = 3, 5, 128, 80, 13
    r = np.random.default_rng(41)
    parents = [inputs.random_tree(r, n, 5, 3),
               np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32),
               np.full(n, -1, np.int32)]
    cfg = inputs.Config("ragged", 90, Bn, H, dk, dv, n, False, 5, 3, inputs.BF16, 1)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0 = _random_problem(42, Bn, H, dk, dv, n, parents)
    say("ragged %s" % route)
    err, *_ = _run_and_check(rnd, S0, cfg, route)
    say("ragged %s err %.3e" % (route, err))
    assert err <= 2e-3


@pytest.mark.parametrize("route", ROUTES)
@pytest.mark.parametrize("dk,dv", [(64, 64), (256, 256), (128, 32)])
def test_head_dims(route, dk, dv):
    Bn, H, n = 2, 3, 9
    r = np.random.default_rng(43)
    parents = [inputs.random_tree(r, n, 4, 3) for _ in range(Bn)]
    cfg = inputs.Config("dims", 91, Bn, H, dk, dv, n, False, 4, 3, inputs.BF16, 1)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0 = _random_problem(44, Bn, H, dk, dv, n, parents)
    say("dims %d %d %s" % (dk, dv, route))
    err, *_ = _run_and_check(rnd, S0, cfg, route)
    say("dims %d %d %s err %.3e" % (dk, dv, route, err))
    assert err <= 2e-3


@pytest.mark.parametrize("route", ROUTES)
def test_max_nodes_deep_and_wide(route):
    """64 nodes: a 64-deep chain given as a tree, a star, and a random tree."""
    Bn, H, dk, dv, n = 3, 2, 128, 64, 64
    r = np.random.default_rng(45)
    parents = [inputs.chain(n), np.concatenate([[-1], np.zeros(n - 1, np.int32)]),
               inputs.random_tree(r, n, 8, 4)]
    cfg = inputs.Config("max", 92, Bn, H, dk, dv, n, False, 64, 64, inputs.BF16, 1)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0 = _random_problem(46, Bn, H, dk, dv, n, parents)
    say("max nodes %s" % route)
    err, *_ = _run_and_check(rnd, S0, cfg, route)
    say("max nodes %s err %.3e" % (route, err))
    assert err <= 2e-3


def test_chain_kernel_equals_tree_kernel_on_chains():
    cfg = inputs.config("chain8_bf16")
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L = Layer(cfg, rnd, 0)
    outs = []
    for topo in ["chain", "tree"]:
        state = torch.from_numpy(S0).cuda()
        out = new_out(cfg)
        f = new_factors(cfg)
        B.sla_verify(state, L.q, L.k, L.v, L.alpha, L.beta, L.parent, out, f, topology=topo,
                     route="serial")
        outs.append((out, f.u))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_deterministic_repeat():
    cfg = inputs.config("tree32_bf16")
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L = Layer(cfg, rnd, 0)
    res = []
    for _ in range(2):
        state = torch.from_numpy(S0).cuda()
        out = new_out(cfg)
        f = new_factors(cfg)
        verify(state, L, out, f)
        B.sla_commit(state, f, L.path, L.length)
        res.append((out, state))
    torch.cuda.synchronize()
    assert torch.equal(res[0][0], res[1][0]) and torch.equal(res[0][1], res[1][1])


# ------------------------------------------------ dyadic probes (bit-exact)
@pytest.mark.parametrize("route", ROUTES)
def test_dyadic_probe_reveals_ancestry_and_commit_indices(route):
    """beta = 0, alpha in {1, 1/2}: o_j / o_j(alpha = 1) equals gamma_j exactly, and
    the committed state is exactly gamma_A H0 -- a bit-exact check of ancestry and
    of which factor records the commit applied."""
    Bn, H, dk, dv, n = 4, 2, 128, 64, 24
    r = np.random.default_rng(47)
    parents = [inputs.random_tree(r, n, 6, 3) for _ in range(Bn)]
    cfg = inputs.Config("dyadic", 93, Bn, H, dk, dv, n, False, 6, 3, inputs.BF16, 1)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0 = _random_problem(48, Bn, H, dk, dv, n, parents)
    rnd.beta[0][:] = 0.0
    ones = rnd.alpha[0].copy()
    ones[:] = 1.0
    probe = np.where(r.random(ones.shape) < 0.3, 0.5, 1.0).astype(np.float32)
    outs = {}
    for tag, al in [("one", ones), ("probe", probe)]:
        rnd.alpha[0] = al
        L = Layer(cfg, rnd, 0)
        state = torch.from_numpy(S0).cuda()
        out = new_out(cfg)
        f = new_factors(cfg)
        verify(state, L, out, f, route=route)
        paths = np.full((Bn, n), -1, np.int32)
        lens = np.zeros(Bn, np.int32)
        for b in range(Bn):
            p = inputs.walk_to_root(rnd.parent[b], n - 1 - b)
            paths[b, :len(p)] = p
            lens[b] = len(p)
        B.sla_commit(state, f, torch.from_numpy(paths).cuda(), torch.from_numpy(lens).cuda())
        torch.cuda.synchronize()
        outs[tag] = (out.cpu().numpy(), state.cpu().numpy(), paths, lens)
    o1, _, _, _ = outs["one"]
    o2, S2, paths, lens = outs["probe"]
    for b in range(Bn):
        for h in range(H):
            for j in range(n):
                g = np.float32(1.0)
                for t in inputs.walk_to_root(rnd.parent[b], j):
                    g = g * probe[b, t, h]
                np.testing.assert_array_equal(o2[b, j, h], g * o1[b, j, h])
            gA = np.float32(1.0)
            for t in paths[b, :lens[b]]:
                gA = gA * probe[b, t, h]
            np.testing.assert_array_equal(S2[b, h], gA * S0[b, h])


@pytest.mark.parametrize("route", ROUTES)
def test_retrieval_property_on_gpu(route):
    """q_j = k_j, beta = 1: every node outputs its own value."""
    Bn, H, dk, dv, n = 2, 4, 128, 64, 16
    r = np.random.default_rng(49)
    parents = [inputs.random_tree(r, n, 5, 3) for _ in range(Bn)]
    cfg = inputs.Config("retr", 94, Bn, H, dk, dv, n, False, 5, 3, inputs.F32, 1)
    if route == "parallel" and not _parallel_ok(cfg):
        pytest.skip("parallel route does not support this shape")
    rnd, S0 = _random_problem(50, Bn, H, dk, dv, n, parents, dtype=inputs.F32)
    rnd.q[0] = rnd.k[0]
    rnd.q32[0] = rnd.k32[0]
    rnd.beta[0][:] = 1.0
    L = Layer(cfg, rnd, 0)
    out = new_out(cfg)
    verify(torch.from_numpy(S0).cuda(), L, out, new_factors(cfg), route=route)
    torch.cuda.synchronize()
    np.testing.assert_allclose(out.cpu().numpy(), rnd.v32[0], atol=2e-5)


# ----------------------------------------------------- device data errors
def test_invalid_topology_sets_status_and_leaves_state():
    cfg = inputs.config("tree32_bf16")
    r0 = inputs.draw_round(cfg, 0, layers=[0])
    r1 = inputs.draw_round(cfg, 1, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L0, L1 = Layer(cfg, r0, 0), Layer(cfg, r1, 0)
    f0, f1 = new_factors(cfg), new_factors(cfg)
    state = torch.from_numpy(S0).cuda()
    verify(state, L0, new_out(cfg), f0)
    L1.parent[0, 5] = 7  # not topological
    st = torch.full((1,), 99, dtype=torch.int32, device="cuda")
    verify(state, L1, new_out(cfg), f1, pending=(f0, L0.path, L0.length), status=st)
    torch.cuda.synchronize()
    assert int(st[0]) == B.SLA_ERR_TOPOLOGY
    np.testing.assert_array_equal(state.cpu().numpy(), S0)


def test_invalid_pending_path_sets_status_and_leaves_state():
    cfg = inputs.config("tree32_bf16")
    r0 = inputs.draw_round(cfg, 0, layers=[0])
    r1 = inputs.draw_round(cfg, 1, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L0, L1 = Layer(cfg, r0, 0), Layer(cfg, r1, 0)
    f0, f1 = new_factors(cfg), new_factors(cfg)
    state = torch.from_numpy(S0).cuda()
    verify(state, L0, new_out(cfg), f0)
    bad_path = L0.path.clone()
    bad_path[0, 0] = 31 if int(L0.parent[0, 31]) != -1 else 30
    length = torch.ones_like(L0.length)
    for p, ln in [(bad_path, length), (L0.path, L0.length + 40), (L0.path, L0.length - 100)]:
        st = torch.full((1,), 99, dtype=torch.int32, device="cuda")
        verify(state, L1, new_out(cfg), f1, pending=(f0, p, ln), status=st)
        st2 = torch.full((1,), 99, dtype=torch.int32, device="cuda")
        B.sla_commit(state, f0, p, ln, status=st2)
        torch.cuda.synchronize()
        assert int(st[0]) == B.SLA_ERR_PATH and int(st2[0]) == B.SLA_ERR_PATH
        np.testing.assert_array_equal(state.cpu().numpy(), S0)


def test_chain_hint_violation_is_reported():
    cfg = inputs.config("tree32_bf16")
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    L = Layer(cfg, rnd, 0)
    st = torch.full((1,), 99, dtype=torch.int32, device="cuda")
    B.sla_verify(torch.from_numpy(inputs.draw_state(cfg, 0)).cuda(), L.q, L.k, L.v, L.alpha, L.beta,
                 L.parent, new_out(cfg), new_factors(cfg), status=st, topology="chain")
    torch.cuda.synchronize()
    assert int(st[0]) == B.SLA_ERR_TOPOLOGY


def test_empty_pending_path_is_a_noop_commit():
    cfg = inputs.config("chain8_bf16")
    r0 = inputs.draw_round(cfg, 0, layers=[0])
    r1 = inputs.draw_round(cfg, 1, layers=[0])
    S0 = inputs.draw_state(cfg, 0)
    L0, L1 = Layer(cfg, r0, 0), Layer(cfg, r1, 0)
    f0, f1 = new_factors(cfg), new_factors(cfg)
    state = torch.from_numpy(S0).cuda()
    verify(state, L0, new_out(cfg), f0)
    zero = torch.zeros_like(L0.length)
    o_a, o_b = new_out(cfg), new_out(cfg)
    verify(state, L1, o_a, f1, pending=(f0, L0.path, zero))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(state.cpu().numpy(), S0)
    verify(torch.from_numpy(S0).cuda(), L1, o_b, new_factors(cfg))
    torch.cuda.synchronize()
    assert torch.equal(o_a, o_b)


# ------------------------- pending path from a differently shaped round
@pytest.mark.parametrize("route", ROUTES)
def test_pending_from_larger_round_with_long_paths(route):
    """Round 0: 24-node chains; the accepted paths (15, 24 and 0 steps) are
    longer than the records staged on chip, so the column waves read the rest
    directly.  Round 1: 16-node trees verified with round 0's path pending
    (the previous store has 24 nodes per sequence, the new one 16)."""
    c0 = inputs.Config("prev24", 110, 3, 4, 128, 128, 24, True, 24, 1, inputs.BF16, 1)
    c1 = inputs.Config("next16", 111, 3, 4, 128, 128, 16, False, 5, 3, inputs.BF16, 1)
    if route == "parallel" and not (_parallel_ok(c0) and _parallel_ok(c1)):
        pytest.skip("parallel route does not support this shape")
    r0 = inputs.draw_round(c0, 0, layers=[0])
    r0.length = np.array([15, 24, 0], np.int32)
    r0.path = np.tile(np.arange(24, dtype=np.int32), (3, 1))
    for b, ln in enumerate(r0.length):
        r0.path[b, ln:] = -1
    r1 = inputs.draw_round(c1, 0, layers=[0])
    S0 = inputs.draw_state(c0, 0)
    L0, L1 = Layer(c0, r0, 0), Layer(c1, r1, 0)
    f0, f1, g0, g1 = new_factors(c0), new_factors(c1), new_factors(c0), new_factors(c1)
    out0, out1, o0, o1 = new_out(c0), new_out(c1), new_out(c0), new_out(c1)
    say("pending from a 24-node round, %s" % route)
    fused = torch.from_numpy(S0).cuda()
    verify(fused, L0, out0, f0, route=route)
    st = torch.full((3,), 99, dtype=torch.int32, device="cuda")
    verify(fused, L1, out1, f1, pending=(f0, L0.path, L0.length), status=st, route=route)
    sep = torch.from_numpy(S0).cuda()
    verify(sep, L0, o0, g0, route=route)
    B.sla_commit(sep, g0, L0.path, L0.length)
    verify(sep, L1, o1, g1, route=route)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep), "fused and standalone commit differ"
    assert torch.equal(out1, o1), "fused and separate verification outputs differ"
    units = [(b, h) for b in range(3) for h in range(4)]
    S1 = oracle_commit_units(S0, r0, 0, units)
    errS = rel_err(np.stack([fused.cpu().numpy()[b, h] for b, h in units]), np.stack([S1[u] for u in units]))
    S1full = S0.astype(np.float64).copy()
    for (b, h), s_ in S1.items():
        S1full[b, h] = s_
    ref = oracle_verify_units(S1full, r1, 0, units)
    got = out1.cpu().numpy()
    err = rel_err(np.stack([got[b, :, h] for b, h in units]), np.stack([ref[u] for u in units]))
    say("pending from a 24-node round, %s: state err %.3e output err %.3e" % (route, errS, err))
    assert errS <= 2e-3 and err <= 2e-3
    # the empty path left sequence 2's state as it was
    np.testing.assert_array_equal(fused.cpu().numpy()[2], S0[2])
