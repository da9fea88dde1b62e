"""GPU parity of the short causal convolution and its conv-state commit
(sla_conv_verify, sla_conv_commit) against the fp64 oracle, through the C ABI.

Bars:
  * conv-state commits and the window indexing are bit-exact: committed rows
    are copies, and with integer inputs and weights (no activation) every fp32
    sum is exact, so outputs must equal the oracle bit for bit;
  * bf16 outputs: elementwise |y - r| <= 2^-8 |r| + 2^-16 max|r| (one bf16
    rounding, u = 2^-8, over fp32 arithmetic whose own error is ~1e-7 of the
    operands' magnitude, covered by the small absolute floor);
  * fp32 outputs: normwise max relative error 1e-5 (the all-fp32 bar).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import act_tensor

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def check_outputs(got, ref, dtype):
    got = np.asarray(got, np.float64)
    if dtype == inputs.BF16:
        bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * np.max(np.abs(ref))
        worst = float(np.max(np.abs(got - ref) - bound))
        assert worst <= 0, "bf16 conv outputs exceed the rounding bound by %.3e" % worst
        return float(np.max(np.abs(got - ref) / (np.abs(ref) + 1e-30)))
    err = float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    assert err <= 1e-5, err
    return err


def to_np(t):
    if t.dtype == torch.bfloat16:
        return inputs.bf16_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


class Draft:
    """One round of conv inputs on the GPU plus their exact values."""

    def __init__(self, x_store, x32, parent, path, length, dtype):
        self.x = act_tensor(x_store, dtype)
        self.x32 = x32
        self.parent = torch.from_numpy(np.ascontiguousarray(parent, np.int32)).cuda()
        self.parent_np = np.ascontiguousarray(parent, np.int32)
        self.path = torch.from_numpy(np.ascontiguousarray(path, np.int32)).cuda()
        self.path_np = np.ascontiguousarray(path, np.int32)
        self.length = torch.from_numpy(np.ascontiguousarray(length, np.int32)).cuda()
        self.length_np = np.ascontiguousarray(length, np.int32)


def random_draft(r, Bn, n, D, dtype, kind="tree", integer=False):
    if kind == "chain":
        par = np.tile(inputs.chain(n), (Bn, 1))
    else:
        rows = []
        for b in range(Bn):
            if b % 3 == 2:  # forests too
                rows.append(np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32))
            else:
                rows.append(inputs.random_tree(r, n, 7, 3))
        par = np.stack(rows)
    path = np.full((Bn, n), -1, np.int32)
    length = np.zeros(Bn, np.int32)
    for b in range(Bn):
        p = inputs.walk_to_root(par[b], int(r.integers(0, n)))
        if b == 1:
            p = []  # an empty accepted path
        path[b, :len(p)] = p
        length[b] = len(p)
    if integer:
        x = r.integers(-6, 7, (Bn, n, D)).astype(np.float32)
    else:
        x = r.standard_normal((Bn, n, D)).astype(np.float32)
    xs, x32 = inputs._to_dtype(x, dtype)
    return Draft(xs, x32, par, path, length, dtype)


def run_verify(C, d: Draft, w, bias, activation, pending=None, status=None):
    Bn, n, D = d.x.shape
    y = torch.empty(Bn, n, D, dtype=d.x.dtype, device="cuda")
    B.sla_conv_verify(C, d.x, w, d.parent, y, bias=bias, pending=pending, status=status, activation=activation)
    return y


@pytest.mark.parametrize("dtype", [inputs.BF16, inputs.F32])
@pytest.mark.parametrize("K", [4, 2, 1])
@pytest.mark.parametrize("activation", [True, False])
def test_conv_verify_matches_oracle(dtype, K, activation):
    """Trees, forests and a chain; D = 1032 (two full 512-channel chunks and a
    ragged 8-channel tail); 13 nodes."""
    r = np.random.default_rng(100 + K)
    Bn, n, D = 4, 13, 1032
    d = random_draft(r, Bn, n, D, dtype)
    w = r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)
    bias = r.standard_normal(D).astype(np.float32) if K != 2 else None
    C = r.standard_normal((Bn, K - 1, D)).astype(np.float32)
    say("conv verify %s K=%d act=%s" % (dtype, K, activation))
    Cg = torch.from_numpy(C).cuda() if K > 1 else None
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    y = run_verify(Cg, d, torch.from_numpy(w).cuda(), torch.from_numpy(bias).cuda() if bias is not None else None,
                   activation, status=st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    if K > 1:
        np.testing.assert_array_equal(Cg.cpu().numpy(), C)  # no pending: read only
    ref, ost = oracle.conv_verify(C if K > 1 else np.zeros((Bn, 0, D)), d.x32, w, bias, d.parent_np,
                                  activation=activation)
    assert (ost == 0).all()
    err = check_outputs(to_np(y), ref, dtype)
    say("conv verify %s K=%d act=%s: max elementwise rel err %.3e" % (dtype, K, activation, err))


@pytest.mark.parametrize("dtype", [inputs.BF16, inputs.F32])
def test_window_indexing_and_commit_bit_exact(dtype):
    """Integer inputs and weights, no activation: every fp32 sum is exact, so the
    outputs equal the oracle bit for bit (window indexing, including the
    committed rows past the root).  Then the standalone commit: bit-exact
    committed rows for every path length, including the empty path."""
    r = np.random.default_rng(110)
    Bn, n, D, K = 5, 40, 520, 4
    d = random_draft(r, Bn, n, D, dtype, integer=True)
    w = r.integers(-3, 4, (D, K)).astype(np.float32)
    bias = r.integers(-2, 3, D).astype(np.float32)
    C = r.integers(-6, 7, (Bn, K - 1, D)).astype(np.float32)
    Cg = torch.from_numpy(C).cuda()
    y = run_verify(Cg, d, torch.from_numpy(w).cuda(), torch.from_numpy(bias).cuda(), False)
    torch.cuda.synchronize()
    ref, _ = oracle.conv_verify(C, d.x32, w, bias, d.parent_np, activation=False)
    np.testing.assert_array_equal(to_np(y).astype(np.float64), ref)
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    B.sla_conv_commit(Cg, d.x, d.parent, d.path, d.length, status=st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    refC, _ = oracle.conv_commit(C, d.x32, d.parent_np, d.path_np, d.length_np)
    np.testing.assert_array_equal(Cg.cpu().numpy().astype(np.float64), refC)


@pytest.mark.parametrize("dtype", [inputs.BF16, inputs.F32])
def test_fused_pending_commit_matches_oracle_and_standalone_bitwise(dtype):
    """Round 0 verified; round 1 verified with round 0's accepted path pending
    (a differently sized previous draft).  The committed rows equal the oracle
    and the standalone commit bit for bit; round-1 outputs equal the separate
    route (commit, then verify) bit for bit and the oracle within its bar."""
    r = np.random.default_rng(120)
    Bn, D, K = 6, 1544, 4
    d0 = random_draft(r, Bn, 24, D, dtype, kind="chain")
    d0.length_np = np.array([24, 0, 2, 1, 17, 5], np.int32)
    d0.path_np = np.tile(np.arange(24, dtype=np.int32), (Bn, 1))
    for b, ln in enumerate(d0.length_np):
        d0.path_np[b, ln:] = -1
    d0.path = torch.from_numpy(d0.path_np).cuda()
    d0.length = torch.from_numpy(d0.length_np).cuda()
    d1 = random_draft(r, Bn, 16, D, dtype)
    w = torch.from_numpy(r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)).cuda()
    C = r.standard_normal((Bn, K - 1, D)).astype(np.float32)
    fused = torch.from_numpy(C).cuda()
    run_verify(fused, d0, w, None, True)
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    y1 = run_verify(fused, d1, w, None, True, pending=(d0.x, d0.parent, d0.path, d0.length), status=st)
    sep = torch.from_numpy(C).cuda()
    B.sla_conv_commit(sep, d0.x, d0.parent, d0.path, d0.length)
    y1s = run_verify(sep, d1, w, None, True)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    assert torch.equal(fused, sep)
    assert torch.equal(y1, y1s)
    refC, _ = oracle.conv_commit(C, d0.x32, d0.parent_np, d0.path_np, d0.length_np)
    np.testing.assert_array_equal(fused.cpu().numpy().astype(np.float64), refC)
    ref, _ = oracle.conv_verify(refC, d1.x32, w.cpu().numpy(), None, d1.parent_np)
    err = check_outputs(to_np(y1), ref, dtype)
    say("fused conv round %s: rel err %.3e" % (dtype, err))
    np.testing.assert_array_equal(fused.cpu().numpy()[1], C[1])  # empty path


def test_invalid_topology_and_path_set_status_and_leave_conv_state():
    r = np.random.default_rng(130)
    Bn, n, D, K = 3, 10, 512, 4
    d0 = random_draft(r, Bn, n, D, inputs.BF16)
    d1 = random_draft(r, Bn, n, D, inputs.BF16)
    w = torch.from_numpy(r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)).cuda()
    C = r.standard_normal((Bn, K - 1, D)).astype(np.float32)
    Cg = torch.from_numpy(C).cuda()
    d1.parent[0, 4] = 6  # not topological
    bad_path = d0.path.clone()
    bad_path[2, 0] = [j for j in range(n) if int(d0.parent_np[2, j]) != -1][0]  # not a root
    bad_len = d0.length.clone()
    bad_len[1] = 0
    bad_len[2] = max(1, int(bad_len[2]))
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    run_verify(Cg, d1, w, None, True, pending=(d0.x, d0.parent, bad_path, bad_len), status=st)
    # standalone commit on a copy: a length past the draft is rejected
    C2 = torch.from_numpy(C).cuda()
    st2 = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    long_len = d0.length.clone()
    long_len[1] = n + 3
    B.sla_conv_commit(C2, d0.x, d0.parent, d0.path, long_len, status=st2)
    torch.cuda.synchronize()
    s = st.cpu().numpy()
    assert s[0] == B.SLA_ERR_TOPOLOGY and s[1] == 0 and s[2] == B.SLA_ERR_PATH
    assert st2.cpu().numpy()[1] == B.SLA_ERR_PATH
    np.testing.assert_array_equal(C2.cpu().numpy()[1], C[1])
    Cn = Cg.cpu().numpy()
    np.testing.assert_array_equal(Cn[0], C[0])  # the draft's own topology was invalid
    np.testing.assert_array_equal(Cn[2], C[2])  # the pending path was invalid
    np.testing.assert_array_equal(Cn[1], C[1])  # an empty pending path commits nothing


@pytest.mark.parametrize("name,checked", [("batched_tree_serving", 64), ("large_batch_tree64", 12),
                                          ("large_batch_chain1", 64)])
def test_full_size_fused_rounds(name, checked):
    """The workloads' full shapes (D = H (2 d_k + d_v) channels), two rounds with
    the first round's accepted paths pending; sampled sequences against the
    oracle, the whole committed conv state bit-exact."""
    cfg = inputs.config(name)
    D = inputs.conv_channels(cfg)
    say("conv full size %s: generating" % name)
    r0 = inputs.draw_topology(cfg, 0)
    r1 = inputs.draw_topology(cfg, 1)
    x0, x0_32 = inputs.draw_conv_x(cfg, 0, 0)
    x1, x1_32 = inputs.draw_conv_x(cfg, 0, 1)
    w = inputs.draw_conv_weight(cfg, 0)
    C = inputs.draw_conv_state(cfg, 0)
    d0 = Draft(x0, x0_32, *r0, cfg.dtype)
    d1 = Draft(x1, x1_32, *r1, cfg.dtype)
    wg = torch.from_numpy(w).cuda()
    Cg = torch.from_numpy(C).cuda()
    say("conv full size %s: fused rounds" % name)
    y0 = run_verify(Cg, d0, wg, None, True)
    st = torch.full((cfg.batch,), 99, dtype=torch.int32, device="cuda")
    y1 = run_verify(Cg, d1, wg, None, True, pending=(d0.x, d0.parent, d0.path, d0.length), status=st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    refC, _ = oracle.conv_commit(C, x0_32, d0.parent_np, d0.path_np, d0.length_np)
    np.testing.assert_array_equal(Cg.cpu().numpy().astype(np.float64), refC)
    bs = np.random.default_rng(140).choice(cfg.batch, size=min(checked, cfg.batch), replace=False)
    bs = np.union1d(bs, [0, cfg.batch - 1])
    for y, x32, d, Cref in [(y0, x0_32, d0, C), (y1, x1_32, d1, refC)]:
        ref, _ = oracle.conv_verify(Cref[bs], x32[bs], w, None, d.parent_np[bs])
        err = check_outputs(to_np(y)[bs], ref, cfg.dtype)
        say("conv full size %s: %d sequences, max elementwise rel err %.3e" % (name, len(bs), err))


@pytest.mark.parametrize("dtype", [inputs.BF16, inputs.F32])
@pytest.mark.parametrize("K", [1, 2, 3, 4])
def test_one_node_drafts_fused_rounds(dtype, K):
    """1-node drafts (the decode step, its own single-wave kernel): two rounds,
    the first accepted or not per sequence, a ragged channel count and a bias;
    the committed conv state bit-exact, outputs within the bars; a draft whose
    only node names itself as parent is refused and leaves its state alone."""
    r = np.random.default_rng(170 + K)
    Bn, D = 5, 8 * 77
    say("conv 1-node: %s K=%d" % (dtype, K))
    d0 = random_draft(r, Bn, 1, D, dtype, kind="chain")
    d1 = random_draft(r, Bn, 1, D, dtype, kind="chain")
    d0.length_np[:] = [1, 0, 1, 1, 0]
    d0.path_np[:, 0] = [0 if a else -1 for a in d0.length_np]
    d0.length = torch.from_numpy(d0.length_np.copy()).cuda()
    d0.path = torch.from_numpy(d0.path_np.copy()).cuda()
    w = r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)
    bias = r.standard_normal(D).astype(np.float32)
    C = inputs._to_dtype(r.standard_normal((Bn, K - 1, D)), inputs.BF16)[1].astype(np.float32)
    Cg = torch.from_numpy(C).cuda() if K > 1 else None
    wg, bg = torch.from_numpy(w).cuda(), torch.from_numpy(bias).cuda()
    y0 = run_verify(Cg, d0, wg, bg, True)
    st = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    y1 = run_verify(Cg, d1, wg, bg, True, pending=(d0.x, d0.parent, d0.path, d0.length), status=st)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == 0).all()
    C0 = C if K > 1 else np.zeros((Bn, 0, D))
    refC, _ = oracle.conv_commit(C0, d0.x32, d0.parent_np, d0.path_np, d0.length_np)
    if K > 1:
        np.testing.assert_array_equal(Cg.cpu().numpy().astype(np.float64), refC)
    for y, d, Cref in [(y0, d0, C0), (y1, d1, refC)]:
        ref, _ = oracle.conv_verify(Cref, d.x32, w, bias, d.parent_np)
        check_outputs(to_np(y), ref, dtype)
    bad = torch.zeros((Bn, 1), dtype=torch.int32, device="cuda")  # node 0 names itself
    st2 = torch.full((Bn,), 99, dtype=torch.int32, device="cuda")
    before = Cg.clone() if K > 1 else None
    y2 = torch.empty_like(d1.x)
    B.sla_conv_verify(Cg, d1.x, wg, bad, y2, bias=bg, pending=(d0.x, d0.parent, d0.path, d0.length), status=st2)
    torch.cuda.synchronize()
    assert (st2.cpu().numpy() == B.SLA_ERR_TOPOLOGY).all()
    if K > 1:
        assert torch.equal(Cg, before)
