"""Out-of-range write detection on the GPU: every buffer a call touches --
inputs, outputs, states, factor stores, pending paths, statuses -- is carved
out of a larger allocation whose guard bands on both sides hold a sentinel
bit pattern.  Verification (every route, the decode step, two rounds with a
pending commit), the standalone commit, the short convolution and its
commit, pruning and the mask converter run at ragged shapes; afterwards
every guard band must be bit-identical, and so must every read-only input."""
import numpy as np
import pytest
import torch

from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import parallel_supported

pytestmark = pytest.mark.gpu

GUARD_BYTES = 1 << 16  # on each side; a multiple of 16 keeps the interior aligned


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


class Guarded:
    """Buffers inside guard bands; all of one allocation's bytes start as
    the sentinel, the interior is then filled with the given contents."""

    def __init__(self):
        self.bufs = []

    def make(self, shape, dtype, contents=None, readonly=False):
        esz = torch.empty(0, dtype=dtype).element_size()
        n = int(np.prod(shape)) if len(shape) else 1
        g = GUARD_BYTES // esz
        raw = torch.empty(n * esz + 2 * GUARD_BYTES, dtype=torch.uint8, device="cuda")
        pat = torch.tensor([0xA5, 0x5A, 0xC3, 0x3C], dtype=torch.uint8).repeat((raw.numel() + 3) // 4)
        raw.copy_(pat[:raw.numel()].cuda())
        t = raw.view(dtype)[g:g + n].view(*shape)
        if contents is not None:
            t.copy_(contents)
        self.bufs.append((raw, raw.clone(), n * esz, readonly))
        return t

    def check(self, what):
        torch.cuda.synchronize()
        for i, (raw, ref, nbytes, ro) in enumerate(self.bufs):
            lo, hi = GUARD_BYTES, GUARD_BYTES + nbytes
            assert torch.equal(raw[:lo], ref[:lo]), "%s: buffer %d written below its start" % (what, i)
            assert torch.equal(raw[hi:], ref[hi:]), "%s: buffer %d written past its end" % (what, i)
            if ro:
                assert torch.equal(raw[lo:hi], ref[lo:hi]), "%s: read-only buffer %d was written" % (what, i)


def _act(x, dt):
    if dt == inputs.BF16:
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))


SHAPES = [  # B, H, dk, dv, n
    (3, 5, 64, 80, 17),
    (2, 3, 128, 144, 33),
    (2, 2, 256, 48, 5),
    (4, 3, 128, 16, 64),
    (3, 2, 128, 80, 1),
]


@pytest.mark.parametrize("dt", [inputs.BF16, inputs.F32])
@pytest.mark.parametrize("fam", ["gdn", "gla"])
@pytest.mark.parametrize("route", ["auto", "serial", "parallel", "hybrid"])
@pytest.mark.parametrize("shape", SHAPES, ids=["B%d_H%d_dk%d_dv%d_n%d" % s for s in SHAPES])
def test_verify_and_commit_stay_in_bounds(shape, route, fam, dt):
    Bn, H, dk, dv, n = shape
    tdt = torch.bfloat16 if dt == inputs.BF16 else torch.float32
    if route == "parallel" and fam == "gla" and dk == 256 and n > 32:
        pytest.skip("GLA's parallel stage holds at most 32 nodes at d_k = 256")
    if route == "parallel" and not parallel_supported(dk, dv, n, dt):
        pytest.skip("the draft's on-chip stage does not fit the parallel route")
    cfg = inputs.Config("canary", 900 + dk + n, Bn, H, dk, dv, n, False, min(n, 6), 4, dt, 1)
    r = np.random.default_rng(Bn * 1000 + dk + n)
    G = Guarded()
    rounds = []
    for ri in range(2):
        rnd = inputs.draw_round(cfg, ri, layers=[0])
        rnd.parent = np.stack([inputs.random_tree(r, n, min(n, 6), 4) if n > 1 else np.array([-1], np.int32)
                               for _ in range(Bn)]).astype(np.int32)
        rnd.path = np.full((Bn, n), -1, np.int32)
        rnd.length = np.zeros(Bn, np.int32)
        for b in range(Bn):
            p = inputs.walk_to_root(rnd.parent[b], int(r.integers(0, n)))
            rnd.path[b, :len(p)] = p
            rnd.length[b] = len(p)
        a, bt = inputs.family_gates(cfg, rnd, 0, fam, layer=0, round_index=ri)
        rounds.append(dict(
            q=G.make((Bn, n, H, dk), tdt, _act(rnd.q[0], dt), True),
            k=G.make((Bn, n, H, dk), tdt, _act(rnd.k[0], dt), True),
            v=G.make((Bn, n, H, dv), tdt, _act(rnd.v[0], dt), True),
            a=G.make(a.shape, torch.float32, torch.from_numpy(a), True),
            b=G.make(bt.shape, torch.float32, torch.from_numpy(bt), True) if bt is not None else None,
            parent=G.make((Bn, n), torch.int32, torch.from_numpy(rnd.parent), True),
            path=G.make((Bn, n), torch.int32, torch.from_numpy(rnd.path), True),
            length=G.make((Bn,), torch.int32, torch.from_numpy(rnd.length), True),
            out=G.make((Bn, n, H, dv), torch.float32),
            f=B.Factors(G.make((Bn, n, H, dk), tdt), G.make((Bn, n, H, dv), torch.float32),
                        G.make(inputs_gate_shape(Bn, n, H, dk, fam), torch.float32), G.make((Bn, n), torch.int32))))
    state = G.make((Bn, H, dk, dv), torch.float32, torch.from_numpy(inputs.draw_state(cfg, 0)))
    status = G.make((Bn,), torch.int32)
    say("canary verify %s route=%s fam=%s dtype=%s" % (shape, route, fam, dt))
    R0, R1 = rounds
    B.sla_verify(state, R0["q"], R0["k"], R0["v"], R0["a"], R0["b"], R0["parent"], R0["out"], R0["f"],
                 status=status, route=route, family=fam)
    G.check("verify")
    B.sla_verify(state, R1["q"], R1["k"], R1["v"], R1["a"], R1["b"], R1["parent"], R1["out"], R1["f"],
                 pending=(R0["f"], R0["path"], R0["length"]), status=status, route=route, family=fam)
    G.check("fused verify")
    assert (status.cpu().numpy() == 0).all()
    B.sla_commit(state, R1["f"], R1["path"], R1["length"], status=status, family=fam)
    G.check("commit")
    assert (status.cpu().numpy() == 0).all()


def inputs_gate_shape(Bn, n, H, dk, fam):
    return B.gate_shape(Bn, n, H, dk, fam)


@pytest.mark.parametrize("n,D,Bn", [(17, 8 * 37, 3), (1, 520, 2), (64, 2056, 2), (5, 1024, 5)])
def test_conv_stays_in_bounds(n, D, Bn):
    r = np.random.default_rng(n * 7 + D)
    K = 4
    G = Guarded()

    def draft():
        par = np.stack([inputs.random_tree(r, n, min(n, 6), 4) if n > 1 else np.array([-1], np.int32)
                        for _ in range(Bn)]).astype(np.int32)
        path = np.full((Bn, n), -1, np.int32)
        ln = np.zeros(Bn, np.int32)
        for b in range(Bn):
            p = inputs.walk_to_root(par[b], int(r.integers(0, n)))
            path[b, :len(p)] = p
            ln[b] = len(p)
        x = inputs.bf16_bits(r.standard_normal((Bn, n, D)).astype(np.float32))
        return dict(x=G.make((Bn, n, D), torch.bfloat16, _act(x, inputs.BF16), True),
                    parent=G.make((Bn, n), torch.int32, torch.from_numpy(par), True),
                    path=G.make((Bn, n), torch.int32, torch.from_numpy(path), True),
                    length=G.make((Bn,), torch.int32, torch.from_numpy(ln), True),
                    y=G.make((Bn, n, D), torch.bfloat16))

    d0, d1 = draft(), draft()
    w = G.make((D, K), torch.float32, torch.from_numpy(r.uniform(-0.5, 0.5, (D, K)).astype(np.float32)), True)
    bias = G.make((D,), torch.float32, torch.from_numpy(r.standard_normal(D).astype(np.float32)), True)
    C = G.make((Bn, K - 1, D), torch.float32, torch.from_numpy(r.standard_normal((Bn, K - 1, D)).astype(np.float32)))
    st = G.make((Bn,), torch.int32)
    say("canary conv n=%d D=%d B=%d" % (n, D, Bn))
    B.sla_conv_verify(C, d0["x"], w, d0["parent"], d0["y"], bias=bias, status=st)
    B.sla_conv_verify(C, d1["x"], w, d1["parent"], d1["y"], bias=bias, status=st,
                      pending=(d0["x"], d0["parent"], d0["path"], d0["length"]))
    B.sla_conv_commit(C, d1["x"], d1["parent"], d1["path"], d1["length"], status=st)
    G.check("conv")
    assert (st.cpu().numpy() == 0).all()


def test_prune_and_mask_stay_in_bounds():
    cfg = inputs.config("large_batch_tree64")
    for n_cand in [64, 37, 5]:
        par_np, lp_np = inputs.draw_rollouts(cfg, 0, batch=7, n_cand=n_cand)
        G = Guarded()
        par = G.make(par_np.shape, torch.int32, torch.from_numpy(par_np), True)
        lp = G.make(lp_np.shape, torch.float32, torch.from_numpy(lp_np), True)
        Bn, n = par_np.shape
        pp, im = G.make((Bn, n), torch.int32), G.make((Bn, n), torch.int32)
        cnt, st, sc = G.make((Bn,), torch.int32), G.make((Bn,), torch.int32), G.make((Bn, n), torch.float32)
        say("canary prune n=%d" % n)
        code = B.lib().sla_prune(par.data_ptr(), lp.data_ptr(), Bn, n, 3.0, max(1, n // 3), pp.data_ptr(),
                                 im.data_ptr(), cnt.data_ptr(), sc.data_ptr(), st.data_ptr(),
                                 torch.cuda.current_stream().cuda_stream)
        assert code == 0
        G.check("prune")
        masks = np.zeros((Bn, n), np.uint64)
        for b in range(Bn):
            masks[b] = B.sla_topology_host(par_np[b])["anc"]
        mk = G.make((Bn, n), torch.int64, torch.from_numpy(masks.view(np.int64)), True)
        out, st2 = G.make((Bn, n), torch.int32), G.make((Bn,), torch.int32)
        code = B.lib().sla_tree_mask_to_parent(mk.data_ptr(), Bn, n, out.data_ptr(), st2.data_ptr(),
                                               torch.cuda.current_stream().cuda_stream)
        assert code == 0
        G.check("mask")
        np.testing.assert_array_equal(out.cpu().numpy(), par_np)
