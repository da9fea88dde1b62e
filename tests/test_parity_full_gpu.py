"""GPU parity at the full benchmark sizes, in the launch configuration the
benchmark times: batched tree serving (B=64, 16 heads, dk=dv=128, 16-node
trees, 24 layers) and the large-batch shapes (B=256, 16 heads, dk=128,
dv=256; 64-node trees and the 1-node decode chain).

Two speculative rounds are run per layer: the second with the first round's
accepted paths pending (fused commit-and-verify).  Every (b, h) unit of every
checked layer is compared with the fp64 oracle: both rounds' outputs and the
committed state, as whole tensors, against the normwise bar (2e-3, bf16
q/k/v), and element by element against the same bar with the tensor's
largest magnitude as the floor.  The whole committed-state tensor is also
compared with the standalone-commit route, bitwise."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import TOL, Layer, new_factors, new_out, rel_err, verify

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def _elementwise_ok(x, ref, tol):
    """|x - r| <= tol * max|r| at every element (the normwise bar, applied to
    each element with the tensor's scale as the floor); also returns the
    worst element's error relative to its own magnitude plus that floor."""
    x = np.asarray(x, np.float64)
    scale = float(np.max(np.abs(ref)))
    d = np.abs(x - ref)
    worst = float(np.max(d / (np.abs(ref) + scale)))
    return bool(np.all(d <= tol * scale)), worst


@pytest.mark.parametrize("name,layers_checked,route", [
    ("batched_tree_serving", list(range(24)), "auto"),
    ("batched_tree_serving", [5], "serial"),
    ("large_batch_tree64", [0], "auto"),
    ("large_batch_tree64", [0], "serial"),
    ("large_batch_chain1", [0], "auto"),
    ("batched_tree_serving_f32", [0, 23], "parallel"),
    ("large_batch_tree64_f32", [0], "parallel"),
    ("large_batch_tree64_f32", [0], "auto"),
])
def test_full_size_two_rounds(name, layers_checked, route):
    cfg = inputs.config(name)
    tol = TOL[cfg.dtype]
    say("full-size %s: generating" % name)
    r0 = inputs.draw_round(cfg, 0)
    r1 = inputs.draw_round(cfg, 1)
    worst = dict(state=0.0, out0=0.0, out1=0.0, elem=0.0)
    for layer in range(cfg.layers):
        S0 = inputs.draw_state(cfg, layer)
        L0, L1 = Layer(cfg, r0, layer), Layer(cfg, r1, layer)
        f0, f1 = new_factors(cfg), new_factors(cfg)
        out0, out1 = new_out(cfg), new_out(cfg)
        state = torch.from_numpy(S0).cuda()
        st = torch.full((cfg.batch,), 99, dtype=torch.int32, device="cuda")
        say("full-size %s %s layer %d: fused rounds" % (name, route, layer))
        verify(state, L0, out0, f0, route=route)
        verify(state, L1, out1, f1, pending=(f0, L0.path, L0.length), status=st, route=route)
        torch.cuda.synchronize()
        assert (st.cpu().numpy() == 0).all()
        if layer not in layers_checked:
            continue
        # standalone route on the same inputs must agree bitwise
        sep = torch.from_numpy(S0).cuda()
        g0 = new_factors(cfg)
        verify(sep, L0, new_out(cfg), g0, route=route)
        B.sla_commit(sep, g0, L0.path, L0.length)
        torch.cuda.synchronize()
        assert torch.equal(sep, state)
        del sep, g0
        # every unit against the oracle
        say("full-size %s %s layer %d: oracle over all %d units" % (name, route, layer, cfg.batch * cfg.heads))
        ref0, s0 = oracle.verify(S0, r0.q32[layer], r0.k32[layer], r0.v32[layer], r0.alpha[layer],
                                 r0.beta[layer], r0.parent)
        S1, s1 = oracle.commit(S0, r0.k32[layer], r0.v32[layer], r0.alpha[layer], r0.beta[layer], r0.parent,
                               r0.path, r0.length)
        ref1, s2 = oracle.verify(S1, r1.q32[layer], r1.k32[layer], r1.v32[layer], r1.alpha[layer],
                                 r1.beta[layer], r1.parent)
        assert (s0 == 0).all() and (s1 == 0).all() and (s2 == 0).all()
        checks = dict(state=(state.cpu().numpy(), S1), out0=(out0.cpu().numpy(), ref0),
                      out1=(out1.cpu().numpy(), ref1))
        for key, (got, ref) in checks.items():
            e = rel_err(got, ref)
            ok, ew = _elementwise_ok(got, ref, tol)
            worst[key] = max(worst[key], e)
            worst["elem"] = max(worst["elem"], ew)
            assert ok, "%s layer %d %s: an element is off by more than %g of the tensor scale" % (
                name, layer, key, tol)
        say("full-size %s %s layer %d: state %.3e out0 %.3e out1 %.3e (normwise), worst element %.3e"
            % (name, route, layer, rel_err(*checks["state"]), rel_err(*checks["out0"]),
               rel_err(*checks["out1"]), worst["elem"]))
        del ref0, ref1, S1, checks
    assert max(worst["state"], worst["out0"], worst["out1"]) <= tol, worst
