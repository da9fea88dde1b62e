"""HIP graph replay of the fused rounds the benchmark times: a graph holding
two consecutive speculative rounds (verify with the previous round's accepted
paths pending, factor stores ping-ponged; the recurrent core and the short
convolution) is replayed several times, with eager work and synchronisations
in between, and every replay's states, outputs and factors are compared bit
for bit with the same rounds run eagerly from the same starting states."""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

from gpu_util import Layer, new_factors, new_out

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("dt", [inputs.BF16, inputs.F32])
def test_graph_replays_match_eager_rounds(dt):
    """dt: the recurrent core's q/k/v (bf16: the bf16 matrix-core contraction;
    fp32: the fp32 one); the convolution runs on bf16 rows in both."""
    cfg = inputs.Config("graph", 120, 8, 4, 128, 128, 16, False, 5, 3, dt, 1)
    ccfg = dataclasses.replace(cfg, dtype=inputs.BF16)
    rnd = inputs.draw_round(cfg, 0, layers=[0])
    L = Layer(cfg, rnd, 0)
    S0 = inputs.draw_state(cfg, 0)
    xa = [inputs.draw_conv_x(ccfg, 0, r)[0] for r in range(2)]
    to_bf = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()
    xs = [to_bf(x) for x in xa]
    w = torch.from_numpy(inputs.draw_conv_weight(ccfg, 0)).cuda()
    C0 = torch.from_numpy(inputs.draw_conv_state(ccfg, 0)).cuda()

    def make():
        return dict(S=torch.from_numpy(S0).cuda(), C=C0.clone(), f=[new_factors(cfg), new_factors(cfg)],
                    o=new_out(cfg), y=torch.empty_like(xs[0]))

    def rounds(st, first):
        # two rounds: round s verifies into store s % 2 with store (s+1) % 2 pending
        for s in range(2):
            pend = None if (first and s == 0) else (st["f"][(s + 1) % 2], L.path, L.length)
            B.sla_verify(st["S"], L.q, L.k, L.v, L.alpha, L.beta, L.parent, st["o"], st["f"][s % 2], pending=pend)
            cp = None if (first and s == 0) else (xs[(s + 1) % 2], L.parent, L.path, L.length)
            B.sla_conv_verify(st["C"], xs[s % 2], w, L.parent, st["y"], pending=cp)

    eager, graph = make(), make()
    rounds(eager, True)
    rounds(graph, True)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    sc = torch.cuda.Stream()
    sc.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(sc):
        with torch.cuda.graph(g, stream=sc):
            rounds(graph, False)
    torch.cuda.synchronize()
    # capture does not run the work: both are still after the first two rounds
    assert torch.equal(eager["S"], graph["S"])
    for rep in range(4):
        g.replay()
        rounds(eager, False)
        torch.cuda.synchronize()
        _ = torch.zeros(1024, device="cuda").sum().item()  # unrelated eager work between replays
        for key in ["S", "C", "o", "y"]:
            assert torch.equal(eager[key], graph[key]), (rep, key)
        for s in range(2):
            assert torch.equal(eager["f"][s].u, graph["f"][s].u), (rep, s)
            assert torch.equal(eager["f"][s].k, graph["f"][s].k), (rep, s)
        say("graph replay %d matches the eager rounds (%s q/k/v)" % (rep, dt))
