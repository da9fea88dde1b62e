"""The paper's tree-verification study as schedules over the library's calls
(Table tab:eval-tree-shape-avg of §8.3; routes of §4.1-4.3).

Proposal trees: a beam top-k rollout of `depth` levels (the drafter's
configured depth; every level expands the k best frontier nodes by path
score, each with its k most likely tokens) pruned by the library's own
draft pruning to the `n` best-scoring nodes (an ancestor-closed set, §6.1)
and packed into the verifier's parent array (§7).  The first level's k
candidates are children of the committed state, so a tree may have up to k
roots.  Synthetic rollouts stand in for the recorded EAGLE proposals of the
paper's runtime, which are not available.

Routes, all from the committed state with no pending commit:
  * r2l       root-to-leaf replay: one chain verification per root-to-leaf
              path, launched one after another (each shared prefix is
              verified once per leaf below it);
  * serial    the state-resident serial route (§4.1) over the whole tree;
  * parallel  the tree-masked factorised route (§4.2);
  * hybrid    the chain-decomposed hybrid route (§4.3).
A node's R2L output is the one its last root-to-leaf path produced; in
exact arithmetic every path through it gives the same value.

Marshalling and scheduling only: every step runs in the library's kernels.
"""
from __future__ import annotations

import numpy as np

from . import binding as B
from . import inputs

# (top-k, configured depth, nodes): the proposal shapes of the paper's table
TREE_SHAPES = [(2, 12, 16), (2, 24, 32), (4, 4, 16), (4, 4, 32), (4, 12, 16), (4, 24, 32)]
ROUTES = ["r2l", "serial", "parallel", "hybrid"]


def proposal_tree(rng: np.random.Generator, k: int, depth: int, n: int, max_candidates: int = 1024):
    """Parent array [n] of one synthetic proposal tree: a top-k rollout of
    `depth` levels pruned (no score margin, budget n) and packed."""
    cand = k + (depth - 1) * k * k
    par, logp = inputs.rollout(rng, min(cand, max_candidates), k, max_depth=depth)
    if len(par) < n:
        raise ValueError("rollout (k=%d, depth=%d) has %d candidates, fewer than %d" % (k, depth, len(par), n))
    res = B.sla_prune_host(par, logp, tau=np.inf, budget=n)
    if res["status"] != B.SLA_OK or res["count"] != n:
        raise RuntimeError("pruning failed: %s" % res)
    return res["packed_parent"][:n].astype(np.int32)


def root_to_leaf_paths(parent):
    parent = np.asarray(parent)
    n = len(parent)
    leaves = [j for j in range(n) if not (parent == j).any()]
    return [inputs.walk_to_root(parent, j) for j in leaves]


class Draft:
    """One tree's device tensors at batch 1: q, k, v in the activation dtype,
    gates and betas fp32, the committed state, and per-route outputs and
    factor stores."""

    def __init__(self, torch, dev, parent, H, dk, dv, seed, dtype="bf16"):
        self.torch, self.dev = torch, dev
        self.parent_np = np.asarray(parent, np.int32)
        n = len(parent)
        self.n, self.H, self.dk, self.dv, self.dtype = n, H, dk, dv, dtype
        cfg = inputs.Config("study", 800 + seed % 100, 1, H, dk, dv, n, False, n, n,
                            inputs.BF16 if dtype == "bf16" else inputs.F32, 1)
        rnd = inputs.draw_layer(cfg, seed, 0)
        self.host = rnd
        self.state_np = inputs.draw_state(cfg, seed)
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

        def act(x):
            if dtype == "bf16":
                return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)
            return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

        self.q, self.k, self.v = act(rnd["q"]), act(rnd["k"]), act(rnd["v"])
        self.alpha = torch.from_numpy(rnd["alpha"]).to(dev)
        self.beta = torch.from_numpy(rnd["beta"]).to(dev)
        self.parent = torch.from_numpy(self.parent_np[None]).to(dev)
        self.state = torch.from_numpy(self.state_np).to(dev)
        self.tdt = tdt
        self.out = {r: torch.empty(1, n, H, dv, dtype=torch.float32, device=dev) for r in ROUTES}
        self.fac = {r: B.Factors.empty(1, n, H, dk, dv, tdt, dev) for r in ROUTES if r != "r2l"}
        # root-to-leaf replay: the rows of each path gathered ahead of time
        self.chains = []
        for pth in root_to_leaf_paths(self.parent_np):
            ix = torch.tensor(pth, dtype=torch.long, device=dev)
            L = len(pth)
            self.chains.append(dict(
                q=self.q[:, ix].contiguous(), k=self.k[:, ix].contiguous(), v=self.v[:, ix].contiguous(),
                a=self.alpha[:, ix].contiguous(), b=self.beta[:, ix].contiguous(),
                p=torch.arange(-1, L - 1, dtype=torch.int32, device=dev)[None],
                o=torch.empty(1, L, H, dv, dtype=torch.float32, device=dev),
                f=B.Factors.empty(1, L, H, dk, dv, tdt, dev), nodes=pth))

    def launch(self, route):
        """Enqueue one verification of the tree by `route` (no host sync)."""
        if route == "r2l":
            for c in self.chains:
                B.sla_verify(self.state, c["q"], c["k"], c["v"], c["a"], c["b"], c["p"], c["o"], c["f"],
                             topology="chain", route="serial")
            return
        B.sla_verify(self.state, self.q, self.k, self.v, self.alpha, self.beta, self.parent, self.out[route],
                     self.fac[route], route=route)

    def outputs(self, route):
        """Host outputs [n][H][dv] of a route (R2L: scattered from its chains)."""
        if route != "r2l":
            return self.out[route].cpu().numpy()[0]
        o = np.zeros((self.n, self.H, self.dv), np.float32)
        for c in self.chains:
            o[c["nodes"]] = c["o"].cpu().numpy()[0]
        return o
