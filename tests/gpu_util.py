"""Helpers shared by the GPU parity tests: move generated inputs to the GPU,
run the library through the binding, run the oracle on the same values, and
measure normwise relative error (max |x - r| / max |r| over a tensor)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

TOL = {inputs.F32: 1e-5, inputs.BF16: 2e-3}


def act_tensor(x, dtype, device="cuda"):
    """Storage array from the generator -> torch tensor on the GPU."""
    if dtype == inputs.BF16:
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def torch_act_dtype(dtype):
    return torch.bfloat16 if dtype == inputs.BF16 else torch.float32


def rel_err(x, ref):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(x - ref)) / max(float(np.max(np.abs(ref))), 1e-300))


class Layer:
    """Device tensors of one layer of one round."""

    def __init__(self, cfg, rnd: inputs.Round, layer_pos: int, device="cuda"):
        self.cfg = cfg
        dt = cfg.dtype
        self.q = act_tensor(rnd.q[layer_pos], dt, device)
        self.k = act_tensor(rnd.k[layer_pos], dt, device)
        self.v = act_tensor(rnd.v[layer_pos], dt, device)
        self.alpha = torch.from_numpy(rnd.alpha[layer_pos]).to(device)
        self.beta = torch.from_numpy(rnd.beta[layer_pos]).to(device)
        self.parent = torch.from_numpy(rnd.parent).to(device)
        self.path = torch.from_numpy(rnd.path).to(device)
        self.length = torch.from_numpy(rnd.length).to(device)


def new_factors(cfg, batch=None, device="cuda"):
    Bn = cfg.batch if batch is None else batch
    return B.Factors.empty(Bn, cfg.n_nodes, cfg.heads, cfg.d_k, cfg.d_v, torch_act_dtype(cfg.dtype), device)


def new_out(cfg, batch=None, device="cuda"):
    Bn = cfg.batch if batch is None else batch
    return torch.empty(Bn, cfg.n_nodes, cfg.heads, cfg.d_v, dtype=torch.float32, device=device)


def verify(state, L: Layer, out, factors, *, pending=None, status=None, route="auto"):
    topo = "chain" if L.cfg.chain else "tree"
    B.sla_verify(state, L.q, L.k, L.v, L.alpha, L.beta, L.parent, out, factors, pending=pending,
                 status=status, topology=topo, route=route)


def oracle_verify_units(state_np, rnd: inputs.Round, layer_pos, units):
    """Oracle outputs for a list of (b, h) units: dict (b, h) -> [n][dv]."""
    res = {}
    for b, h in units:
        out, st = oracle.verify(state_np[b:b + 1, h:h + 1], rnd.q32[layer_pos][b:b + 1, :, h:h + 1],
                                rnd.k32[layer_pos][b:b + 1, :, h:h + 1],
                                rnd.v32[layer_pos][b:b + 1, :, h:h + 1],
                                rnd.alpha[layer_pos][b:b + 1, :, h:h + 1],
                                rnd.beta[layer_pos][b:b + 1, :, h:h + 1], rnd.parent[b:b + 1])
        assert st[0] == 0
        res[(b, h)] = out[0, :, 0]
    return res


def oracle_commit_units(state_np, rnd: inputs.Round, layer_pos, units):
    """Oracle committed states for (b, h) units along rnd.path: (b, h) -> [dk][dv]."""
    res = {}
    for b, h in units:
        S, st = oracle.commit(state_np[b:b + 1, h:h + 1], rnd.k32[layer_pos][b:b + 1, :, h:h + 1],
                              rnd.v32[layer_pos][b:b + 1, :, h:h + 1],
                              rnd.alpha[layer_pos][b:b + 1, :, h:h + 1],
                              rnd.beta[layer_pos][b:b + 1, :, h:h + 1], rnd.parent[b:b + 1],
                              rnd.path[b:b + 1], rnd.length[b:b + 1])
        assert st[0] == 0
        res[(b, h)] = S[0, 0]
    return res


def sample_units(cfg, count, seed, batch=None):
    Bn = cfg.batch if batch is None else batch
    r = np.random.default_rng(seed)
    allu = [(b, h) for b in range(Bn) for h in range(cfg.heads)]
    if len(allu) <= count:
        return allu
    idx = r.choice(len(allu), size=count, replace=False)
    # always include the corners (first and last unit)
    units = {allu[0], allu[-1]} | {allu[i] for i in idx}
    return sorted(units)


def parallel_supported(dk, dv, n, dtype):
    """Whether an explicit PARALLEL request for a GDN draft of this shape is
    accepted: a shape outside the route, or a draft whose on-chip stage does
    not fit, is refused with SLA_ERR_UNSUPPORTED before any launch."""
    try:
        z = torch.zeros
        dt = torch.bfloat16 if dtype == inputs.BF16 else torch.float32
        q = z(1, n, 1, dk, dtype=dt, device="cuda")
        v = z(1, n, 1, dv, dtype=dt, device="cuda")
        par = torch.arange(-1, n - 1, dtype=torch.int32, device="cuda")[None]
        B.sla_verify(z(1, 1, dk, dv, device="cuda"), q, q, v, z(1, n, 1, device="cuda"),
                     z(1, n, 1, device="cuda"), par, z(1, n, 1, dv, device="cuda"),
                     B.Factors.empty(1, n, 1, dk, dv, dt), route="parallel")
        torch.cuda.synchronize()
        return True
    except B.SlaError as e:
        if e.code == B.SLA_ERR_UNSUPPORTED:
            return False
        raise
