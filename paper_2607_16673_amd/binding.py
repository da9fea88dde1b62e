"""Thin ctypes binding of libsla (C ABI in include/sla.h).

Argument marshalling only: torch tensors are checked for device, dtype,
shape and contiguity, turned into raw device pointers plus the current HIP
stream, and passed to the library.  Every step of the verification and
commit runs in the library's HIP kernels; there is no fallback of any kind.
If ``libsla.so`` has not been built, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsla.so")

SLA_OK = 0
SLA_ERR_NULL = -1
SLA_ERR_SHAPE = -2
SLA_ERR_DTYPE = -3
SLA_ERR_TOPOLOGY = -4
SLA_ERR_PATH = -5
SLA_ERR_ALIAS = -6
SLA_ERR_UNSUPPORTED = -7
SLA_ERR_HIP = -8
SLA_ERR_SCORE = -9

SLA_DTYPE_F32 = 0
SLA_DTYPE_BF16 = 1
SLA_TOPO_TREE = 0
SLA_TOPO_CHAIN = 1
SLA_ROUTE_AUTO = 0
SLA_ROUTE_SERIAL = 1
SLA_ROUTE_PARALLEL = 2
SLA_ROUTE_HYBRID = 3
SLA_MAX_NODES = 64
SLA_FAMILY_GDN = 0
SLA_FAMILY_DELTANET = 1
SLA_FAMILY_DECAY = 2
SLA_FAMILY_GLA = 3
FAMILIES = {"gdn": SLA_FAMILY_GDN, "deltanet": SLA_FAMILY_DELTANET, "decay": SLA_FAMILY_DECAY,
            "gla": SLA_FAMILY_GLA}
SLA_ACT_NONE = 0
SLA_ACT_SILU = 1
SLA_CONV_MAX_KERNEL = 4

ROUTES = {"auto": SLA_ROUTE_AUTO, "serial": SLA_ROUTE_SERIAL, "parallel": SLA_ROUTE_PARALLEL,
          "hybrid": SLA_ROUTE_HYBRID}
TOPOLOGIES = {"tree": SLA_TOPO_TREE, "chain": SLA_TOPO_CHAIN}


class SlaShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("d_k", ctypes.c_int32),
                ("d_v", ctypes.c_int32), ("n_nodes", ctypes.c_int32), ("qkv_dtype", ctypes.c_int32),
                ("topology", ctypes.c_int32), ("family", ctypes.c_int32), ("route", ctypes.c_int32)]


class SlaFactors(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("u", ctypes.c_void_p), ("alpha", ctypes.c_void_p),
                ("parent", ctypes.c_void_p)]


class SlaPending(ctypes.Structure):
    _fields_ = [("f", SlaFactors), ("n_nodes", ctypes.c_int32), ("path", ctypes.c_void_p),
                ("len", ctypes.c_void_p)]


class SlaConvShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("channels", ctypes.c_int32), ("kernel_size", ctypes.c_int32),
                ("n_nodes", ctypes.c_int32), ("x_dtype", ctypes.c_int32), ("activation", ctypes.c_int32)]


class SlaConvPending(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("parent", ctypes.c_void_p), ("n_nodes", ctypes.c_int32),
                ("path", ctypes.c_void_p), ("len", ctypes.c_void_p)]


class SlaError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        self.code = code
        super().__init__("%s: %s (%d)" % (what or "libsla", status_string(code), code))


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libsla.so is not built (run `python -m paper_2607_16673_amd.build`)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        L.sla_verify.argtypes = [ctypes.POINTER(SlaShape), vp, ctypes.POINTER(SlaPending),
                                 vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(SlaFactors), vp, vp]
        L.sla_verify.restype = ctypes.c_int
        L.sla_commit.argtypes = [ctypes.POINTER(SlaShape), vp, ctypes.POINTER(SlaFactors), vp, vp, vp, vp]
        L.sla_commit.restype = ctypes.c_int
        L.sla_topology.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp, vp]
        L.sla_topology.restype = ctypes.c_int
        L.sla_topology_host.argtypes = [vp, i32, vp, vp, vp, vp, vp]
        L.sla_topology_host.restype = ctypes.c_int
        L.sla_validate_path_host.argtypes = [vp, i32, vp, i32]
        L.sla_validate_path_host.restype = ctypes.c_int
        L.sla_factors_bytes.argtypes = [ctypes.POINTER(SlaShape)]
        L.sla_factors_bytes.restype = ctypes.c_size_t
        L.sla_status_string.argtypes = [ctypes.c_int]
        L.sla_status_string.restype = ctypes.c_char_p
        L.sla_version.restype = ctypes.c_int
        L.sla_conv_verify.argtypes = [ctypes.POINTER(SlaConvShape), vp, ctypes.POINTER(SlaConvPending),
                                      vp, vp, vp, vp, vp, vp, vp]
        L.sla_conv_verify.restype = ctypes.c_int
        L.sla_conv_commit.argtypes = [ctypes.POINTER(SlaConvShape), vp, vp, vp, vp, vp, vp, vp]
        L.sla_conv_commit.restype = ctypes.c_int
        L.sla_prune.argtypes = [vp, vp, i32, i32, ctypes.c_float, i32, vp, vp, vp, vp, vp, vp]
        L.sla_prune.restype = ctypes.c_int
        L.sla_prune_host.argtypes = [vp, vp, i32, ctypes.c_float, i32, vp, vp, vp, vp]
        L.sla_prune_host.restype = ctypes.c_int
        L.sla_tree_mask_to_parent.argtypes = [vp, i32, i32, vp, vp, vp]
        L.sla_tree_mask_to_parent.restype = ctypes.c_int
        L.sla_tree_mask_to_parent_host.argtypes = [vp, i32, vp]
        L.sla_tree_mask_to_parent_host.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().sla_status_string(int(code)).decode()


def sla_version() -> int:
    return lib().sla_version()


# ------------------------------------------------------------- host helpers
def sla_topology_host(parent) -> dict:
    p = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    n = len(p)
    depth = np.zeros(max(n, 1), np.int32)
    anc = np.zeros(max(n, 1), np.uint64)
    order = np.zeros(max(n, 1), np.int32)
    kids = np.zeros(max(n, 1), np.int32)
    md = np.zeros(1, np.int32)
    st = lib().sla_topology_host(p.ctypes.data, n, depth.ctypes.data, anc.ctypes.data,
                                 order.ctypes.data, kids.ctypes.data, md.ctypes.data)
    return dict(status=st, depth=depth[:n], anc=anc[:n], order=order[:n], n_children=kids[:n],
                max_depth=int(md[0]))


def sla_validate_path_host(parent, path, length) -> int:
    p = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    pa = np.ascontiguousarray(np.asarray(path, dtype=np.int32)) if len(path) else np.zeros(1, np.int32)
    return lib().sla_validate_path_host(p.ctypes.data, len(p), pa.ctypes.data, int(length))


def make_shape(batch, heads, d_k, d_v, n_nodes, dtype="bf16", topology="tree", family="gdn",
               route="auto") -> SlaShape:
    return SlaShape(int(batch), int(heads), int(d_k), int(d_v), int(n_nodes),
                    SLA_DTYPE_BF16 if dtype == "bf16" else SLA_DTYPE_F32, TOPOLOGIES[topology],
                    FAMILIES[family], ROUTES[route] if isinstance(route, str) else int(route))


def gate_shape(batch, n, heads, d_k, family="gdn") -> tuple:
    """Shape of the gate input and of the gate factor record for a family."""
    return (batch, n, heads, d_k) if family == "gla" else (batch, n, heads)


def sla_factors_bytes(shape: SlaShape) -> int:
    return int(lib().sla_factors_bytes(ctypes.byref(shape)))


# ------------------------------------------------------------- device calls
def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return SLA_DTYPE_BF16
    if t.dtype == torch.float32:
        return SLA_DTYPE_F32
    raise TypeError("q/k/v must be bfloat16 or float32, got %s" % t.dtype)


def _dev(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must live on the GPU" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(_torch().cuda.current_stream(device).cuda_stream)


@dataclass
class Factors:
    """A factor store (see sla_factors in include/sla.h) as torch tensors."""
    k: object       # [B][n][H][dk] activation dtype
    u: object       # [B][n][H][dv] fp32
    alpha: object   # [B][n][H] fp32 gate ([B][n][H][dk] for GLA)
    parent: object  # [B][n] int32

    @staticmethod
    def empty(batch, n, heads, d_k, d_v, dtype, device="cuda", family="gdn"):
        torch = _torch()
        return Factors(torch.empty(batch, n, heads, d_k, dtype=dtype, device=device),
                       torch.empty(batch, n, heads, d_v, dtype=torch.float32, device=device),
                       torch.empty(gate_shape(batch, n, heads, d_k, family), dtype=torch.float32, device=device),
                       torch.empty(batch, n, dtype=torch.int32, device=device))

    def c(self, dtype, B, n, H, dk, dv, family="gdn") -> SlaFactors:
        torch = _torch()
        return SlaFactors(_dev(self.k, dtype, (B, n, H, dk), "factors.k"),
                          _dev(self.u, torch.float32, (B, n, H, dv), "factors.u"),
                          _dev(self.alpha, torch.float32, gate_shape(B, n, H, dk, family), "factors.alpha"),
                          _dev(self.parent, torch.int32, (B, n), "factors.parent"))


def _check(code, what):
    if code != SLA_OK:
        raise SlaError(code, what)


def sla_verify(state, q, k, v, alpha, beta, parent_idx, out, factors: Factors, *,
               pending: Optional[tuple] = None, status=None, topology: str = "tree",
               route: str = "auto", family: str = "gdn"):
    """Enqueue one verification on the current stream (see sla_verify in sla.h).

    alpha: [B][n][H] fp32 ([B][n][H][dk] per-key gates for "gla"; None for
    "deltanet"); beta: [B][n][H] fp32 (None for "decay" and "gla").
    pending: None or (factors_prev: Factors, path [B][n_prev] int32, len [B] int32).
    Raises SlaError on a host-detected error."""
    torch = _torch()
    B, n, H, dk = q.shape
    dv = v.shape[-1]
    dt = _dtype_code(q)
    shape = SlaShape(B, H, dk, dv, n, dt, TOPOLOGIES[topology], FAMILIES[family], ROUTES[route])
    f = factors.c(q.dtype, B, n, H, dk, dv, family)
    pend_p = None
    if pending is not None:
        pf, ppath, plen = pending
        pn = pf.parent.shape[1]
        pend = SlaPending(pf.c(q.dtype, B, pn, H, dk, dv, family), pn,
                          _dev(ppath, torch.int32, (B, pn), "pending.path"),
                          _dev(plen, torch.int32, (B,), "pending.len"))
        pend_p = ctypes.byref(pend)
    st_p = _dev(status, torch.int32, (B,), "status") if status is not None else None
    code = lib().sla_verify(
        ctypes.byref(shape), _dev(state, torch.float32, (B, H, dk, dv), "state"), pend_p,
        _dev(q, q.dtype, (B, n, H, dk), "q"), _dev(k, q.dtype, (B, n, H, dk), "k"),
        _dev(v, q.dtype, (B, n, H, dv), "v"),
        _dev(alpha, torch.float32, gate_shape(B, n, H, dk, family), "alpha") if alpha is not None else None,
        _dev(beta, torch.float32, (B, n, H), "beta") if beta is not None else None,
        _dev(parent_idx, torch.int32, (B, n), "parent_idx"),
        _dev(out, torch.float32, (B, n, H, dv), "out"), ctypes.byref(f), st_p, _stream(q.device))
    _check(code, "sla_verify")


def sla_commit(state, factors: Factors, path, length, *, status=None, family: str = "gdn"):
    """Enqueue an immediate commit of the accepted paths (see sla_commit)."""
    torch = _torch()
    B, n, H, dk = factors.k.shape
    dv = factors.u.shape[-1]
    shape = SlaShape(B, H, dk, dv, n, _dtype_code(factors.k), SLA_TOPO_TREE, FAMILIES[family], SLA_ROUTE_AUTO)
    f = factors.c(factors.k.dtype, B, n, H, dk, dv, family)
    st_p = _dev(status, torch.int32, (B,), "status") if status is not None else None
    code = lib().sla_commit(ctypes.byref(shape), _dev(state, torch.float32, (B, H, dk, dv), "state"),
                            ctypes.byref(f), _dev(path, torch.int32, (B, n), "path"),
                            _dev(length, torch.int32, (B,), "len"), st_p, _stream(state.device))
    _check(code, "sla_commit")


def sla_topology(parent_idx):
    """Device topology table (see sla_topology); returns tensors on the GPU."""
    torch = _torch()
    B, n = parent_idx.shape
    dev = parent_idx.device
    depth = torch.empty(B, n, dtype=torch.int32, device=dev)
    anc = torch.empty(B, n, dtype=torch.int64, device=dev)
    order = torch.empty(B, n, dtype=torch.int32, device=dev)
    kids = torch.empty(B, n, dtype=torch.int32, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    code = lib().sla_topology(_dev(parent_idx, torch.int32, (B, n), "parent_idx"), B, n,
                              _dev(depth, None, None, "depth"), _dev(anc, None, None, "anc"),
                              _dev(order, None, None, "order"), _dev(kids, None, None, "n_children"),
                              _dev(status, None, None, "status"), _stream(dev))
    _check(code, "sla_topology")
    return dict(depth=depth, anc=anc, order=order, n_children=kids, status=status)


# ------------------------------------------------- short causal convolution
def make_conv_shape(batch, channels, kernel_size, n_nodes, dtype="bf16", activation=True) -> SlaConvShape:
    return SlaConvShape(int(batch), int(channels), int(kernel_size), int(n_nodes),
                        SLA_DTYPE_BF16 if dtype == "bf16" else SLA_DTYPE_F32,
                        SLA_ACT_SILU if activation else SLA_ACT_NONE)


def sla_conv_verify(conv_state, x, weight, parent_idx, y, *, bias=None, pending: Optional[tuple] = None,
                    status=None, activation: bool = True):
    """Enqueue the draft's short causal convolution on the current stream
    (see sla_conv_verify in sla.h).

    conv_state [B][K-1][D] fp32 (None when K = 1); x, y [B][n][D]; weight
    [D][K] fp32; bias [D] fp32 or None; parent_idx [B][n] int32.
    pending: None or (x_prev [B][n_prev][D], parent_prev [B][n_prev], path
    [B][n_prev] int32, len [B] int32).  Raises SlaError on a host-detected error."""
    torch = _torch()
    B, n, D = x.shape
    K = weight.shape[1]
    shape = make_conv_shape(B, D, K, n, "bf16" if x.dtype == torch.bfloat16 else "f32", activation)
    _dtype_code(x)
    cs = _dev(conv_state, torch.float32, (B, K - 1, D), "conv_state") if conv_state is not None else None
    pend_p = None
    if pending is not None:
        px, ppar, ppath, plen = pending
        pn = ppar.shape[1]
        pend = SlaConvPending(_dev(px, x.dtype, (B, pn, D), "pending.x"),
                              _dev(ppar, torch.int32, (B, pn), "pending.parent"), pn,
                              _dev(ppath, torch.int32, (B, pn), "pending.path"),
                              _dev(plen, torch.int32, (B,), "pending.len"))
        pend_p = ctypes.byref(pend)
    bias_p = _dev(bias, torch.float32, (D,), "bias") if bias is not None else None
    st_p = _dev(status, torch.int32, (B,), "status") if status is not None else None
    code = lib().sla_conv_verify(ctypes.byref(shape), cs, pend_p, _dev(x, x.dtype, (B, n, D), "x"),
                                 _dev(weight, torch.float32, (D, K), "weight"), bias_p,
                                 _dev(parent_idx, torch.int32, (B, n), "parent_idx"),
                                 _dev(y, x.dtype, (B, n, D), "y"), st_p, _stream(x.device))
    _check(code, "sla_conv_verify")


def sla_conv_commit(conv_state, x, parent_idx, path, length, *, kernel_size=None, status=None):
    """Enqueue an immediate conv-state commit of the accepted paths (see
    sla_conv_commit).  conv_state [B][K-1][D] fp32 (None when K = 1)."""
    torch = _torch()
    B, n, D = x.shape
    K = kernel_size if kernel_size is not None else conv_state.shape[1] + 1
    shape = make_conv_shape(B, D, K, n, "bf16" if x.dtype == torch.bfloat16 else "f32")
    _dtype_code(x)
    cs = _dev(conv_state, torch.float32, (B, K - 1, D), "conv_state") if conv_state is not None else None
    st_p = _dev(status, torch.int32, (B,), "status") if status is not None else None
    code = lib().sla_conv_commit(ctypes.byref(shape), cs, _dev(x, x.dtype, (B, n, D), "x"),
                                 _dev(parent_idx, torch.int32, (B, n), "parent_idx"),
                                 _dev(path, torch.int32, (B, n), "path"),
                                 _dev(length, torch.int32, (B,), "len"), st_p, _stream(x.device))
    _check(code, "sla_conv_commit")


# ------------------------------------------------- draft pruning and packing
def sla_prune_host(parent, logp, tau: float, budget: int = 0) -> dict:
    """Prune and pack one draft on the CPU (see sla_prune_host in sla.h).
    Returns dict(status, count, packed_parent, index_map, scores)."""
    p = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    lp = np.ascontiguousarray(np.asarray(logp, dtype=np.float32))
    n = len(p)
    pp = np.zeros(max(n, 1), np.int32)
    im = np.zeros(max(n, 1), np.int32)
    sc = np.zeros(max(n, 1), np.float32)
    cnt = np.zeros(1, np.int32)
    st = lib().sla_prune_host(p.ctypes.data, lp.ctypes.data, n, float(tau), int(budget), pp.ctypes.data,
                              im.ctypes.data, cnt.ctypes.data, sc.ctypes.data)
    return dict(status=st, count=int(cnt[0]), packed_parent=pp[:n], index_map=im[:n], scores=sc[:n])


def sla_prune(parent, logp, tau: float, budget: int = 0, *, with_scores: bool = False):
    """Enqueue batched pruning and packing on the current stream (see
    sla_prune).  parent [B][n] int32, logp [B][n] fp32 (device tensors).
    Returns dict of device tensors: packed_parent, index_map, count, status
    (and scores)."""
    torch = _torch()
    B, n = parent.shape
    dev = parent.device
    pp = torch.empty(B, n, dtype=torch.int32, device=dev)
    im = torch.empty(B, n, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, dtype=torch.int32, device=dev)
    st = torch.empty(B, dtype=torch.int32, device=dev)
    sc = torch.empty(B, n, dtype=torch.float32, device=dev) if with_scores else None
    code = lib().sla_prune(_dev(parent, torch.int32, (B, n), "parent"), _dev(logp, torch.float32, (B, n), "logp"),
                           B, n, float(tau), int(budget), _dev(pp, None, None, "packed_parent"),
                           _dev(im, None, None, "index_map"), _dev(cnt, None, None, "count"),
                           _dev(sc, None, None, "scores") if sc is not None else None,
                           _dev(st, None, None, "status"), _stream(dev))
    _check(code, "sla_prune")
    out = dict(packed_parent=pp, index_map=im, count=cnt, status=st)
    if sc is not None:
        out["scores"] = sc
    return out


def sla_tree_mask_to_parent_host(mask_rows):
    """(status, parent) from one tree mask given as uint64 row bit sets."""
    m = np.ascontiguousarray(np.asarray(mask_rows, dtype=np.uint64))
    n = len(m)
    out = np.zeros(max(n, 1), np.int32)
    st = lib().sla_tree_mask_to_parent_host(m.ctypes.data, n, out.ctypes.data)
    return st, out[:n]


def sla_tree_mask_to_parent(mask_rows):
    """Batched device converter: mask_rows [B][n] int64 (uint64 bit sets).
    Returns (parent [B][n] int32, status [B] int32) device tensors."""
    torch = _torch()
    B, n = mask_rows.shape
    dev = mask_rows.device
    par = torch.full((B, n), -2, dtype=torch.int32, device=dev)
    st = torch.empty(B, dtype=torch.int32, device=dev)
    code = lib().sla_tree_mask_to_parent(_dev(mask_rows, torch.int64, (B, n), "mask"), B, n,
                                         _dev(par, None, None, "parent"), _dev(st, None, None, "status"),
                                         _stream(dev))
    _check(code, "sla_tree_mask_to_parent")
    return par, st
