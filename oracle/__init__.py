"""fp64 CPU oracle for GDN speculative verification and accepted-path commit.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the package smoke check
and by the benchmark's CPU-baseline leg.  It shares no code with the HIP
library and never calls it.  All arithmetic lives in ``oracle.c``; this file
only converts numpy arrays to fp64/int32 and passes pointers.

Parity status of every function is pinned by ``tests/test_oracle.py``; see
the function docstrings for the passage each follows (SpecLA, arXiv
2607.16673).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK = 0
ERR_SHAPE = -2
ERR_TOPOLOGY = -4
ERR_PATH = -5

# Layer families (the factor-record remark closing §5.1); see oracle.c.
GDN = 0
DELTANET = 1
DECAY = 2
GLA = 3
FAMILIES = {"gdn": GDN, "deltanet": DELTANET, "decay": DECAY, "gla": GLA}

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_up = ctypes.POINTER(ctypes.c_uint64)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b  # noqa: F401  (plain gcc build of oracle.c)
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_gdn_step.argtypes = [ctypes.c_int, ctypes.c_int, _dp, _dp, _dp,
                                    ctypes.c_double, ctypes.c_double, _dp]
    lib.oracle_readout.argtypes = [ctypes.c_int, ctypes.c_int, _dp, _dp, _dp]
    lib.oracle_check_parent.argtypes = [_ip, ctypes.c_int]
    lib.oracle_check_parent.restype = ctypes.c_int
    lib.oracle_root_path.argtypes = [_ip, ctypes.c_int, ctypes.c_int, _ip]
    lib.oracle_root_path.restype = ctypes.c_int
    lib.oracle_topology.argtypes = [_ip, ctypes.c_int, _ip, _up, _ip, _ip, _ip]
    lib.oracle_topology.restype = ctypes.c_int
    lib.oracle_validate_path.argtypes = [_ip, ctypes.c_int, _ip, ctypes.c_int]
    lib.oracle_validate_path.restype = ctypes.c_int
    lib.oracle_verify.argtypes = [ctypes.c_int] * 5 + [_dp] * 6 + [_ip, _dp, _ip]
    lib.oracle_verify.restype = ctypes.c_int
    lib.oracle_commit.argtypes = [ctypes.c_int] * 5 + [_dp] * 5 + [_ip, _ip, ctypes.c_int, _ip, _ip]
    lib.oracle_commit.restype = ctypes.c_int
    lib.oracle_layer_step.argtypes = [ctypes.c_int] * 3 + [_dp] * 4 + [ctypes.c_double, _dp]
    lib.oracle_verify_family.argtypes = [ctypes.c_int] * 6 + [_dp] * 6 + [_ip, _dp, _ip]
    lib.oracle_verify_family.restype = ctypes.c_int
    lib.oracle_commit_family.argtypes = [ctypes.c_int] * 6 + [_dp] * 5 + [_ip, _ip, ctypes.c_int, _ip, _ip]
    lib.oracle_commit_family.restype = ctypes.c_int
    lib.oracle_conv_verify.argtypes = [ctypes.c_int] * 4 + [_dp] * 4 + [ctypes.c_int, _ip, _dp, _ip]
    lib.oracle_conv_verify.restype = ctypes.c_int
    lib.oracle_conv_commit.argtypes = [ctypes.c_int] * 4 + [_dp, _dp, _ip, _ip, ctypes.c_int, _ip, _ip]
    lib.oracle_conv_commit.restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _i32(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _p(a, t):
    return a.ctypes.data_as(t)


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use (OMP_NUM_THREADS or all cores)."""
    return _load().oracle_num_threads()


def set_num_threads(n: int) -> None:
    """Threads for the following calls (timing only; results are identical
    for any count)."""
    _load().oracle_set_num_threads(int(n))


def gdn_step(Hs, k, v, alpha, beta):
    """One GDN step on the transposed state H = S^T ([dk][dv]); returns a copy.

    S' = alpha S (I - beta k k^T) + beta v k^T (gated delta rule; the plain
    form is Eq. (state-update), §2.2)."""
    lib = _load()
    H = _f64(Hs).copy()
    dk, dv = H.shape
    k = _f64(k)
    v = _f64(v)
    scratch = np.zeros(dv)
    lib.oracle_gdn_step(dk, dv, _p(H, _dp), _p(k, _dp), _p(v, _dp), float(alpha),
                        float(beta), _p(scratch, _dp))
    return H


def _family(f):
    return FAMILIES[f] if isinstance(f, str) else int(f)


def layer_step(Hs, k, v, gate, beta, family=GDN):
    """One step of a layer family on H = S^T ([dk][dv]); returns a copy.

    gate: alpha (GDN, DECAY), the dk per-key gates (GLA), unused (DELTANET);
    beta: unused for DECAY and GLA."""
    lib = _load()
    fam = _family(family)
    H = _f64(Hs).copy()
    dk, dv = H.shape
    k = _f64(k)
    v = _f64(v)
    g = _f64(np.reshape(gate if gate is not None else 0.0, (-1,)))
    scratch = np.zeros(dv)
    lib.oracle_layer_step(fam, dk, dv, _p(H, _dp), _p(k, _dp), _p(v, _dp), _p(g, _dp),
                          float(beta if beta is not None else 0.0), _p(scratch, _dp))
    return H


def readout(Hs, q):
    """o = H^T q = S q for one head."""
    lib = _load()
    H = _f64(Hs)
    dk, dv = H.shape
    q = _f64(q)
    o = np.zeros(dv)
    lib.oracle_readout(dk, dv, _p(H, _dp), _p(q, _dp), _p(o, _dp))
    return o


def check_parent(parent) -> int:
    """OK when parent[j] is -1 or an earlier node (topological order, §4.2)."""
    p = _i32(parent)
    return _load().oracle_check_parent(_p(p, _ip), len(p))


def root_path(parent, j):
    """Root path P(j), root first, j last."""
    p = _i32(parent)
    out = np.zeros(len(p), np.int32)
    ln = _load().oracle_root_path(_p(p, _ip), len(p), int(j), _p(out, _ip))
    if ln < 0:
        raise ValueError("invalid parent array")
    return out[:ln].copy()


def topology(parent):
    """Topology table of one draft (tree mask of §4.2, parent array of §7).

    Returns dict(status, depth, anc, order, n_children, max_depth)."""
    p = _i32(parent)
    n = len(p)
    depth = np.zeros(n, np.int32)
    anc = np.zeros(n, np.uint64)
    order = np.zeros(n, np.int32)
    nch = np.zeros(n, np.int32)
    md = np.zeros(1, np.int32)
    st = _load().oracle_topology(_p(p, _ip), n, _p(depth, _ip), _p(anc, _up), _p(order, _ip),
                                 _p(nch, _ip), _p(md, _ip))
    return dict(status=st, depth=depth, anc=anc, order=order, n_children=nch,
                max_depth=int(md[0]))


def validate_path(parent, path, length) -> int:
    """OK when path[0..length) is a root path of the draft."""
    p = _i32(parent)
    pa = _i32(path) if len(path) else np.zeros(1, np.int32)
    return _load().oracle_validate_path(_p(p, _ip), len(p), _p(pa, _ip), int(length))


def _gates(family, alpha, beta, B, n, H, dk):
    """fp64 gate and beta arrays (None where the family does not read them)."""
    if family == DELTANET:
        g = None
    else:
        g = _f64(alpha)
        want = (B, n, H, dk) if family == GLA else (B, n, H)
        assert g.shape == want, (g.shape, want)
    if family in (DECAY, GLA):
        bt = None
    else:
        bt = _f64(beta)
        assert bt.shape == (B, n, H)
    return g, bt


def _opt(a):
    return _p(a, _dp) if a is not None else None


def verify(state, q, k, v, alpha, beta, parent, family=GDN):
    """Per-node outputs by definition (§4; tree mask §4.2).

    state [B][H][dk][dv]; q,k [B][n][H][dk]; v [B][n][H][dv]; parent [B][n].
    alpha: [B][n][H] (GDN, DECAY), [B][n][H][dk] per-key gates (GLA), or None
    (DELTANET); beta: [B][n][H] (GDN, DELTANET) or None (DECAY, GLA).
    Returns (out [B][n][H][dv] fp64, status [B])."""
    lib = _load()
    fam = _family(family)
    S = _f64(state)
    B, H, dk, dv = S.shape
    q, k, v = _f64(q), _f64(k), _f64(v)
    n = q.shape[1]
    g, bt = _gates(fam, alpha, beta, B, n, H, dk)
    par = _i32(parent).reshape(B, n)
    assert q.shape == (B, n, H, dk) and k.shape == (B, n, H, dk) and v.shape == (B, n, H, dv)
    out = np.zeros((B, n, H, dv))
    status = np.zeros(B, np.int32)
    lib.oracle_verify_family(fam, B, H, dk, dv, n, _p(S, _dp), _p(q, _dp), _p(k, _dp), _p(v, _dp),
                             _opt(g), _opt(bt), _p(par, _ip), _p(out, _dp), _p(status, _ip))
    return out, status


def commit(state, k, v, alpha, beta, parent, path, length, family=GDN):
    """Committed state after decoding the accepted tokens one by one (§5.1-5.2).

    path [B][stride] (-1 padded), length [B]; alpha and beta as for verify.
    Returns (state', status)."""
    lib = _load()
    fam = _family(family)
    S = _f64(state).copy()
    B, H, dk, dv = S.shape
    k, v = _f64(k), _f64(v)
    n = k.shape[1]
    g, bt = _gates(fam, alpha, beta, B, n, H, dk)
    par = _i32(parent).reshape(B, n)
    pa = _i32(path).reshape(B, -1)
    if pa.shape[1] == 0:
        pa = np.full((B, 1), -1, np.int32)
    ln = _i32(length).reshape(B)
    status = np.zeros(B, np.int32)
    lib.oracle_commit_family(fam, B, H, dk, dv, n, _p(S, _dp), _p(k, _dp), _p(v, _dp), _opt(g),
                             _opt(bt), _p(par, _ip), _p(pa, _ip), pa.shape[1], _p(ln, _ip),
                             _p(status, _ip))
    return S, status


def conv_verify(conv_state, x, w, bias, parent, activation=True):
    """Per-node outputs of the short causal convolution by definition.

    Node j's window is the last K inputs of [conv_state rows, x along P(j)]
    (the GDN layer's depthwise convolution, §7; tree mask of §4.2).
    conv_state [B][K-1][D]; x [B][n][D]; w [D][K]; bias [D] or None; parent
    [B][n].  Returns (y [B][n][D] fp64, status [B])."""
    lib = _load()
    x = _f64(x)
    B, n, D = x.shape
    w = _f64(w)
    K = w.shape[1]
    C = _f64(conv_state).reshape(B, K - 1, D) if K > 1 else np.zeros((B, 1, D))
    bias_p = _p(_f64(bias), _dp) if bias is not None else None
    par = _i32(parent).reshape(B, n)
    y = np.zeros((B, n, D))
    status = np.zeros(B, np.int32)
    lib.oracle_conv_verify(B, D, K, n, _p(C, _dp), _p(x, _dp), _p(w, _dp), bias_p, int(bool(activation)),
                           _p(par, _ip), _p(y, _dp), _p(status, _ip))
    return y, status


def conv_commit(conv_state, x, parent, path, length):
    """Conv state after decoding the accepted tokens one by one (§5.1-5.2):
    each token drops the oldest row and appends its input.

    conv_state [B][K-1][D]; x [B][n][D]; path [B][stride] (-1 padded);
    length [B].  Returns (conv_state', status)."""
    lib = _load()
    x = _f64(x)
    B, n, D = x.shape
    C = _f64(conv_state).copy()
    K = C.shape[1] + 1
    Cp = C if K > 1 else np.zeros((B, 1, D))
    par = _i32(parent).reshape(B, n)
    pa = _i32(path).reshape(B, -1)
    if pa.shape[1] == 0:
        pa = np.full((B, 1), -1, np.int32)
    ln = _i32(length).reshape(B)
    status = np.zeros(B, np.int32)
    lib.oracle_conv_commit(B, D, K, n, _p(Cp, _dp), _p(x, _dp), _p(par, _ip), _p(pa, _ip), pa.shape[1],
                           _p(ln, _ip), _p(status, _ip))
    return (Cp if K > 1 else C), status
