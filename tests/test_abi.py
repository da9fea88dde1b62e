"""CPU tests of the C ABI: the library loads and exports every declared
symbol, the host topology helpers are bit-exact with the oracle's builder,
and every host-detectable argument error returns its code before any launch
(no GPU is touched by these tests)."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_16673_amd import binding as B
from paper_2607_16673_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sla.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sla_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = B.lib()
    syms = declared_symbols()
    assert {"sla_verify", "sla_commit", "sla_topology", "sla_topology_host",
            "sla_validate_path_host", "sla_factors_bytes", "sla_status_string",
            "sla_version", "sla_conv_verify", "sla_conv_commit"} <= set(syms)
    for s in syms:
        assert hasattr(L, s), s


def test_status_codes_match_header():
    text = open(HEADER).read()
    for name, val in re.findall(r"#define (SLA_\w+) \(?(-?\d+)\)?", text):
        if hasattr(B, name):
            assert getattr(B, name) == int(val), name
    for code in range(-8, 1):
        assert B.status_string(code) not in ("", "unknown status")
    assert B.status_string(-99) == "unknown status"
    assert B.sla_version() >= 10000


def _same_table(parent):
    o = oracle.topology(parent)
    h = B.sla_topology_host(parent)
    assert h["status"] == o["status"]
    if o["status"] == 0:
        for key in ("depth", "anc", "order", "n_children"):
            np.testing.assert_array_equal(h[key], o[key], err_msg=key)
        assert h["max_depth"] == o["max_depth"]


def test_host_topology_bit_exact_exhaustive_small():
    for n in range(1, 7):
        for par in itertools.product(*[range(-1, j) for j in range(n)]):
            _same_table(np.array(par, np.int32))


def test_host_topology_bit_exact_random_and_configs():
    r = np.random.default_rng(30)
    for n in [7, 16, 31, 32, 63, 64]:
        for _ in range(25):
            _same_table(inputs.random_tree(r, n, 64, 8))
            _same_table(np.array([int(r.integers(-1, j)) if j else -1 for j in range(n)], np.int32))
    for name in ["tree32_bf16", "batched_tree_serving", "large_batch_tree64"]:
        cfg = inputs.config(name)
        parent, _, _ = inputs.draw_topology(cfg, 0, batch=min(cfg.batch, 16))
        for row in parent:
            _same_table(row)


def test_host_topology_rejects_invalid():
    for bad in ([-1, 1], [-1, 0, 2], [-2], [0], [-1, 0, 5, 1]):
        assert B.sla_topology_host(np.array(bad, np.int32))["status"] == B.SLA_ERR_TOPOLOGY
    assert B.sla_topology_host(np.full(65, -1, np.int32))["status"] == B.SLA_ERR_SHAPE


def test_host_path_validation_matches_oracle():
    r = np.random.default_rng(31)
    for _ in range(30):
        parent = inputs.random_tree(r, 24, 7, 3)
        for j in range(24):
            p = inputs.walk_to_root(parent, j)
            assert B.sla_validate_path_host(parent, p, len(p)) == 0 == oracle.validate_path(parent, p, len(p))
            cand = list(r.integers(-1, 24, size=len(p)))
            assert (B.sla_validate_path_host(parent, cand, len(cand)) == 0) == \
                   (oracle.validate_path(parent, cand, len(cand)) == 0)
    assert B.sla_validate_path_host([-1, 0], [], 0) == 0
    assert B.sla_validate_path_host([-1, 0], [0, 1], 3) == B.SLA_ERR_PATH
    assert B.sla_validate_path_host([-1, 5], [0], 1) == B.SLA_ERR_TOPOLOGY


def test_factor_store_bytes():
    s = B.make_shape(64, 16, 128, 128, 16, "bf16")
    bnh = 64 * 16 * 16
    assert B.sla_factors_bytes(s) == bnh * 128 * 2 + bnh * 128 * 4 + bnh * 4 + 64 * 16 * 4
    s = B.make_shape(1, 8, 256, 256, 8, "f32")
    assert B.sla_factors_bytes(s) == 8 * 8 * (256 * 4 + 256 * 4 + 4) + 8 * 4
    assert B.sla_factors_bytes(B.make_shape(1, 1, 64, 64, 0)) == 0


# ------------------------------------------ argument errors (no launch happens)
FAKE = 1 << 20  # never dereferenced: every call below fails host-side checks


def _ptr(i=0):
    return ctypes.c_void_p(FAKE + i * (1 << 24))


def _verify(shape, route=0, pending=None, nulls=(), factors=None):
    args = [_ptr(i) for i in range(9)]
    for i in nulls:
        args[i] = None
    f = factors or B.SlaFactors(_ptr(10), _ptr(11), _ptr(12), _ptr(13))
    if shape is not None:
        shape.route = route
    return B.lib().sla_verify(ctypes.byref(shape) if shape is not None else None, args[0],
                              ctypes.byref(pending) if pending is not None else None,
                              args[1], args[2], args[3], args[4], args[5], args[6], args[7],
                              ctypes.byref(f), None, None)


def test_verify_argument_errors_return_before_launch():
    ok = B.make_shape(2, 4, 128, 128, 8, "bf16")
    assert _verify(None) == B.SLA_ERR_NULL
    for i in range(8):
        assert _verify(ok, nulls=(i,)) == B.SLA_ERR_NULL, i
    assert _verify(ok, factors=B.SlaFactors(None, _ptr(11), _ptr(12), _ptr(13))) == B.SLA_ERR_NULL
    bad = [B.make_shape(0, 4, 128, 128, 8), B.make_shape(2, 0, 128, 128, 8),
           B.make_shape(2, 4, 128, 128, 0), B.make_shape(2, 4, 128, 128, 65),
           B.make_shape(2, 4, 128, 100, 8), B.make_shape(2, 4, 128, 8, 8),
           B.make_shape(2, 4, 0, 128, 8)]
    for s in bad:
        assert _verify(s) == B.SLA_ERR_SHAPE
    s = B.make_shape(2, 4, 128, 128, 8)
    s.qkv_dtype = 7
    assert _verify(s) == B.SLA_ERR_DTYPE
    s = B.make_shape(2, 4, 128, 128, 8)
    s.topology = 3
    assert _verify(s) == B.SLA_ERR_SHAPE
    assert _verify(B.make_shape(2, 4, 96, 128, 8)) == B.SLA_ERR_UNSUPPORTED
    # a sequence's rows must stay addressable with 32-bit offsets
    assert _verify(B.make_shape(1, 2048, 128, 4096, 8)) == B.SLA_ERR_SHAPE
    assert _verify(ok, route=9) == B.SLA_ERR_SHAPE


def test_verify_rejects_pending_aliasing_output_factors():
    ok = B.make_shape(2, 4, 128, 128, 8, "bf16")
    out_f = B.SlaFactors(_ptr(10), _ptr(11), _ptr(12), _ptr(13))
    # pending u overlaps the output u store
    pend = B.SlaPending(B.SlaFactors(_ptr(20), ctypes.c_void_p(FAKE + 11 * (1 << 24) + 4096), _ptr(22),
                                     _ptr(23)), 8, _ptr(24), _ptr(25))
    assert _verify(ok, pending=pend, factors=out_f) == B.SLA_ERR_ALIAS
    same = B.SlaPending(out_f, 8, _ptr(24), _ptr(25))
    assert _verify(ok, pending=same, factors=out_f) == B.SLA_ERR_ALIAS
    incomplete = B.SlaPending(B.SlaFactors(_ptr(20), None, _ptr(22), _ptr(23)), 8, _ptr(24), _ptr(25))
    assert _verify(ok, pending=incomplete) == B.SLA_ERR_NULL
    badn = B.SlaPending(B.SlaFactors(_ptr(20), _ptr(21), _ptr(22), _ptr(23)), 0, _ptr(24), _ptr(25))
    assert _verify(ok, pending=badn) == B.SLA_ERR_SHAPE
    # misaligned state pointer
    args = [ctypes.c_void_p(FAKE + 4)] + [_ptr(i) for i in range(1, 9)]
    f = B.SlaFactors(_ptr(10), _ptr(11), _ptr(12), _ptr(13))
    ok.route = 0
    assert B.lib().sla_verify(ctypes.byref(ok), args[0], None, *args[1:8], ctypes.byref(f),
                              None, None) == B.SLA_ERR_UNSUPPORTED


def test_family_argument_rules_return_before_launch():
    """Each family requires exactly the inputs its step reads.  A call whose
    pointers pass the null checks is stopped by a misaligned state pointer, so
    nothing is launched."""
    L = B.lib()
    f = B.SlaFactors(_ptr(10), _ptr(11), _ptr(12), _ptr(13))

    def call(family, alpha, beta, state=None, route=0, shape=None):
        s = shape or B.make_shape(2, 4, 128, 128, 8, "bf16", family=family)
        s.route = route
        args = [state or _ptr(0)] + [_ptr(i) for i in range(1, 9)]
        args[4], args[5] = alpha, beta
        return L.sla_verify(ctypes.byref(s), args[0], None, *args[1:8], ctypes.byref(f), None, None)

    mis = ctypes.c_void_p(FAKE + 4)
    # DeltaNet: beta required, alpha not read
    assert call("deltanet", _ptr(4), None) == B.SLA_ERR_NULL
    assert call("deltanet", None, _ptr(5), state=mis) == B.SLA_ERR_UNSUPPORTED
    # no-delta families: alpha (gates) required, beta not read
    for fam in ("decay", "gla"):
        assert call(fam, None, _ptr(5)) == B.SLA_ERR_NULL
        assert call(fam, _ptr(4), None, state=mis) == B.SLA_ERR_UNSUPPORTED
    assert call("gdn", None, _ptr(5)) == B.SLA_ERR_NULL
    assert call("gdn", _ptr(4), None) == B.SLA_ERR_NULL
    # the parallel route's on-chip stage: a draft that does not fit (64 nodes
    # of fp32 keys at d_k = 256) is refused before any launch; fp32
    # activations otherwise pass its host checks (stopped here by the
    # misaligned state pointer)
    big = B.make_shape(2, 4, 256, 64, 64, "f32", family="gdn")
    assert call("gdn", _ptr(4), _ptr(5), route=B.SLA_ROUTE_PARALLEL, shape=big) == B.SLA_ERR_UNSUPPORTED
    s32 = B.make_shape(2, 4, 128, 128, 8, "f32", family="gla")
    assert call("gla", _ptr(4), None, state=mis, route=B.SLA_ROUTE_PARALLEL, shape=s32) == B.SLA_ERR_UNSUPPORTED
    assert call("gla", ctypes.c_void_p(FAKE + 4 * (1 << 24) + 4), None) == B.SLA_ERR_UNSUPPORTED  # gates misaligned
    bad = B.make_shape(2, 4, 128, 128, 8, "bf16")
    bad.family = 4
    assert call("gdn", _ptr(4), _ptr(5), shape=bad) == B.SLA_ERR_SHAPE
    assert L.sla_commit(ctypes.byref(bad), _ptr(0), ctypes.byref(f), _ptr(1), _ptr(2), None, None) == B.SLA_ERR_SHAPE


def test_factor_store_bytes_per_family():
    bnh = 2 * 8 * 4
    base = bnh * 128 * 2 + bnh * 64 * 4 + 2 * 8 * 4
    for fam in ("gdn", "deltanet", "decay"):
        assert B.sla_factors_bytes(B.make_shape(2, 4, 128, 64, 8, "bf16", family=fam)) == base + bnh * 4
    assert B.sla_factors_bytes(B.make_shape(2, 4, 128, 64, 8, "bf16", family="gla")) == base + bnh * 128 * 4


def test_commit_and_topology_argument_errors():
    L = B.lib()
    ok = B.make_shape(2, 4, 128, 128, 8, "bf16")
    f = B.SlaFactors(_ptr(10), _ptr(11), _ptr(12), _ptr(13))
    assert L.sla_commit(None, _ptr(0), ctypes.byref(f), _ptr(1), _ptr(2), None, None) == B.SLA_ERR_NULL
    assert L.sla_commit(ctypes.byref(ok), None, ctypes.byref(f), _ptr(1), _ptr(2), None, None) == B.SLA_ERR_NULL
    assert L.sla_commit(ctypes.byref(ok), _ptr(0), ctypes.byref(f), None, _ptr(2), None, None) == B.SLA_ERR_NULL
    assert L.sla_commit(ctypes.byref(ok), _ptr(0), ctypes.byref(f), _ptr(1), None, None, None) == B.SLA_ERR_NULL
    bad = B.make_shape(2, 4, 128, 128, 70)
    assert L.sla_commit(ctypes.byref(bad), _ptr(0), ctypes.byref(f), _ptr(1), _ptr(2), None, None) == B.SLA_ERR_SHAPE
    assert L.sla_topology(None, 1, 4, _ptr(1), _ptr(2), _ptr(3), _ptr(4), _ptr(5), None) == B.SLA_ERR_NULL
    assert L.sla_topology(_ptr(0), 0, 4, _ptr(1), _ptr(2), _ptr(3), _ptr(4), _ptr(5), None) == B.SLA_ERR_SHAPE
    assert L.sla_topology(_ptr(0), 1, 65, _ptr(1), _ptr(2), _ptr(3), _ptr(4), _ptr(5), None) == B.SLA_ERR_SHAPE


def test_binding_refuses_host_tensors():
    import torch
    x = torch.zeros(1, 4, 1, 64)
    with pytest.raises((ValueError, TypeError)):
        B.sla_verify(torch.zeros(1, 1, 64, 64), x, x, x, torch.zeros(1, 4, 1), torch.zeros(1, 4, 1),
                     torch.zeros(1, 4, dtype=torch.int32), torch.zeros(1, 4, 1, 64),
                     B.Factors(x, x, torch.zeros(1, 4, 1), torch.zeros(1, 4, dtype=torch.int32)))


def _conv_verify(shape, pending=None, nulls=(), cs=None, x=None, y=None):
    args = [_ptr(i) for i in range(6)]
    for i in nulls:
        args[i] = None
    return B.lib().sla_conv_verify(ctypes.byref(shape) if shape is not None else None,
                                   cs if cs is not None else args[0],
                                   ctypes.byref(pending) if pending is not None else None,
                                   x if x is not None else args[1], args[2], args[3], args[4],
                                   y if y is not None else args[5], None, None)


def test_conv_argument_errors_return_before_launch():
    L = B.lib()
    ok = B.make_conv_shape(4, 6144, 4, 16)
    assert _conv_verify(None) == B.SLA_ERR_NULL
    for i in [0, 1, 2, 4, 5]:  # conv_state, x, weight, parent, y (bias may be NULL)
        assert _conv_verify(ok, nulls=(i,)) == B.SLA_ERR_NULL, i
    # with K = 1 there is no conv state, so a NULL one is fine (fails later on alignment)
    k1 = B.make_conv_shape(4, 6144, 1, 16)
    assert _conv_verify(k1, nulls=(0,), x=ctypes.c_void_p(FAKE + 8)) == B.SLA_ERR_UNSUPPORTED
    for s in [B.make_conv_shape(0, 64, 4, 16), B.make_conv_shape(4, 60, 4, 16), B.make_conv_shape(4, 0, 4, 16),
              B.make_conv_shape(4, 64, 0, 16), B.make_conv_shape(4, 64, 5, 16), B.make_conv_shape(4, 64, 4, 0),
              B.make_conv_shape(4, 64, 4, 65), B.make_conv_shape(4, (1 << 20) + 8, 4, 16)]:
        assert _conv_verify(s) == B.SLA_ERR_SHAPE
    s = B.make_conv_shape(4, 64, 4, 16)
    s.x_dtype = 5
    assert _conv_verify(s) == B.SLA_ERR_DTYPE
    s = B.make_conv_shape(4, 64, 4, 16)
    s.activation = 2
    assert _conv_verify(s) == B.SLA_ERR_SHAPE
    # pending rows overlapping the outputs, incomplete or mis-sized pending
    y = _ptr(5)
    alias = B.SlaConvPending(ctypes.c_void_p(FAKE + 5 * (1 << 24) + 1024), _ptr(7), 16, _ptr(8), _ptr(9))
    assert _conv_verify(ok, pending=alias, y=y) == B.SLA_ERR_ALIAS
    assert _conv_verify(ok, pending=B.SlaConvPending(_ptr(6), None, 16, _ptr(8), _ptr(9))) == B.SLA_ERR_NULL
    assert _conv_verify(ok, pending=B.SlaConvPending(_ptr(6), _ptr(7), 0, _ptr(8), _ptr(9))) == B.SLA_ERR_SHAPE
    assert _conv_verify(ok, x=ctypes.c_void_p(FAKE + 8)) == B.SLA_ERR_UNSUPPORTED
    # standalone commit
    c = L.sla_conv_commit
    assert c(None, _ptr(0), _ptr(1), _ptr(2), _ptr(3), _ptr(4), None, None) == B.SLA_ERR_NULL
    for i in range(5):
        args = [_ptr(j) for j in range(5)]
        args[i] = None
        assert c(ctypes.byref(ok), *args, None, None) == B.SLA_ERR_NULL, i
    assert c(ctypes.byref(B.make_conv_shape(4, 64, 4, 70)), *[_ptr(j) for j in range(5)], None, None) == \
        B.SLA_ERR_SHAPE
