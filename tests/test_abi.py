"""The C ABI on the host: exported symbols and argument validation.

Every call here carries at least one invalid argument, so the library returns
its status before any device work; nothing is launched.  (Fake pointers are
only ever paired with an argument that fails validation.)
"""

import ctypes
import math
import os
import re

import pytest

from paper_1802_01561_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vtrace.h")

OK, NULL, SHAPE, DTYPE, PARAM, ALIGN, WS = 0, 1, 2, 3, 4, 5, 6
P = 0x10000  # a 16-byte-aligned fake device address, never dereferenced


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vtrace_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) == 14
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(_lib.SIGNATURES)


def test_version_and_strings(L):
    assert L.vtrace_abi_version() == 1
    for s in range(8):
        assert len(L.vtrace_status_string(s)) > 0
    assert L.vtrace_status_string(99) == b"unknown status"
    assert L.vtrace_max_elements() == 1 << 40


def test_workspace_bytes(L):
    assert L.vtrace_workspace_bytes(0, 4, 9) == 0
    assert L.vtrace_workspace_bytes(5, -1, 9) == 0
    assert L.vtrace_workspace_bytes(1 << 20, 1 << 20, 2) == 0
    n1 = L.vtrace_workspace_bytes(5, 4, 9)
    n2 = L.vtrace_workspace_bytes(5, 4096, 9)
    assert 256 <= n1 < n2
    assert L.vtrace_workspace_bytes(1000, 16384, 18) == L.vtrace_workspace_bytes(1, 16384, 1)


def _targets(L, **kw):
    a = dict(T=5, B=4, A=9, dt=0, tl=P, bl=P, act=P, r=P, d=P, v=P, boot=P, rho=1.0, c=1.0,
             lam=1.0, vs=P, pg=P, ws=None, nws=0)
    a.update(kw)
    return L.vtrace_targets(a["T"], a["B"], a["A"], a["dt"], a["tl"], a["bl"], a["act"], a["r"],
                            a["d"], a["v"], a["boot"], a["rho"], a["c"], a["lam"], a["vs"], a["pg"],
                            a["ws"], a["nws"], None)


def _loss(L, **kw):
    a = dict(T=5, B=4, A=9, dt=0, tl=P, bl=P, act=P, r=P, d=P, v=P, boot=P, rho=1.0, c=1.0,
             lam=1.0, cv=0.5, ce=0.01, losses=P, dl=P, dv=P, vs=None, pg=None, lane=None,
             ws=P, nws=1 << 20)
    a.update(kw)
    return L.vtrace_loss_grad(a["T"], a["B"], a["A"], a["dt"], a["tl"], a["bl"], a["act"], a["r"],
                              a["d"], a["v"], a["boot"], a["rho"], a["c"], a["lam"], a["cv"],
                              a["ce"], a["losses"], a["dl"], a["dv"], a["vs"], a["pg"], a["lane"],
                              a["ws"], a["nws"], None)


INVALID = [
    # (kwargs, expected status) -- each case is rejected before any launch
    (dict(tl=None), NULL), (dict(bl=None), NULL), (dict(act=None), NULL), (dict(r=None), NULL),
    (dict(d=None), NULL), (dict(v=None), NULL), (dict(boot=None), NULL),
    (dict(T=0), SHAPE), (dict(B=0), SHAPE), (dict(A=0), SHAPE), (dict(T=-3), SHAPE),
    (dict(T=1 << 21, B=1 << 20), SHAPE),
    (dict(dt=2), DTYPE), (dict(dt=-1), DTYPE),
    (dict(rho=math.nan), PARAM), (dict(c=math.nan), PARAM), (dict(rho=-1.0), PARAM),
    (dict(c=-0.5), PARAM), (dict(lam=1.5), PARAM), (dict(lam=-0.1), PARAM),
    (dict(lam=math.nan), PARAM),
    (dict(tl=P + 4), ALIGN), (dict(bl=P + 8), ALIGN), (dict(act=P + 2), ALIGN),
    (dict(r=P + 1), ALIGN),
]


@pytest.mark.parametrize("kw,status", INVALID)
def test_targets_rejects(L, kw, status):
    assert _targets(L, **kw) == status


def test_targets_rejects_outputs(L):
    assert _targets(L, vs=None) == NULL
    assert _targets(L, pg=None) == NULL
    assert _targets(L, vs=P + 2) == ALIGN
    assert _targets(L, ws=P + 4, nws=4096, rho=math.nan) == PARAM
    assert _targets(L, ws=P + 4, nws=4096) == ALIGN
    assert _targets(L, ws=P, nws=16) == WS


@pytest.mark.parametrize("kw,status", INVALID)
def test_loss_grad_rejects(L, kw, status):
    assert _loss(L, **kw) == status


def test_loss_grad_rejects_outputs_and_workspace(L):
    assert _loss(L, losses=None) == NULL
    assert _loss(L, dl=None) == NULL
    assert _loss(L, dv=None) == NULL
    assert _loss(L, dl=P + 4) == ALIGN
    assert _loss(L, vs=P + 2) == ALIGN
    assert _loss(L, lane=P + 1) == ALIGN
    assert _loss(L, cv=math.inf) == PARAM
    assert _loss(L, ce=math.nan) == PARAM
    assert _loss(L, ws=None) == WS
    assert _loss(L, nws=16) == WS
    assert _loss(L, B=4096, nws=L.vtrace_workspace_bytes(5, 4096, 9) - 1) == WS
    assert _loss(L, ws=P + 8) == ALIGN


def test_variant_validation(L):
    V = _lib.Variant
    base = dict(T=5, B=4, A=9, dt=0, tl=P, bl=P, act=P, r=P, d=P, v=P, boot=P)

    def loss_ex(variant, **kw):
        a = dict(base, rho=1.0, c=1.0, lam=1.0, cv=0.5, ce=0.01, losses=P, dl=P, dv=P, ws=P,
                 nws=1 << 20)
        a.update(kw)
        return L.vtrace_loss_grad_ex(a["T"], a["B"], a["A"], a["dt"], a["tl"], a["bl"], a["act"],
                                     a["r"], a["d"], a["v"], a["boot"], a["rho"], a["c"], a["lam"],
                                     a["cv"], a["ce"], variant, a["losses"], a["dl"], a["dv"], None,
                                     None, None, a["ws"], a["nws"], None)

    def targets_ex(variant, **kw):
        a = dict(base, rho=1.0, c=1.0, lam=1.0)
        a.update(kw)
        return L.vtrace_targets_ex(a["T"], a["B"], a["A"], a["dt"], a["tl"], a["bl"], a["act"],
                                   a["r"], a["d"], a["v"], a["boot"], a["rho"], a["c"], a["lam"],
                                   variant, P, P, None, 0, None)

    for bad in (V(4, 0, 1e-6), V(-1, 0, 1e-6), V(0, 2, 1e-6), V(0, -1, 1e-6), V(2, 0, 0.0),
                V(2, 0, -1e-6), V(2, 0, math.nan), V(2, 0, math.inf), V(0, 0, 0.0, 2, 0, 0),
                V(0, 0, 0.0, -1, 0, 0), V(0, 0, 0.0, 0, 3, 0), V(0, 0, 0.0, 0, -1, 0)):
        assert loss_ex(ctypes.byref(bad)) == PARAM
        assert targets_ex(ctypes.byref(bad)) == PARAM
    assert loss_ex(ctypes.byref(V(0, 0, 0.0, 0, 0, 2))) == DTYPE
    # behaviour logits need 16-byte alignment, behaviour log-probabilities 4
    assert loss_ex(None, bl=P + 4, ws=None) == WS
    assert loss_ex(None, bl=P + 4) == ALIGN
    assert loss_ex(ctypes.byref(V(0, 0, 0.0, 1, 0, 0)), bl=P + 4, T=0) == SHAPE
    assert loss_ex(ctypes.byref(V(0, 0, 0.0, 1, 0, 0)), bl=P + 2) == ALIGN
    # a valid variant with another invalid argument is still rejected before launch
    for good in (None, ctypes.byref(V(0, 0, 0.0)), ctypes.byref(V(3, 1, 0.0)),
                 ctypes.byref(V(2, 0, 1e-6))):
        assert loss_ex(good, T=0) == SHAPE
        assert loss_ex(good, ws=None) == WS
        assert targets_ex(good, lam=2.0) == PARAM


def test_python_variant_names():
    from paper_1802_01561_amd import binding
    import torch
    assert binding._variant("one_step_is", "baseline", 1e-6).correction == 3
    assert binding._variant("epsilon", "vtrace", 1e-6).q_estimate == 0
    v = binding._variant(behaviour="log_probs", reward_transform="asymmetric",
                         grad_dtype=torch.bfloat16)
    assert (v.behaviour_input, v.reward_transform, v.grad_dtype) == (1, 2, 1)
    for bad in (dict(correction="retrace"), dict(behaviour="probs"), dict(reward_transform="tanh"),
                dict(grad_dtype=torch.float16)):
        with pytest.raises(ValueError):
            binding._variant(**bad)


def test_gather_and_flag_reject(L):
    g = L.vtrace_gather_logits
    assert g(5, 4, 9, 0, None, P, P, P, None) == NULL
    assert g(5, 4, 9, 0, P, P, P, None, None) == NULL
    assert g(0, 4, 9, 0, P, P, P, P, None) == SHAPE
    assert g(5, 4, 9, 7, P, P, P, P, None) == DTYPE
    assert g(5, 4, 9, 0, P, P, P, P + 4, None) == ALIGN
    flag = ctypes.c_int32(0)
    assert L.vtrace_error_flag(None, ctypes.byref(flag), None) == NULL
    assert L.vtrace_error_flag(P, None, None) == NULL
    assert L.vtrace_error_flag(P + 4, ctypes.byref(flag), None) == ALIGN
    assert L.vtrace_workspace_init(None, 1024, None) == NULL
    assert L.vtrace_workspace_init(P + 4, 1024, None) == ALIGN
    assert L.vtrace_workspace_init(P, 100, None) == WS


def test_python_binding_validates_before_calling():
    torch = pytest.importorskip("torch")
    import paper_1802_01561_amd as v
    z = torch.zeros(2, 3, 4)
    with pytest.raises(ValueError):
        v.vtrace_targets(z, z, torch.zeros(2, 3, dtype=torch.int32), torch.zeros(2, 3),
                         torch.zeros(2, 3), torch.zeros(2, 3), torch.zeros(3))
    with pytest.raises(TypeError):
        v.binding._dtype_code(torch.zeros(1, dtype=torch.float16))


def _head(L, **kw):
    V = _lib.Variant
    a = dict(T=5, B=4, A=9, H=64, dt=0, h=P, W=P, bias=P, beh=P, act=P, r=P, d=P, boot=P, rho=1.0,
             c=1.0, lam=1.0, cv=0.5, ce=0.01, variant=None, losses=P, dh=P, dW=P, db=P, vs=None,
             pg=None, lane=None, outs=None, ws=P, nws=1 << 24)
    a.update(kw)
    return L.vtrace_head_loss_grad(a["T"], a["B"], a["A"], a["H"], a["dt"], a["h"], a["W"], a["bias"],
                                   a["beh"], a["act"], a["r"], a["d"], a["boot"], a["rho"], a["c"],
                                   a["lam"], a["cv"], a["ce"], a["variant"], a["losses"], a["dh"],
                                   a["dW"], a["db"], a["vs"], a["pg"], a["lane"], a["outs"], a["ws"],
                                   a["nws"], None)


def test_head_workspace_bytes(L):
    n = L.vtrace_head_workspace_bytes
    assert n(5, 4, 9, 64) >= 256 + 3 * 8 + 65 * 16 * 4
    assert n(5, 4, 16, 64) > n(5, 4, 15, 64)  # 17 outputs need two column tiles
    assert n(1000, 16384, 18, 256) == n(1, 16384, 18, 256)
    for bad in ((0, 4, 9, 64), (5, 0, 9, 64), (5, 4, 0, 64), (5, 4, 32, 64), (5, 4, 9, 100),
                (5, 4, 9, 512), (1 << 21, 1 << 20, 9, 64)):
        assert n(*bad) == 0, bad


HEAD_INVALID = [
    (dict(h=None), NULL), (dict(W=None), NULL), (dict(bias=None), NULL), (dict(beh=None), NULL),
    (dict(act=None), NULL), (dict(r=None), NULL), (dict(d=None), NULL), (dict(boot=None), NULL),
    (dict(losses=None), NULL), (dict(dh=None), NULL), (dict(dW=None), NULL), (dict(db=None), NULL),
    (dict(T=0), SHAPE), (dict(A=32), SHAPE), (dict(A=0), SHAPE), (dict(H=96), SHAPE),
    (dict(H=512), SHAPE), (dict(dt=5), DTYPE),
    (dict(rho=math.nan), PARAM), (dict(lam=1.5), PARAM), (dict(cv=math.inf), PARAM),
    (dict(h=P + 8), ALIGN), (dict(dh=P + 8), ALIGN), (dict(W=P + 1), ALIGN), (dict(beh=P + 2), ALIGN),
    (dict(bias=P + 2), ALIGN), (dict(outs=P + 2), ALIGN),
    (dict(ws=None), WS), (dict(nws=1024), WS), (dict(ws=P + 8), ALIGN),
]


@pytest.mark.parametrize("kw,status", HEAD_INVALID)
def test_head_rejects(L, kw, status):
    assert _head(L, **kw) == status


def test_head_variant_and_behaviour_alignment(L):
    V = _lib.Variant
    assert _head(L, variant=ctypes.byref(V(5, 0, 0.0))) == PARAM
    assert _head(L, variant=ctypes.byref(V(0, 0, 0.0, 0, 0, 3))) == DTYPE
    # bfloat16 behaviour logits are read element by element: 2-byte alignment,
    # checked together with another invalid argument so that nothing launches
    assert _head(L, dt=1, beh=P + 2, T=0) == SHAPE
    assert _head(L, dt=1, beh=P + 1) == ALIGN
    assert _head(L, variant=ctypes.byref(V(0, 0, 0.0, 1, 0, 0)), beh=P + 2) == ALIGN


def test_python_head_binding_validates_before_calling():
    torch = pytest.importorskip("torch")
    import paper_1802_01561_amd as v
    T, B, A, H = 3, 2, 5, 64
    h = torch.zeros(T, B, H, dtype=torch.bfloat16)
    W = torch.zeros(H, A + 1, dtype=torch.bfloat16)
    args = [h, W, torch.zeros(A + 1), torch.zeros(T, B, A), torch.zeros(T, B, dtype=torch.int32),
            torch.zeros(T, B), torch.zeros(T, B), torch.zeros(B)]
    with pytest.raises(ValueError):  # CPU tensors are refused before any device work
        v.vtrace_head_loss_grad(*args)
    with pytest.raises(ValueError):
        v.vtrace_head_loss_grad(h[0], *args[1:])  # hidden must be [T, B, H]
    with pytest.raises(ValueError):
        v.vtrace_head_loss_grad(*args, correction="retrace")
    with pytest.raises(ValueError):
        v.vtrace_head_loss_grad(*args, grad_dtype=torch.float16)


def test_static_loss_grad_rejects_before_any_device_call(L):
    """vtrace_loss_grad_static validates like vtrace_loss_grad_ex and refuses
    batches wider than its fixed device array; every call here fails before
    the library asks for that array."""
    V = _lib.Variant
    base = dict(T=5, B=4, A=9, dt=0, tl=P, bl=P, act=P, r=P, d=P, v=P, boot=P, rho=1.0, c=1.0,
                lam=1.0, cv=0.5, ce=0.01, losses=P, dl=P, dv=P, variant=None)

    def st(**kw):
        a = dict(base)
        a.update(kw)
        return L.vtrace_loss_grad_static(a["T"], a["B"], a["A"], a["dt"], a["tl"], a["bl"],
                                         a["act"], a["r"], a["d"], a["v"], a["boot"], a["rho"],
                                         a["c"], a["lam"], a["cv"], a["ce"], a["variant"],
                                         a["losses"], a["dl"], a["dv"], None, None, None, None)

    assert st(B=65537) == WS
    assert st(B=1 << 20, T=1, A=2) == WS
    assert st(T=0) == SHAPE
    assert st(losses=None) == NULL
    assert st(dl=P + 4) == ALIGN
    assert st(dt=7) == DTYPE
    assert st(lam=1.5) == PARAM
    assert st(cv=math.nan) == PARAM
    assert st(variant=ctypes.byref(V(9, 0, 1e-6))) == PARAM
    assert st(B=65537, variant=ctypes.byref(V(9, 0, 1e-6))) == WS
