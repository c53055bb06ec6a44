"""C ABI checks that need no GPU: every declared symbol is exported, and
argument validation answers before any HIP call (so it is safe without a
device). Fake device pointers are never dereferenced on these paths."""
import ctypes
import os
import re

import pytest

from paper_2512_19743_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apml.h")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"\b(apml_[a-z_]+)\s*\(", text))
    types = set(re.findall(r"typedef\s+[^;]*?\(\s*\*\s*(apml_[a-z_]+)\s*\)", text))
    return sorted(names - types)


def test_header_declares_the_paths_entry_points():
    names = declared_functions()
    for required in ("apml_forward", "apml_backward", "apml_plan_destroy", "apml_plan_nnz",
                     "apml_plan_export", "apml_params_default"):
        assert required in names


def test_every_declared_symbol_is_exported():
    lib = _lib.load()
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_defaults_are_the_papers():
    p = _lib.apml_params_default()
    assert p.struct_size == ctypes.sizeof(_lib.apml_params) == 72
    assert (p.tau, p.n_iter, p.eps_stab) == (1e-8, 10, 1e-8)  # Sec. III-E, Sec. IV-C
    assert (p.p_min, p.delta, p.eps_gap, p.eps_dist) == (0.8, 1e-8, 1e-6, 1e-12)
    # clamp, half sum, full gradient
    assert (p.dense_scan, p.gap_mode, p.sym_mode, p.tgrad_mode) == (0, 0, 0, 0)


def _forward(B=2, N=8, M=8, d=3, params=None, x=FAKE, y=FAKE, loss=FAKE):
    lib = _lib.load()
    plan = ctypes.c_void_p(0x1)
    prm = params if params is not None else _lib.apml_params_default()
    st = lib.apml_forward(x, y, B, N, M, d, ctypes.byref(prm), loss, ctypes.byref(plan), None)
    return st, plan


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), 1), (dict(y=None), 1), (dict(loss=None), 1),
    (dict(B=0), 1), (dict(N=1), 1), (dict(M=1), 1), (dict(d=2), 2), (dict(d=4), 2),
    (dict(B=1 << 20, N=1 << 12), 2),
])
def test_forward_rejects_bad_shapes(kw, status):
    st, plan = _forward(**kw)
    assert st == status
    assert plan.value is None  # *plan is cleared on error
    assert _lib.load().apml_last_error()


@pytest.mark.parametrize("field,value", [
    ("p_min", 1.0), ("p_min", 0.0), ("p_min", 0.1), ("tau", -1e-3), ("tau", 1.5), ("n_iter", -1),
    ("delta", -1.0), ("eps_gap", 0.0), ("eps_stab", -1.0), ("eps_dist", -1.0), ("eps_gap", float("inf")),
    ("dense_scan", 3), ("gap_mode", 2), ("sym_mode", -1), ("tgrad_mode", 2),
])
def test_forward_rejects_bad_params(field, value):
    prm = _lib.apml_params_default(**{field: value})
    st, _ = _forward(N=8, M=8, params=prm)  # p_min = 0.1 fails 1/min(N,M) < p_min
    assert st == 1, (field, value)


def test_backward_and_plan_calls_reject_null():
    lib = _lib.load()
    assert lib.apml_backward(None, FAKE, FAKE, FAKE, FAKE, None, None) == 1
    assert lib.apml_plan_destroy(None) == 0
    assert lib.apml_plan_nnz(None, None) == 1
    assert lib.apml_plan_get_info(None, None) == 1
    assert lib.apml_plan_export(None, 0, 0, None, None, None, None, None, None, None) == 1


def test_host_only_utilities():
    lib = _lib.load()
    assert lib.apml_version() == 1
    assert lib.apml_status_string(0) == b"ok"
    assert lib.apml_status_string(3) == b"out of memory"
    assert [lib.apml_phase_name(k).decode() for k in range(8)] == [
        "stats", "support", "build", "softmax", "sinkhorn", "loss", "bwd_sinkhorn", "bwd_softmax"]
    assert lib.apml_phase_name(8) == b""
    stats = _lib.apml_get_memory_stats()
    assert stats["in_use"] == 0
    assert lib.apml_profile_enable(1) == 0 and lib.apml_profile_enable(0) == 0
    # the allocator hooks must come in pairs
    assert lib.apml_set_allocator(_lib.ALLOC_FN(lambda n, s, u: None), _lib.FREE_FN(), None) == 1


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 4, 3)
    with pytest.raises(ValueError, match="GPU"):
        _lib.apml_forward(x, x)


def test_loss_params_by_name():
    from paper_2512_19743_amd.loss import loss_params
    p = loss_params(gap_mode="uniform_fallback", sym_mode="mean_dup", tgrad_mode="detached", dense_scan="skip",
                    n_iter=3)
    assert (p.gap_mode, p.sym_mode, p.tgrad_mode, p.dense_scan, p.n_iter) == (1, 1, 1, 2, 3)
    d = loss_params()
    assert (d.gap_mode, d.sym_mode, d.tgrad_mode, d.dense_scan) == (0, 0, 0, 0)
    with pytest.raises(ValueError):
        loss_params(sym_mode="average")


def test_noalloc_validates_before_any_hip_call():
    lib = _lib.load()
    prm = _lib.apml_params_default()
    call = lambda B=2, N=8, M=8, d=3, loss=FAKE, gl=FAKE, gx=FAKE: lib.apml_forward_backward_noalloc(  # noqa: E731
        FAKE, FAKE, B, N, M, d, ctypes.byref(prm), loss, gl, gx, None, None)
    assert call(loss=None) == 1
    assert call(d=2) == 2
    assert call(N=1) == 1
    assert call(gl=None) == 1  # gradients requested without an upstream gradient
    assert call(B=1792) == 2 and "at most 1791" in lib.apml_last_error().decode()


def test_dense_validates_before_any_hip_call():
    lib = _lib.load()
    prm = _lib.apml_params_default()
    plan = ctypes.c_void_p(0x1)
    call = lambda B=2, N=8, M=8, d=3, loss=FAKE, params=prm: lib.apml_dense_forward(  # noqa: E731
        FAKE, FAKE, B, N, M, d, ctypes.byref(params), loss, ctypes.byref(plan), None)
    assert call(loss=None) == 1 and plan.value is None
    assert call(N=1) == 1
    assert call(d=0) == 2 and call(d=17) == 2
    assert call(params=_lib.apml_params_default(gap_mode=1)) == 2
    assert call(params=_lib.apml_params_default(sym_mode=1)) == 2
    assert call(params=_lib.apml_params_default(p_min=1.0)) == 1
    assert lib.apml_dense_backward(None, FAKE, FAKE, FAKE, FAKE, None, None) == 1
    assert lib.apml_dense_plan_destroy(None) == 0
