"""Host-side paths of the C ABI on the GPU: the caller's allocator (PyTorch's
caching allocator, and one that runs out), and the bounded wait of the
forward's read-back. Every failure here is forced from the host; every kernel
still runs to its normal end."""
import ctypes
import gc

import numpy as np
import pytest
import torch

import paper_2512_19743_amd as apml
from paper_2512_19743_amd import _lib
from workloads import batch, config, custom

from ._parity import note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    apml.load()


def _run(X, Y, **prm):
    x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    loss, plan = apml.apml_forward(x, y, apml.apml_params_default(**prm))
    gx, gy = apml.apml_backward(plan, x, y, torch.ones(X.shape[0], device="cuda"), want_grad_y=True)
    torch.cuda.synchronize()
    out = loss.cpu().numpy(), gx.cpu().numpy(), gy.cpu().numpy()
    plan.close()
    torch.cuda.synchronize()
    return out


def test_torch_caching_allocator_route():
    w = config(1)
    X, Y = batch(w)
    note("allocator: torch caching allocator")
    gc.collect()  # plans of earlier tests: the allocator may change only while none is alive
    ref = _run(X, Y, n_iter=w.n_iter)
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    apml.apml_set_allocator_torch()
    try:
        x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
        base = torch.cuda.memory_allocated()
        loss, plan = apml.apml_forward(x, y, apml.apml_params_default(n_iter=w.n_iter))
        held = torch.cuda.memory_allocated() - base
        assert held - 4 * w.B >= plan.info().bytes > 0  # the plan's arrays come from PyTorch
        gx, gy = apml.apml_backward(plan, x, y, torch.ones(w.B, device="cuda"), want_grad_y=True)
        torch.cuda.synchronize()
        got = loss.cpu().numpy(), gx.cpu().numpy(), gy.cpu().numpy()
        del loss, gx, gy
        plan.close()
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == base  # everything given back
        for a, b in zip(got, ref):
            assert np.array_equal(a, b)
    finally:
        apml.apml_set_allocator_default()


class _CountingAllocator:
    """PyTorch-backed allocator that returns NULL from its n-th call on. Its
    callbacks never raise into C (a ctypes callback that raises returns an
    undefined pointer): failures are recorded in errors and checked by the
    test."""

    def __init__(self, fail_from: int):
        self.fail_from = fail_from
        self.calls = 0
        self.live = {}
        self.errors = []
        self.alloc = _lib.ALLOC_FN(self._alloc)
        self.free = _lib.FREE_FN(self._free)

    def _alloc(self, size, stream, user):
        try:
            self.calls += 1
            if self.calls >= self.fail_from:
                return None
            p = torch.cuda.caching_allocator_alloc(int(size), torch.cuda.current_device(), stream or 0)
            self.live[p] = size
            return p
        except BaseException as e:  # noqa: BLE001
            self.errors.append(repr(e))
            return None

    def _free(self, ptr, size, stream, user):
        try:
            if self.live.pop(ptr, None) != size:
                self.errors.append(f"free of {ptr:#x} with size {size} that was not handed out")
            torch.cuda.caching_allocator_delete(ptr)
        except BaseException as e:  # noqa: BLE001
            self.errors.append(repr(e))


def _forward_raw(lib, x, y, loss, plan):
    B, N, M = x.shape[0], x.shape[1], y.shape[1]
    return lib.apml_forward(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), B, N, M, 3,
                            ctypes.byref(apml.apml_params_default()), ctypes.c_void_p(loss.data_ptr()),
                            ctypes.byref(plan), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


@pytest.mark.parametrize("where", ["first", "middle", "last_forward", "backward"])
def test_allocator_returning_null(where):
    # the allocator fails at its first call, halfway through the forward's
    # calls, at the forward's last call (after the read-back and the sparse
    # build), or in the backward
    X, Y = custom(51, 2, 300, 280, sigma=0.05)
    x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    lib = apml.load()
    gc.collect()  # plans of earlier tests: the allocator may change only while none is alive
    count = _CountingAllocator(1 << 30)
    assert lib.apml_set_allocator(count.alloc, count.free, None) == 0
    try:
        plan = ctypes.c_void_p()
        assert _forward_raw(lib, x, y, torch.empty(2, device="cuda"), plan) == 0
        n_forward = count.calls
        lib.apml_plan_destroy(plan)
        torch.cuda.synchronize()
    finally:
        assert lib.apml_set_allocator(_lib.ALLOC_FN(), _lib.FREE_FN(), None) == 0
    fail_from = {"first": 1, "middle": max(1, n_forward // 2), "last_forward": n_forward,
                 "backward": n_forward + 1}[where]
    note(f"allocator: NULL from call {fail_from} of the forward's {n_forward}")
    a = _CountingAllocator(fail_from)
    assert lib.apml_set_allocator(a.alloc, a.free, None) == 0
    try:
        before = apml.apml_get_memory_stats()["in_use"]
        loss = torch.full((2,), 7.0, device="cuda")
        plan = ctypes.c_void_p(0x1)
        st = _forward_raw(lib, x, y, loss, plan)
        if where == "backward":
            assert st == 0, lib.apml_last_error()
            gx = torch.empty_like(x)
            st = lib.apml_backward(plan, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                                   ctypes.c_void_p(torch.ones(2, device="cuda").data_ptr()),
                                   ctypes.c_void_p(gx.data_ptr()), None,
                                   ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            assert st == 3, lib.apml_last_error()
            assert lib.apml_plan_destroy(plan) == 0
        else:
            assert st == 3, lib.apml_last_error()
            assert plan.value is None
            torch.cuda.synchronize()
            assert (loss == 7.0).all()  # the loss is written by the last kernels of the forward
        torch.cuda.synchronize()
        assert a.errors == [] and count.errors == []
        assert a.live == {}, "every block the library took must be given back"
        assert apml.apml_get_memory_stats()["in_use"] == before
    finally:
        assert lib.apml_set_allocator(_lib.ALLOC_FN(), _lib.FREE_FN(), None) == 0


def test_forward_wait_deadline(monkeypatch):
    # a spin kernel queued ahead keeps the stream busy; with a zero deadline
    # the forward must report the device as not finishing instead of waiting
    X, Y = custom(52, 1, 64, 64, sigma=0.05)
    x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    note("read-back deadline")
    torch.cuda.synchronize()
    monkeypatch.setenv("APML_WAIT_TIMEOUT_S", "0")
    torch.cuda._sleep(50_000_000)
    with pytest.raises(apml.ApmlError) as err:
        apml.apml_forward(x, y)
    assert err.value.status == 4 and "APML_WAIT_TIMEOUT_S" in str(err.value)
    torch.cuda.synchronize()
    monkeypatch.delenv("APML_WAIT_TIMEOUT_S")
    loss, plan = apml.apml_forward(x, y)
    torch.cuda.synchronize()
    assert np.isfinite(loss.cpu().numpy()).all()


@pytest.mark.parametrize("fail_at", [1, 4])
def test_torch_route_out_of_memory(monkeypatch, fail_at):
    # PyTorch's allocator raising (as it does when the device is full) must
    # reach the library as NULL: the call reports APML_ERR_OUT_OF_MEMORY and
    # every block taken before is given back
    X, Y = custom(53, 2, 300, 280, sigma=0.05)
    x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    note(f"allocator: PyTorch route raising at call {fail_at}")
    gc.collect()
    torch.cuda.synchronize()
    real = torch.cuda.caching_allocator_alloc
    calls = [0]

    def flaky(size, device=None, stream=None):
        calls[0] += 1
        if calls[0] >= fail_at:
            raise torch.OutOfMemoryError("forced by the test")
        return real(size, device, stream)

    apml.apml_set_allocator_torch()
    try:
        base = torch.cuda.memory_allocated()
        before = apml.apml_get_memory_stats()["in_use"]
        monkeypatch.setattr(torch.cuda, "caching_allocator_alloc", flaky)
        with pytest.raises(apml.ApmlError) as err:
            apml.apml_forward(x, y)
        assert err.value.status == 3 and "forced by the test" in str(err.value)
        monkeypatch.setattr(torch.cuda, "caching_allocator_alloc", real)
        del err  # its traceback holds the wrapper's output tensor
        gc.collect()
        torch.cuda.synchronize()
        assert apml.apml_get_memory_stats()["in_use"] == before
        assert torch.cuda.memory_allocated() == base
        loss, plan = apml.apml_forward(x, y)
        torch.cuda.synchronize()
        assert np.isfinite(loss.cpu().numpy()).all()
        plan.close()
        del loss
        torch.cuda.synchronize()
    finally:
        monkeypatch.setattr(torch.cuda, "caching_allocator_alloc", real)
        apml.apml_set_allocator_default()
