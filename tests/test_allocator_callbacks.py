"""The PyTorch allocator route's callbacks on the CPU: an exception raised in
a ctypes callback does not reach the C caller as NULL (ctypes reports it and
returns an undefined value), so the binding's callbacks must catch every
failure and return NULL themselves."""
import ctypes

import pytest
import torch

from paper_2512_19743_amd import _lib


@pytest.mark.filterwarnings("ignore::pytest.PytestUnraisableExceptionWarning")
def test_raising_ctypes_callback_does_not_return_null():
    # the reason for the wrappers below: the return value of a callback that
    # raises is not defined (it is not NULL in practice)
    def boom(size, stream, user):
        raise MemoryError("no memory")

    f = _lib.ALLOC_FN(boom)
    g = ctypes.cast(f, _lib.ALLOC_FN)
    got = [g(1024, None, None) for _ in range(4)]
    assert any(v not in (None, 0) for v in got)


def test_torch_alloc_returns_null_when_pytorch_raises(monkeypatch):
    def oom(size, device=None, stream=None):
        raise torch.OutOfMemoryError("device full")

    monkeypatch.setattr(torch.cuda, "caching_allocator_alloc", oom)
    monkeypatch.setattr(torch.cuda, "current_device", lambda: 0)
    _lib.torch_alloc_error = None
    f = _lib.ALLOC_FN(_lib.torch_alloc)
    g = ctypes.cast(f, _lib.ALLOC_FN)
    assert g(1 << 20, None, None) is None
    assert isinstance(_lib.torch_alloc_error, torch.OutOfMemoryError)
    _lib.torch_alloc_error = None


def test_torch_alloc_passes_the_pointer_and_stream(monkeypatch):
    seen = []

    def fake(size, device=None, stream=None):
        seen.append((size, device, stream))
        return 0x7F0000001000

    monkeypatch.setattr(torch.cuda, "caching_allocator_alloc", fake)
    monkeypatch.setattr(torch.cuda, "current_device", lambda: 0)
    g = ctypes.cast(_lib.ALLOC_FN(_lib.torch_alloc), _lib.ALLOC_FN)
    assert g(4096, ctypes.c_void_p(0x1234), None) == 0x7F0000001000
    assert g(4096, None, None) == 0x7F0000001000
    assert seen == [(4096, 0, 0x1234), (4096, 0, 0)]


def test_torch_free_never_raises(monkeypatch):
    def bad(ptr):
        raise RuntimeError("unknown pointer")

    monkeypatch.setattr(torch.cuda, "caching_allocator_delete", bad)
    _lib.torch_alloc_error = None
    g = ctypes.cast(_lib.FREE_FN(_lib.torch_free), _lib.FREE_FN)
    g(ctypes.c_void_p(0x1000), 16, None, None)
    assert isinstance(_lib.torch_alloc_error, RuntimeError)
    _lib.torch_alloc_error = None


def test_out_of_memory_error_names_the_allocator_exception():
    _lib.torch_alloc_error = torch.OutOfMemoryError("device full")
    try:
        _lib._check("apml_forward", 3)
    except _lib.ApmlError as e:
        assert e.status == 3 and "device full" in str(e)
    else:
        raise AssertionError("no error raised")
    assert _lib.torch_alloc_error is None
