"""ctypes binding of libapml.so (include/apml.h), same names as the C ABI.

Only argument marshalling happens here: tensors are checked (device,
dtype, layout), outputs are allocated with PyTorch and their pointers handed to
the library, which does all the computation on the GPU. There is no CPU
fallback: if libapml.so is missing or a tensor is not on a GPU, a call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libapml.so")

APML_OK = 0
N_PHASES = 8
_STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "out of memory", 4: "device error",
           5: "internal error"}


class ApmlError(RuntimeError):
    def __init__(self, func: str, status: int, detail: str):
        super().__init__(f"{func}: {_STATUS.get(status, status)}: {detail}")
        self.status = status


class apml_params(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("n_iter", ctypes.c_int32),
        ("p_min", ctypes.c_double),
        ("tau", ctypes.c_double),
        ("eps_stab", ctypes.c_double),
        ("delta", ctypes.c_double),
        ("eps_gap", ctypes.c_double),
        ("eps_dist", ctypes.c_double),
        ("dense_scan", ctypes.c_int32),
        ("gap_mode", ctypes.c_int32),
        ("sym_mode", ctypes.c_int32),
        ("tgrad_mode", ctypes.c_int32),
    ]


class apml_plan_info(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("N", ctypes.c_int32), ("M", ctypes.c_int32),
                ("n_iter", ctypes.c_int32), ("stored_pairs", ctypes.c_int64), ("bytes", ctypes.c_int64),
                ("scanned_min", ctypes.c_int64), ("scanned_support", ctypes.c_int64)]


class apml_memory_stats(ctypes.Structure):
    _fields_ = [("in_use", ctypes.c_int64), ("peak_in_use", ctypes.c_int64), ("reserved", ctypes.c_int64)]


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)

_lib = None
_lock = threading.Lock()


def load() -> ctypes.CDLL:
    """Loads libapml.so from the package directory (built by build_lib.build())."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2512_19743_amd.build_lib.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, vp = ctypes.POINTER, ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.apml_params_default.argtypes = [P(apml_params)]
        L.apml_params_default.restype = None
        L.apml_forward.argtypes = [vp, vp, i32, i32, i32, i32, P(apml_params), vp, P(vp), vp]
        L.apml_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.apml_forward_backward_noalloc.argtypes = [vp, vp, i32, i32, i32, i32, P(apml_params), vp, vp, vp, vp,
                                                    vp]
        L.apml_plan_destroy.argtypes = [vp]
        L.apml_dense_forward.argtypes = [vp, vp, i32, i32, i32, i32, P(apml_params), vp, P(vp), vp]
        L.apml_dense_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.apml_dense_plan_destroy.argtypes = [vp]
        L.apml_plan_get_info.argtypes = [vp, P(apml_plan_info)]
        L.apml_plan_nnz.argtypes = [vp, P(i64)]
        L.apml_plan_export.argtypes = [vp, i32, i64, P(i32), P(i32), P(ctypes.c_uint8), P(ctypes.c_float),
                                       P(ctypes.c_float), P(ctypes.c_float), P(ctypes.c_float)]
        L.apml_plan_export_stats.argtypes = [vp, i32, P(ctypes.c_double), P(i32), P(i32), P(ctypes.c_uint8),
                                             P(ctypes.c_double), P(i32), P(i32), P(ctypes.c_uint8)]
        L.apml_set_allocator.argtypes = [ALLOC_FN, FREE_FN, vp]
        L.apml_get_memory_stats.argtypes = [P(apml_memory_stats)]
        L.apml_reset_peak_memory.argtypes = []
        L.apml_release_cached_memory.argtypes = []
        L.apml_profile_enable.argtypes = [i32]
        L.apml_profile_reset.argtypes = []
        L.apml_profile_read.argtypes = [i32, P(ctypes.c_double), P(i64)]
        L.apml_phase_name.argtypes = [i32]
        L.apml_phase_name.restype = ctypes.c_char_p
        L.apml_status_string.argtypes = [ctypes.c_int]
        L.apml_status_string.restype = ctypes.c_char_p
        L.apml_last_error.argtypes = []
        L.apml_last_error.restype = ctypes.c_char_p
        L.apml_version.argtypes = []
        L.apml_version.restype = i32
        for name in ("apml_forward", "apml_backward", "apml_forward_backward_noalloc", "apml_plan_destroy",
                     "apml_dense_forward", "apml_dense_backward", "apml_dense_plan_destroy", "apml_plan_get_info",
                     "apml_plan_nnz", "apml_plan_export", "apml_plan_export_stats", "apml_set_allocator",
                     "apml_get_memory_stats", "apml_reset_peak_memory", "apml_release_cached_memory",
                     "apml_profile_enable", "apml_profile_reset", "apml_profile_read"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
        return L


def _check(func: str, status: int):
    global torch_alloc_error
    if status != APML_OK:
        detail = load().apml_last_error().decode()
        if status == 3 and torch_alloc_error is not None:
            detail += f" (PyTorch's allocator: {type(torch_alloc_error).__name__}: {torch_alloc_error})"
        torch_alloc_error = None
        raise ApmlError(func, status, detail)


def apml_params_default(**overrides) -> apml_params:
    p = apml_params()
    load().apml_params_default(ctypes.byref(p))
    for k, v in overrides.items():
        if not hasattr(p, k) or k == "struct_size":
            raise TypeError(f"unknown APML parameter {k!r}")
        setattr(p, k, v)
    return p


def _stream_handle(stream: Optional[torch.cuda.Stream], device: torch.device) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return ctypes.c_void_p(s.cuda_stream)


def _gpu_f32(t: torch.Tensor, name: str, shape_tail=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a tensor on a GPU (libapml has no CPU path)")
    if t.dtype != torch.float32:
        raise ValueError(f"{name} must be float32, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


class Plan:
    """Owns an apml_plan handle; destroyed with the object."""

    def __init__(self, handle: ctypes.c_void_p, B: int, N: int, M: int, device: torch.device):
        self.handle = handle
        self.B, self.N, self.M = B, N, M
        self.device = device

    def close(self):
        if self.handle:
            with torch.cuda.device(self.device):
                load().apml_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> apml_plan_info:
        inf = apml_plan_info()
        _check("apml_plan_get_info", load().apml_plan_get_info(self.handle, ctypes.byref(inf)))
        return inf

    def nnz(self) -> np.ndarray:
        out = np.zeros(self.B, dtype=np.int64)
        with torch.cuda.device(self.device):
            _check("apml_plan_nnz", load().apml_plan_nnz(
                self.handle, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))))
        return out

    def export(self, b: int) -> dict:
        n = int(self.nnz()[b])
        i, j = np.empty(n, np.int32), np.empty(n, np.int32)
        fl = np.empty(n, np.uint8)
        arr = [np.empty(n, np.float32) for _ in range(4)]
        f = lambda a, ct: a.ctypes.data_as(ctypes.POINTER(ct))  # noqa: E731
        with torch.cuda.device(self.device):
            _check("apml_plan_export", load().apml_plan_export(
                self.handle, int(b), n, f(i, ctypes.c_int32), f(j, ctypes.c_int32), f(fl, ctypes.c_uint8),
                *[f(a, ctypes.c_float) for a in arr]))
        return dict(i=i, j=j, flags=fl, p_row=arr[0], p_col=arr[1], p0=arr[2], v=arr[3])

    def export_stats(self, b: int) -> dict:
        N, M = self.N, self.M
        Tr, Tc = np.empty(N), np.empty(M)
        j1, j2, i1, i2 = (np.empty(n, np.int32) for n in (N, N, M, M))
        cr, cc = np.empty(N, np.uint8), np.empty(M, np.uint8)
        f = lambda a, ct: a.ctypes.data_as(ctypes.POINTER(ct))  # noqa: E731
        with torch.cuda.device(self.device):
            _check("apml_plan_export_stats", load().apml_plan_export_stats(
                self.handle, int(b), f(Tr, ctypes.c_double), f(j1, ctypes.c_int32), f(j2, ctypes.c_int32),
                f(cr, ctypes.c_uint8), f(Tc, ctypes.c_double), f(i1, ctypes.c_int32), f(i2, ctypes.c_int32),
                f(cc, ctypes.c_uint8)))
        return dict(T_row=Tr, j1=j1, j2=j2, clamp_row=cr.astype(bool), T_col=Tc, i1=i1, i2=i2,
                    clamp_col=cc.astype(bool))


def apml_forward(x: torch.Tensor, y: torch.Tensor, params: Optional[apml_params] = None,
                 keep_plan: bool = True, stream: Optional[torch.cuda.Stream] = None
                 ) -> Tuple[torch.Tensor, Optional[Plan]]:
    """Per-sample losses (B,) float32 and, if keep_plan, the plan for apml_backward."""
    _gpu_f32(x, "x")
    _gpu_f32(y, "y")
    if x.dim() != 3 or y.dim() != 3 or x.shape[0] != y.shape[0] or x.device != y.device:
        raise ValueError("x must be (B,N,d) and y (B,M,d) on the same device")
    B, N, d = x.shape
    M = y.shape[1]
    if y.shape[2] != d:
        raise ValueError("x and y must have the same point dimension")
    params = params if params is not None else apml_params_default()
    loss = torch.empty(B, dtype=torch.float32, device=x.device)
    handle = ctypes.c_void_p()
    with torch.cuda.device(x.device):
        st = load().apml_forward(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), B, N, M, d,
                                 ctypes.byref(params), ctypes.c_void_p(loss.data_ptr()),
                                 ctypes.byref(handle) if keep_plan else None, _stream_handle(stream, x.device))
    _check("apml_forward", st)
    return loss, (Plan(handle, B, N, M, x.device) if keep_plan else None)


def apml_backward(plan: Plan, x: torch.Tensor, y: torch.Tensor, grad_loss: torch.Tensor,
                  want_grad_y: bool = False, stream: Optional[torch.cuda.Stream] = None
                  ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Gradients (B,N,3) and optionally (B,M,3) of sum_b grad_loss[b] * loss_b."""
    if plan is None or not plan.handle:
        raise ValueError("apml_backward needs a live plan from apml_forward(keep_plan=True)")
    _gpu_f32(x, "x")
    _gpu_f32(y, "y")
    _gpu_f32(grad_loss, "grad_loss")
    if tuple(x.shape) != (plan.B, plan.N, 3) or tuple(y.shape) != (plan.B, plan.M, 3):
        raise ValueError("x and y must have the shapes of the forward call")
    if grad_loss.numel() != plan.B or grad_loss.device != x.device:
        raise ValueError("grad_loss must have B entries on the device of x")
    gx = torch.empty_like(x)
    gy = torch.empty_like(y) if want_grad_y else None
    with torch.cuda.device(x.device):
        st = load().apml_backward(plan.handle, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                                  ctypes.c_void_p(grad_loss.data_ptr()), ctypes.c_void_p(gx.data_ptr()),
                                  ctypes.c_void_p(gy.data_ptr()) if gy is not None else None,
                                  _stream_handle(stream, x.device))
    _check("apml_backward", st)
    return gx, gy


def apml_forward_backward_noalloc(x: torch.Tensor, y: torch.Tensor, params: Optional[apml_params] = None,
                                  grad_loss: Optional[torch.Tensor] = None, want_grad: bool = True,
                                  want_grad_y: bool = False, stream: Optional[torch.cuda.Stream] = None
                                  ) -> Tuple[torch.Tensor, Optional[torch.Tensor], Optional[torch.Tensor]]:
    """Per-sample losses and (if want_grad) the gradients of sum_b grad_loss[b] * loss_b, in one call
    that allocates no device memory inside the library (its static scratch array holds every
    temporary). The output tensors are allocated here, by PyTorch, before the call."""
    _gpu_f32(x, "x")
    _gpu_f32(y, "y")
    if x.dim() != 3 or y.dim() != 3 or x.shape[0] != y.shape[0] or x.device != y.device:
        raise ValueError("x must be (B,N,d) and y (B,M,d) on the same device")
    B, N, d = x.shape
    M = y.shape[1]
    if y.shape[2] != d:
        raise ValueError("x and y must have the same point dimension")
    params = params if params is not None else apml_params_default()
    loss = torch.empty(B, dtype=torch.float32, device=x.device)
    gx = gy = None
    if want_grad:
        if grad_loss is None:
            grad_loss = torch.ones(B, dtype=torch.float32, device=x.device)
        _gpu_f32(grad_loss, "grad_loss")
        if grad_loss.numel() != B or grad_loss.device != x.device:
            raise ValueError("grad_loss must have B entries on the device of x")
        gx = torch.empty_like(x)
        gy = torch.empty_like(y) if want_grad_y else None
    ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None  # noqa: E731
    with torch.cuda.device(x.device):
        st = load().apml_forward_backward_noalloc(
            ptr(x), ptr(y), B, N, M, d, ctypes.byref(params), ptr(loss), ptr(grad_loss) if want_grad else None,
            ptr(gx), ptr(gy), _stream_handle(stream, x.device))
    _check("apml_forward_backward_noalloc", st)
    return loss, gx, gy


class DensePlan:
    """Owns an apml_dense_plan handle; destroyed with the object."""

    def __init__(self, handle: ctypes.c_void_p, B: int, N: int, M: int, d: int, device: torch.device):
        self.handle = handle
        self.B, self.N, self.M, self.d = B, N, M, d
        self.device = device

    def close(self):
        if self.handle:
            with torch.cuda.device(self.device):
                load().apml_dense_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def apml_dense_forward(x: torch.Tensor, y: torch.Tensor, params: Optional[apml_params] = None,
                       keep_plan: bool = True, stream: Optional[torch.cuda.Stream] = None
                       ) -> Tuple[torch.Tensor, Optional[DensePlan]]:
    """Dense APML (every pair, any d): per-sample losses (B,) and, if keep_plan, the plan."""
    _gpu_f32(x, "x")
    _gpu_f32(y, "y")
    if x.dim() != 3 or y.dim() != 3 or x.shape[0] != y.shape[0] or x.device != y.device:
        raise ValueError("x must be (B,N,d) and y (B,M,d) on the same device")
    B, N, d = x.shape
    M = y.shape[1]
    if y.shape[2] != d:
        raise ValueError("x and y must have the same point dimension")
    params = params if params is not None else apml_params_default()
    loss = torch.empty(B, dtype=torch.float32, device=x.device)
    handle = ctypes.c_void_p()
    with torch.cuda.device(x.device):
        st = load().apml_dense_forward(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), B, N, M, d,
                                       ctypes.byref(params), ctypes.c_void_p(loss.data_ptr()),
                                       ctypes.byref(handle) if keep_plan else None,
                                       _stream_handle(stream, x.device))
    _check("apml_dense_forward", st)
    return loss, (DensePlan(handle, B, N, M, d, x.device) if keep_plan else None)


def apml_dense_backward(plan: DensePlan, x: torch.Tensor, y: torch.Tensor, grad_loss: torch.Tensor,
                        want_grad_y: bool = False, stream: Optional[torch.cuda.Stream] = None
                        ) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Gradients (B,N,d) and optionally (B,M,d) of sum_b grad_loss[b] * loss_b (dense APML)."""
    if plan is None or not plan.handle:
        raise ValueError("apml_dense_backward needs a live plan from apml_dense_forward(keep_plan=True)")
    _gpu_f32(x, "x")
    _gpu_f32(y, "y")
    _gpu_f32(grad_loss, "grad_loss")
    if tuple(x.shape) != (plan.B, plan.N, plan.d) or tuple(y.shape) != (plan.B, plan.M, plan.d):
        raise ValueError("x and y must have the shapes of the forward call")
    if grad_loss.numel() != plan.B or grad_loss.device != x.device:
        raise ValueError("grad_loss must have B entries on the device of x")
    gx = torch.empty_like(x)
    gy = torch.empty_like(y) if want_grad_y else None
    with torch.cuda.device(x.device):
        st = load().apml_dense_backward(plan.handle, ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                                        ctypes.c_void_p(grad_loss.data_ptr()), ctypes.c_void_p(gx.data_ptr()),
                                        ctypes.c_void_p(gy.data_ptr()) if gy is not None else None,
                                        _stream_handle(stream, x.device))
    _check("apml_dense_backward", st)
    return gx, gy


def apml_get_memory_stats() -> dict:
    s = apml_memory_stats()
    _check("apml_get_memory_stats", load().apml_get_memory_stats(ctypes.byref(s)))
    return dict(in_use=s.in_use, peak_in_use=s.peak_in_use, reserved=s.reserved)


def apml_reset_peak_memory():
    _check("apml_reset_peak_memory", load().apml_reset_peak_memory())


def apml_release_cached_memory():
    _check("apml_release_cached_memory", load().apml_release_cached_memory())


def apml_profile_enable(on: bool = True):
    _check("apml_profile_enable", load().apml_profile_enable(1 if on else 0))


def apml_profile_reset():
    _check("apml_profile_reset", load().apml_profile_reset())


def apml_profile_read() -> dict:
    ms = (ctypes.c_double * N_PHASES)()
    cnt = (ctypes.c_int64 * N_PHASES)()
    _check("apml_profile_read", load().apml_profile_read(N_PHASES, ms, cnt))
    L = load()
    return {L.apml_phase_name(k).decode(): (ms[k], cnt[k]) for k in range(N_PHASES)}


_torch_alloc_refs = None
# the last exception raised inside the PyTorch-backed allocation callback
torch_alloc_error: Optional[BaseException] = None


def torch_alloc(size, stream, user):
    """Allocation callback of the PyTorch route. A Python exception must never
    cross into C: a ctypes callback that raises hands the caller an undefined
    pointer instead of NULL, so every failure (PyTorch running out of memory
    included) returns NULL, which the library reports as
    APML_ERR_OUT_OF_MEMORY; the exception is kept in torch_alloc_error."""
    global torch_alloc_error
    try:
        p = torch.cuda.caching_allocator_alloc(int(size), torch.cuda.current_device(), stream or 0)
        return int(p) if p else None
    except BaseException as e:  # noqa: BLE001 - nothing may propagate into C
        torch_alloc_error = e
        return None


def torch_free(ptr, size, stream, user):
    """Release callback of the PyTorch route; never raises into C."""
    global torch_alloc_error
    try:
        torch.cuda.caching_allocator_delete(ptr)
    except BaseException as e:  # noqa: BLE001
        torch_alloc_error = e


def apml_set_allocator_torch():
    """Routes libapml's device allocations through PyTorch's caching allocator."""
    global _torch_alloc_refs
    a, f = ALLOC_FN(torch_alloc), FREE_FN(torch_free)
    _check("apml_set_allocator", load().apml_set_allocator(a, f, None))
    _torch_alloc_refs = (a, f)


def apml_set_allocator_default():
    global _torch_alloc_refs
    _check("apml_set_allocator", load().apml_set_allocator(ALLOC_FN(), FREE_FN(), None))
    _torch_alloc_refs = None
