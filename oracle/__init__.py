"""CPU oracle for the sparse APML loss.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The GPU library never
calls it and shares no code with it.

``apml_oracle.c`` holds the computation (double precision, Algorithm 1 of the
paper step by step, hand-written reverse mode); this module only marshals NumPy
arrays in and out through ctypes. ``dense.py`` holds a second, dense
formulation in float64 PyTorch used to pin the C code on tiny inputs.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
import threading
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "apml_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile liboracle.so next to its source with gcc (OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class Params(ctypes.Structure):
    _fields_ = [
        ("p_min", ctypes.c_double),
        ("tau", ctypes.c_double),
        ("eps_stab", ctypes.c_double),
        ("delta", ctypes.c_double),
        ("eps_gap", ctypes.c_double),
        ("eps_dist", ctypes.c_double),
        ("n_iter", ctypes.c_int32),
        ("gap_mode", ctypes.c_int32),    # 0 clamp, 1 uniform fallback
        ("sym_mode", ctypes.c_int32),    # 0 half sum, 1 mean of the present sides
        ("tgrad_mode", ctypes.c_int32),  # 0 full, 1 temperature detached
        ("select_mode", ctypes.c_int32),  # 0 minima decided in float32 (R2), 1 in float64
    ]


DEFAULTS = dict(p_min=0.8, tau=1e-8, eps_stab=1e-8, delta=1e-8, eps_gap=1e-6, eps_dist=1e-12, n_iter=10,
                gap_mode=0, sym_mode=0, tgrad_mode=0, select_mode=0)


def params(**kw) -> Params:
    d = dict(DEFAULTS)
    d.update(kw)
    return Params(d["p_min"], d["tau"], d["eps_stab"], d["delta"], d["eps_gap"], d["eps_dist"],
                  int(d["n_iter"]), int(d["gap_mode"]), int(d["sym_mode"]), int(d["tgrad_mode"]),
                  int(d["select_mode"]))


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER
        dp, ip, bp, lp = P(ctypes.c_double), P(ctypes.c_int32), P(ctypes.c_uint8), P(ctypes.c_int64)
        lib.orc_run.argtypes = [dp, dp, ctypes.c_int, ctypes.c_int, P(Params), ctypes.c_int,
                                ctypes.c_double, ctypes.c_int, P(ctypes.c_void_p)]
        lib.orc_run.restype = ctypes.c_int
        lib.orc_free.argtypes = [ctypes.c_void_p]
        lib.orc_nnz.argtypes = [ctypes.c_void_p]
        lib.orc_nnz.restype = ctypes.c_int64
        lib.orc_loss.argtypes = [ctypes.c_void_p]
        lib.orc_loss.restype = ctypes.c_double
        lib.orc_entries.argtypes = [ctypes.c_void_p, ip, ip, bp, dp, dp, dp, dp, dp]
        lib.orc_row_stats.argtypes = [ctypes.c_void_p, dp, dp, dp, ip, ip, bp]
        lib.orc_col_stats.argtypes = [ctypes.c_void_p, dp, dp, dp, ip, ip, bp]
        lib.orc_last_sums.argtypes = [ctypes.c_void_p, dp, dp]
        lib.orc_grads.argtypes = [ctypes.c_void_p, dp, dp]
        lib.orc_owner_stats.argtypes = [dp, ctypes.c_int, dp, ctypes.c_int, P(Params), ip, ctypes.c_int,
                                        ctypes.c_int, dp, dp, dp, ip, ip, bp, lp]
        lib.orc_owner_stats.restype = ctypes.c_int
        lib.orc_owner_support.argtypes = [dp, ctypes.c_int, dp, ctypes.c_int, P(Params), ctypes.c_int,
                                          ctypes.c_int64, ip, dp, dp]
        lib.orc_owner_support.restype = ctypes.c_int64
        lib.orc_max_threads.argtypes = []
        lib.orc_max_threads.restype = ctypes.c_int
        _lib = lib
        return lib


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _f64(a) -> np.ndarray:
    """Widen float32 coordinates exactly (or take float64 as is) into C order."""
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


@dataclasses.dataclass
class SampleResult:
    loss: float
    nnz: int
    i: np.ndarray
    j: np.ndarray
    flags: np.ndarray  # bit 0: kept by the row softmax, bit 1: kept by the column softmax
    p_row: np.ndarray
    p_col: np.ndarray
    p0: np.ndarray
    v: np.ndarray
    C: np.ndarray
    row: Dict[str, np.ndarray]
    col: Dict[str, np.ndarray]
    colsum_last: Optional[np.ndarray]
    rowsum_last: Optional[np.ndarray]
    grad_x: Optional[np.ndarray]
    grad_y: Optional[np.ndarray]


def _stats(fn, handle, n):
    T, c1, g = np.empty(n), np.empty(n), np.empty(n)
    k1, k2 = np.empty(n, np.int32), np.empty(n, np.int32)
    cl = np.empty(n, np.uint8)
    fn(handle, _ptr(T, ctypes.c_double), _ptr(c1, ctypes.c_double), _ptr(g, ctypes.c_double),
       _ptr(k1, ctypes.c_int32), _ptr(k2, ctypes.c_int32), _ptr(cl, ctypes.c_uint8))
    return dict(T=T, c1=c1, g=g, k1=k1, k2=k2, clamped=cl.astype(bool))


def run_sample(x, y, prm: Optional[Params] = None, grad: bool = True, gbar: float = 1.0,
               threads: int = 0) -> SampleResult:
    """Forward (and backward for upstream gradient gbar) of one sample x (N,3), y (M,3)."""
    lib = _load()
    prm = prm or params()
    x, y = _f64(x), _f64(y)
    N, M = x.shape[0], y.shape[0]
    h = ctypes.c_void_p()
    rc = lib.orc_run(_ptr(x, ctypes.c_double), _ptr(y, ctypes.c_double), N, M, ctypes.byref(prm),
                     int(grad), float(gbar), int(threads), ctypes.byref(h))
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    try:
        n = lib.orc_nnz(h)
        i, j = np.empty(n, np.int32), np.empty(n, np.int32)
        fl = np.empty(n, np.uint8)
        arrs = [np.empty(n) for _ in range(5)]
        lib.orc_entries(h, _ptr(i, ctypes.c_int32), _ptr(j, ctypes.c_int32), _ptr(fl, ctypes.c_uint8),
                        *[_ptr(a, ctypes.c_double) for a in arrs])
        row = _stats(lib.orc_row_stats, h, N)
        col = _stats(lib.orc_col_stats, h, M)
        cs = rs = None
        if prm.n_iter > 0:
            cs, rs = np.empty(M), np.empty(N)
            lib.orc_last_sums(h, _ptr(cs, ctypes.c_double), _ptr(rs, ctypes.c_double))
        gx = gy = None
        if grad:
            gx, gy = np.empty((N, 3)), np.empty((M, 3))
            lib.orc_grads(h, _ptr(gx, ctypes.c_double), _ptr(gy, ctypes.c_double))
        return SampleResult(lib.orc_loss(h), n, i, j, fl, *arrs, row, col, cs, rs, gx, gy)
    finally:
        lib.orc_free(h)


def run_batch(X, Y, prm: Optional[Params] = None, grad: bool = True,
              gbar: Optional[Sequence[float]] = None, threads: int = 0):
    """Per-sample losses (B,) and gradients (B,N,3), (B,M,3) of a batch."""
    X, Y = np.asarray(X), np.asarray(Y)
    B = X.shape[0]
    gb = np.ones(B) if gbar is None else np.asarray(gbar, dtype=np.float64)
    loss = np.empty(B)
    gx = np.empty(X.shape) if grad else None
    gy = np.empty(Y.shape) if grad else None
    for b in range(B):
        r = run_sample(X[b], Y[b], prm, grad=grad, gbar=float(gb[b]), threads=threads)
        loss[b] = r.loss
        if grad:
            gx[b], gy[b] = r.grad_x, r.grad_y
    return loss, gx, gy


def max_threads() -> int:
    """OpenMP threads the oracle uses by default (OMP_NUM_THREADS or all cores)."""
    return int(_load().orc_max_threads())


def owner_stats(P, Q, owners, prm: Optional[Params] = None, threads: int = 0) -> Dict[str, np.ndarray]:
    """Statistics (T, c1, g, k1, k2, clamped) and kept count of sampled owners of P against Q.

    Rows: P = x, Q = y. Columns: P = y, Q = x."""
    lib = _load()
    prm = prm or params()
    P, Q = _f64(P), _f64(Q)
    own = np.ascontiguousarray(owners, dtype=np.int32)
    n = own.shape[0]
    T, c1, g = np.empty(n), np.empty(n), np.empty(n)
    k1, k2 = np.empty(n, np.int32), np.empty(n, np.int32)
    cl, cnt = np.empty(n, np.uint8), np.empty(n, np.int64)
    rc = lib.orc_owner_stats(_ptr(P, ctypes.c_double), P.shape[0], _ptr(Q, ctypes.c_double), Q.shape[0],
                             ctypes.byref(prm), _ptr(own, ctypes.c_int32), n, int(threads),
                             _ptr(T, ctypes.c_double), _ptr(c1, ctypes.c_double), _ptr(g, ctypes.c_double),
                             _ptr(k1, ctypes.c_int32), _ptr(k2, ctypes.c_int32), _ptr(cl, ctypes.c_uint8),
                             _ptr(cnt, ctypes.c_int64))
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    return dict(T=T, c1=c1, g=g, k1=k1, k2=k2, clamped=cl.astype(bool), count=cnt)


def owner_support(P, Q, owner: int, prm: Optional[Params] = None):
    """(indices, s, p) of the kept support of one owner of P against Q."""
    lib = _load()
    prm = prm or params()
    P, Q = _f64(P), _f64(Q)
    n = lib.orc_owner_support(_ptr(P, ctypes.c_double), P.shape[0], _ptr(Q, ctypes.c_double), Q.shape[0],
                              ctypes.byref(prm), int(owner), 0, None, None, None)
    if n < 0:
        raise ValueError("oracle rejected the input")
    idx, s, p = np.empty(n, np.int32), np.empty(n), np.empty(n)
    lib.orc_owner_support(_ptr(P, ctypes.c_double), P.shape[0], _ptr(Q, ctypes.c_double), Q.shape[0],
                          ctypes.byref(prm), int(owner), n, _ptr(idx, ctypes.c_int32),
                          _ptr(s, ctypes.c_double), _ptr(p, ctypes.c_double))
    return idx, s, p
