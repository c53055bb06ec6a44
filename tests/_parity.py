"""Helpers for the GPU parity tests: run the C-ABI path and the oracle on the
same seeded float32 inputs and compare them at the stated tolerances.

Tolerances (float32 inputs, float32 outputs):
  loss         relative 1e-5 per sample
  gradients    normwise relative 1e-4 per sample, ||g_gpu - g_ref|| / ||g_ref||; the
               largest per-point error max_i ||g_gpu,i - g_ref,i|| / ||g_ref|| is
               reported beside it (it is bounded by the normwise figure)
  support      identical, except pairs whose oracle similarity lies within
               1e-6 (absolute) of tau for the flag that differs
  indices      bit-exact (i, j) on the agreed support and for the argmins
  P_row, P_col, P0   relative 2e-6 (single-precision storage of double values)
  temperatures relative 1e-12 (double precision on both sides)
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import paper_2512_19743_amd as apml

LOSS_RTOL = 1e-5
GRAD_RTOL = 1e-4
SUPPORT_BAND = 1e-6
PROB_RTOL = 2e-6


def note(msg: str):
    """Progress line that bypasses pytest's capture, flushed before GPU work."""
    sys.__stdout__.write(f"[gpu] {msg}\n")
    sys.__stdout__.flush()


def oracle_params(**kw):
    return oracle.params(**kw)


def gpu_params(**kw):
    return apml.apml_params_default(**kw)


def run_gpu(X, Y, want_grad_y=True, gbar=None, **prm):
    x = torch.from_numpy(np.ascontiguousarray(X)).cuda()
    y = torch.from_numpy(np.ascontiguousarray(Y)).cuda()
    loss, plan = apml.apml_forward(x, y, gpu_params(**prm))
    gl = torch.ones(x.shape[0], device="cuda") if gbar is None else torch.tensor(gbar, dtype=torch.float32,
                                                                                 device="cuda")
    gx, gy = apml.apml_backward(plan, x, y, gl, want_grad_y=want_grad_y)
    torch.cuda.synchronize()
    return dict(loss=loss.cpu().numpy().astype(np.float64), gx=gx.cpu().numpy().astype(np.float64),
                gy=None if gy is None else gy.cpu().numpy().astype(np.float64), plan=plan)


def rel_norm(a, b):
    den = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (den if den > 0 else 1.0)


def row_max_rel(a, b):
    """Largest per-point error of a gradient, relative to the norm of the whole reference gradient."""
    den = np.linalg.norm(b)
    return float(np.max(np.linalg.norm(a - b, axis=-1)) / (den if den > 0 else 1.0))


def _similarity(T, c1, C):
    return np.exp(-T * (C - c1))


def compare_sample(g: dict, b: int, x: np.ndarray, y: np.ndarray, ref: oracle.SampleResult, tau: float,
                   check_grad_y: bool = True, prob_rtol: float = PROB_RTOL, grad_rtol: float = GRAD_RTOL):
    """Element-by-element comparison of sample b of a GPU run with the oracle."""
    N, M = x.shape[0], y.shape[0]
    plan: apml.Plan = g["plan"]
    # loss and gradients
    loss_rel = abs(g["loss"][b] - ref.loss) / abs(ref.loss)
    assert loss_rel <= LOSS_RTOL, (b, g["loss"][b], ref.loss)
    gx_rel = rel_norm(g["gx"][b], ref.grad_x)
    assert gx_rel <= grad_rtol, (b, "grad_x", gx_rel)
    gx_row = row_max_rel(g["gx"][b], ref.grad_x)
    gy_rel = gy_row = 0.0
    if check_grad_y and g["gy"] is not None:
        gy_rel = rel_norm(g["gy"][b], ref.grad_y)
        assert gy_rel <= grad_rtol, (b, "grad_y", gy_rel)
        gy_row = row_max_rel(g["gy"][b], ref.grad_y)
    # statistics: argmins bit-exact, temperatures to double precision
    st = plan.export_stats(b)
    np.testing.assert_array_equal(st["j1"], ref.row["k1"])
    np.testing.assert_array_equal(st["j2"], ref.row["k2"])
    np.testing.assert_array_equal(st["i1"], ref.col["k1"])
    np.testing.assert_array_equal(st["i2"], ref.col["k2"])
    np.testing.assert_array_equal(st["clamp_row"], ref.row["clamped"])
    np.testing.assert_array_equal(st["clamp_col"], ref.col["clamped"])
    np.testing.assert_allclose(st["T_row"], ref.row["T"], rtol=1e-12)
    np.testing.assert_allclose(st["T_col"], ref.col["T"], rtol=1e-12)
    # support
    ex = plan.export(b)
    gk = ex["i"].astype(np.int64) * M + ex["j"]
    ok = ref.i.astype(np.int64) * M + ref.j
    assert np.all(np.diff(gk) > 0), "export must be sorted by (i, j) without duplicates"
    x64, y64 = x.astype(np.float64), y.astype(np.float64)

    def s_pair(keys):
        i, j = keys // M, keys % M
        C = np.linalg.norm(x64[i] - y64[j], axis=1)
        return (_similarity(ref.row["T"][i], ref.row["c1"][i], C),
                _similarity(ref.col["T"][j], ref.col["c1"][j], C))

    flips = 0
    for keys, flags in ((np.setdiff1d(gk, ok), None), (np.setdiff1d(ok, gk), None)):
        if keys.size:
            sr, sc = s_pair(keys)
            near = (np.abs(sr - tau) <= SUPPORT_BAND) | (np.abs(sc - tau) <= SUPPORT_BAND)
            assert near.all(), f"sample {b}: {int((~near).sum())} support differences outside the band"
            flips += keys.size
    common, gi, oi = np.intersect1d(gk, ok, return_indices=True)
    fg, fo = ex["flags"][gi], ref.flags[oi]
    diff = fg != fo
    if diff.any():
        sr, sc = s_pair(common[diff])
        rowd = (fg[diff] & 1) != (fo[diff] & 1)
        cold = (fg[diff] & 2) != (fo[diff] & 2)
        ok_r = ~rowd | (np.abs(sr - tau) <= SUPPORT_BAND)
        ok_c = ~cold | (np.abs(sc - tau) <= SUPPORT_BAND)
        assert (ok_r & ok_c).all(), f"sample {b}: flag differences outside the band"
        flips += int(diff.sum())
    same = ~diff
    for name, gv, ov in (("p_row", ex["p_row"], ref.p_row), ("p_col", ex["p_col"], ref.p_col),
                         ("p0", ex["p0"], ref.p0)):
        a, r = gv[gi][same].astype(np.float64), ov[oi][same]
        bad = np.abs(a - r) > prob_rtol * np.abs(r) + 1e-30
        assert not bad.any(), (b, name, int(bad.sum()), float(np.max(np.abs(a - r) / np.maximum(np.abs(r), 1e-300))))
    v_err = rel_norm(ex["v"][gi].astype(np.float64), ref.v[oi])
    assert v_err <= 1e-5, (b, "v", v_err)
    return dict(nnz_gpu=len(gk), nnz_ref=ref.nnz, flips=flips, loss_rel=loss_rel, gx_rel=gx_rel, gy_rel=gy_rel,
                gx_row=gx_row, gy_row=gy_row, v_rel=v_err)
