"""PyTorch autograd wrapper of the sparse APML loss (forward and backward in libapml)."""
from __future__ import annotations

import torch

from . import _lib


class APMLFunction(torch.autograd.Function):
    """Per-sample sparse APML loss; the plan from the forward call feeds backward."""

    @staticmethod
    def forward(ctx, x, y, params):
        loss, plan = _lib.apml_forward(x, y, params, keep_plan=True)
        ctx.plan = plan
        ctx.save_for_backward(x, y)
        return loss

    @staticmethod
    def backward(ctx, grad_loss):
        x, y = ctx.saved_tensors
        gl = grad_loss.contiguous().to(torch.float32)
        gx, gy = _lib.apml_backward(ctx.plan, x, y, gl, want_grad_y=ctx.needs_input_grad[1])
        return (gx if ctx.needs_input_grad[0] else None), gy, None


_MODES = {
    "dense_scan": {"auto": 0, "full": 1, "skip": 2},
    "gap_mode": {"clamp": 0, "uniform_fallback": 1},
    "sym_mode": {"half_sum": 0, "mean_dup": 1},
    "tgrad_mode": {"full": 0, "detached": 1},
}


def loss_params(*, p_min: float = 0.8, tau: float = 1e-8, n_iter: int = 10, eps_stab: float = 1e-8,
                delta: float = 1e-8, eps_gap: float = 1e-6, eps_dist: float = 1e-12, dense_scan: str = "auto",
                gap_mode: str = "clamp", sym_mode: str = "half_sum", tgrad_mode: str = "full") -> _lib.apml_params:
    """apml_params from keyword values; the modes are given by name (see include/apml.h)."""
    modes = {}
    for field, value in (("dense_scan", dense_scan), ("gap_mode", gap_mode), ("sym_mode", sym_mode),
                         ("tgrad_mode", tgrad_mode)):
        table = _MODES[field]
        if value not in table:
            raise ValueError(f"{field} must be one of {sorted(table)}, got {value!r}")
        modes[field] = table[value]
    return _lib.apml_params_default(p_min=p_min, tau=tau, n_iter=n_iter, eps_stab=eps_stab, delta=delta,
                                    eps_gap=eps_gap, eps_dist=eps_dist, **modes)


def apml_loss(x: torch.Tensor, y: torch.Tensor, *, reduction: str = "mean", **params) -> torch.Tensor:
    """Sparse APML between predicted x (B,N,3) and reference y (B,M,3) float32 GPU tensors.

    params: the keywords of loss_params (p_min, tau, n_iter, eps_stab, delta,
    eps_gap, eps_dist, dense_scan, gap_mode, sym_mode, tgrad_mode).
    reduction: 'none' (per-sample losses), 'sum' or 'mean' over the batch.
    """
    if reduction not in ("none", "sum", "mean"):
        raise ValueError(f"unknown reduction {reduction!r}")
    per = APMLFunction.apply(x.contiguous(), y.contiguous(), loss_params(**params))
    if reduction == "none":
        return per
    if reduction == "sum":
        return per.sum()
    if reduction == "mean":
        return per.mean()
    raise ValueError(f"unknown reduction {reduction!r}")
