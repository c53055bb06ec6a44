"""Dense float64 PyTorch formulation of the (thresholded) APML loss.

TEST INFRASTRUCTURE, tiny inputs only. It restates the same definition as
``apml_oracle.c`` in matrix form over all N x M pairs, so that PyTorch autograd
can differentiate it: a check of the hand-written reverse mode that does not
share its derivation. With tau = 0 it is dense APML (Sec. III-A) with the gap
clamp of Sec. III-D; with tau > 0 the pruned entries are zeros of the masks of
Sec. III-B and the plan is the symmetrized sparse plan of Sec. III-C.

The two argmins per row and per column are inputs (the C oracle decides them
in single precision); when omitted they are decided here in double precision.
"""
from __future__ import annotations

import math
from typing import Optional, Tuple

import torch


def _two_smallest(C: torch.Tensor, dim: int) -> Tuple[torch.Tensor, torch.Tensor]:
    idx = torch.topk(C.detach(), 2, dim=dim, largest=False, sorted=True).indices
    return (idx[:, 0], idx[:, 1]) if dim == 1 else (idx[0, :], idx[1, :])


def dense_apml(x: torch.Tensor, y: torch.Tensor, *, p_min=0.8, tau=1e-8, n_iter=10, eps_stab=1e-8,
               delta=1e-8, eps_gap=1e-6, row_argmins: Optional[Tuple] = None,
               col_argmins: Optional[Tuple] = None, gap_mode=0, sym_mode=0, tgrad_mode=0):
    """Loss and intermediate matrices for x (N,3), y (M,3) float64 tensors.

    gap_mode 1: an owner whose gap C2 - C1 is below eps_gap gets the uniform
    distribution 1/K over all K entries (a constant). sym_mode 1: P0 is the
    mean of the directions that keep a pair. tgrad_mode 1: the temperatures
    are constants (detached)."""
    N, M = x.shape[0], y.shape[0]
    C = torch.sqrt(((x[:, None, :] - y[None, :, :]) ** 2).sum(-1))  # Sec. III-A
    rN, rM = torch.arange(N), torch.arange(M)

    j1, j2 = row_argmins if row_argmins is not None else _two_smallest(C, 1)
    i1, i2 = col_argmins if col_argmins is not None else _two_smallest(C, 0)
    j1, j2, i1, i2 = (torch.as_tensor(a, dtype=torch.long) for a in (j1, j2, i1, i2))

    def temperature(c1, c2, K):
        gap = c2 - c1 + delta
        g = torch.where(gap < eps_gap, torch.full_like(gap, eps_gap), gap)  # Sec. III-D clamp
        T = math.log((K - 1) * p_min / (1 - p_min)) / g  # Eq. 1
        return T.detach() if tgrad_mode == 1 else T

    def fallback(c1, c2):  # uniform fallback (Sec. III-A) where the raw gap is below eps_gap
        if gap_mode != 1:
            return torch.zeros_like(c1, dtype=torch.bool)
        return ((c2 - c1) < eps_gap).detach()

    c1r = C[rN, j1]
    Tr = temperature(c1r, C[rN, j2], M)
    s_row = torch.exp(-Tr[:, None] * (C - c1r[:, None]))  # Sec. III-B
    keep_r = (s_row >= tau).detach()
    kr = torch.where(keep_r, s_row, torch.zeros_like(s_row))
    P_row = kr / kr.sum(1, keepdim=True)  # kept-sum normalisation (Sec. III-C)
    fb_r = fallback(c1r, C[rN, j2])
    P_row = torch.where(fb_r[:, None], torch.full_like(P_row, 1.0 / M), P_row)
    keep_r = keep_r | fb_r[:, None]

    c1c = C[i1, rM]
    Tc = temperature(c1c, C[i2, rM], N)
    s_col = torch.exp(-Tc[None, :] * (C - c1c[None, :]))
    keep_c = (s_col >= tau).detach()
    kc = torch.where(keep_c, s_col, torch.zeros_like(s_col))
    P_col = kc / kc.sum(0, keepdim=True)
    fb_c = fallback(c1c, C[i2, rM])
    P_col = torch.where(fb_c[None, :], torch.full_like(P_col, 1.0 / N), P_col)
    keep_c = keep_c | fb_c[None, :]

    if sym_mode == 1:  # duplicates averaged, a single value kept as is
        P0 = torch.where(keep_r & keep_c, 0.5 * (P_row + P_col), P_row + P_col)
    else:
        P0 = 0.5 * (P_row + P_col)  # initial plan on the union support
    P = P0
    for _ in range(n_iter):  # Eq. 3 then Eq. 4
        P = P / (P.sum(0, keepdim=True) + eps_stab)
        P = P / (P.sum(1, keepdim=True) + eps_stab)
    loss = (P * C).sum()
    return loss, dict(C=C, P_row=P_row, P_col=P_col, P0=P0, P=P, keep_row=keep_r, keep_col=keep_c,
                      T_row=Tr, T_col=Tc)
