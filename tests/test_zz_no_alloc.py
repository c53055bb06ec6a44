"""apml_forward_backward_noalloc (the entry point that allocates nothing)
against apml_forward + apml_backward, through the C ABI on the GPU: two calls
in a row, the second on a smaller input, each compared with the allocating
entry points at the parity tolerances and bit for bit (the same kernels run
on the same inputs); a call too large for the static scratch is rejected
before it writes its outputs."""
import numpy as np
import pytest
import torch

import paper_2512_19743_amd as apml
from workloads import batch, config

from ._parity import LOSS_RTOL, GRAD_RTOL, note, rel_norm

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    apml.load()


def _allocating(x, y, prm, gl):
    loss, plan = apml.apml_forward(x, y, prm)
    gx, gy = apml.apml_backward(plan, x, y, gl, want_grad_y=True)
    torch.cuda.synchronize()
    plan.close()
    return loss.cpu().numpy(), gx.cpu().numpy(), gy.cpu().numpy()


def test_noalloc_matches_the_allocating_entry_points_twice():
    for cfg in (2, 1):  # shape-completion (32 x 2048 x 2048), then the tiny workload (2 x 256 x 256)
        w = config(cfg)
        X, Y = batch(w)
        note(f"no-alloc {w.name}: B={w.B} N={w.N} M={w.M}")
        x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
        prm = apml.apml_params_default(n_iter=w.n_iter)
        gl = torch.linspace(0.5, 1.5, w.B, device="cuda")
        ref_loss, ref_gx, ref_gy = _allocating(x, y, prm, gl)
        before = apml.apml_get_memory_stats()
        loss, gx, gy = apml.apml_forward_backward_noalloc(x, y, prm, grad_loss=gl, want_grad_y=True)
        torch.cuda.synchronize()
        after = apml.apml_get_memory_stats()
        assert after == before, "the no-alloc call must not touch the library's device memory pool"
        loss, gx, gy = loss.cpu().numpy(), gx.cpu().numpy(), gy.cpu().numpy()
        for b in range(w.B):
            assert abs(loss[b] - ref_loss[b]) <= LOSS_RTOL * abs(ref_loss[b])
            assert rel_norm(gx[b].astype(np.float64), ref_gx[b].astype(np.float64)) <= GRAD_RTOL
            assert rel_norm(gy[b].astype(np.float64), ref_gy[b].astype(np.float64)) <= GRAD_RTOL
        assert np.array_equal(loss, ref_loss) and np.array_equal(gx, ref_gx) and np.array_equal(gy, ref_gy)
        # the loss alone
        loss_only, none_x, none_y = apml.apml_forward_backward_noalloc(x, y, prm, want_grad=False)
        assert none_x is None and none_y is None
        assert np.array_equal(loss_only.cpu().numpy(), ref_loss)


def test_noalloc_rejects_a_call_beyond_its_scratch():
    w = config(3)  # 64 clouds of 8192 points: far more than the static scratch holds
    X, Y = batch(w)
    note(f"no-alloc too large: B={w.B} N={w.N} M={w.M}")
    x, y = torch.from_numpy(X).cuda(), torch.from_numpy(Y).cuda()
    loss = torch.full((w.B,), 7.0, device="cuda")
    gx = torch.full_like(x, 7.0)
    lib = apml.load()
    import ctypes
    prm = apml.apml_params_default(n_iter=w.n_iter)
    st = lib.apml_forward_backward_noalloc(
        ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), w.B, w.N, w.M, 3, ctypes.byref(prm),
        ctypes.c_void_p(loss.data_ptr()), ctypes.c_void_p(torch.ones(w.B, device="cuda").data_ptr()),
        ctypes.c_void_p(gx.data_ptr()), None, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert st == 3, (st, lib.apml_last_error().decode())
    assert "APML_NOALLOC_SCRATCH_BYTES" in lib.apml_last_error().decode()
    assert (loss == 7.0).all() and (gx == 7.0).all()
    # and a call that fits still works after the rejection
    w1 = config(1)
    X1, Y1 = batch(w1)
    x1, y1 = torch.from_numpy(X1).cuda(), torch.from_numpy(Y1).cuda()
    prm1 = apml.apml_params_default(n_iter=w1.n_iter)
    ref_loss, ref_gx, _ = _allocating(x1, y1, prm1, torch.ones(w1.B, device="cuda"))
    l1, g1, _ = apml.apml_forward_backward_noalloc(x1, y1, prm1)
    assert np.array_equal(l1.cpu().numpy(), ref_loss) and np.array_equal(g1.cpu().numpy(), ref_gx)
