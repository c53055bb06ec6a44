"""The split streamed Sinkhorn kernels (several workgroups per sample, with a
meeting after every half-sweep; Eq. 3, Eq. 4 and their reverse sweeps)
against the one-workgroup streamed kernels on the same inputs: the loss, both
gradients and the final plan must agree bit for bit (every owner's sum is
formed by the same lanes in the same order), and no meeting's bounded wait
may expire (apml_plan_nnz reports that)."""
import numpy as np
import pytest
import torch

import paper_2512_19743_amd as apml
from workloads import batch, config, custom

from ._parity import note, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    apml.load()


def _run(X, Y, n_iter, mode, monkeypatch):
    # mode "0": one workgroup per sample; "1": split, pieces (or the reverse
    # adjoint) in registers where a workgroup's share allows; "streamed":
    # split, streamed variants only
    monkeypatch.setenv("APML_SINKHORN_SPLIT", mode)
    # an untimed call first: the phase times below are of loaded kernels
    run_gpu(X, Y, n_iter=n_iter)["plan"].close()
    torch.cuda.synchronize()
    apml.apml_profile_reset()
    apml.apml_profile_enable(True)
    g = run_gpu(X, Y, n_iter=n_iter)
    torch.cuda.synchronize()
    apml.apml_profile_enable(False)
    ph = apml.apml_profile_read()
    g["nnz"] = g["plan"].nnz()  # raises if a meeting's wait expired
    g["v"] = [g["plan"].export(b)["v"] for b in range(X.shape[0])]
    g["ms"] = (ph["sinkhorn"][0], ph["bwd_sinkhorn"][0])
    g["plan"].close()
    return g


CASES = {
    # B = 3: eight workgroups per sample, ragged clouds
    "ragged_b3": lambda: custom(71, 3, 3000, 5000, reference="primitives", prediction="perm_noise", sigma=0.05),
    # B = 16 (a multiple of 8: a sample's workgroups on one XCD), 8 per sample
    "b16_n4096": lambda: custom(72, 16, 4096, 4096, reference="primitives", prediction="perm_noise", sigma=0.02),
    # the large-batch workload, 64 x 8192 x 8192: four per sample
    "large_batch": lambda: batch(config(3)),
    # one sample, sizes not multiples of 16: the saved scalings of successive
    # iterations share a cache line at every region boundary
    "b1_n3000": lambda: custom(73, 1, 3000, 3001, reference="primitives", prediction="perm_noise", sigma=0.05),
    # B N below 8192 words: a sample's whole-chunk reads would reach the next
    # iteration's region
    "b2_n3000": lambda: custom(74, 2, 3000, 2999, reference="primitives", prediction="perm_noise", sigma=0.05),
    # one sample with enough pieces for the split forward kernel, B N < 8192
    # (and B not a multiple of 8: seven of the grid's eight rounds end at once)
    "b1_n8000": lambda: custom(75, 1, 8000, 7990, reference="primitives", prediction="perm_noise", sigma=0.02),
    # B = 37 (not a multiple of 8), four workgroups per sample, ragged
    # clouds of 7000 and 6500 points: about three slots per workgroup, the
    # reverse kernel that keeps the adjoint in registers and loads its
    # pieces in every phase
    "b37_ragged": lambda: custom(77, 37, 7000, 6500, reference="primitives", prediction="perm_noise", sigma=0.02),
    # B = 72: three workgroups per sample (a grid of 216), a larger share of
    # each sample's pieces per workgroup
    "b72_n8000": lambda: custom(76, 72, 8000, 8000, reference="primitives", prediction="perm_noise", sigma=0.02),
}


@pytest.mark.parametrize("case", list(CASES))
def test_split_matches_one_workgroup(case, monkeypatch):
    X, Y = CASES[case]()
    n_iter = 20 if case == "large_batch" else 10
    note(f"split streamed Sinkhorn: {case} B={X.shape[0]} N={X.shape[1]} M={Y.shape[1]} L={n_iter}")
    one = _run(X, Y, n_iter, "0", monkeypatch)
    streamed = _run(X, Y, n_iter, "streamed", monkeypatch)
    split = _run(X, Y, n_iter, "1", monkeypatch)
    note(f"{case}: Sinkhorn {one['ms'][0]:.3f} -> {streamed['ms'][0]:.3f} (streamed) / {split['ms'][0]:.3f} ms, "
         f"reverse sweeps {one['ms'][1]:.3f} -> {streamed['ms'][1]:.3f} (streamed) / {split['ms'][1]:.3f} ms")
    for other in (streamed, split):
        np.testing.assert_array_equal(other["nnz"], one["nnz"])
        np.testing.assert_array_equal(other["loss"], one["loss"])
        np.testing.assert_array_equal(other["gx"], one["gx"])
        np.testing.assert_array_equal(other["gy"], one["gy"])
        for b in range(X.shape[0]):
            np.testing.assert_array_equal(other["v"][b], one["v"][b])
        assert np.isfinite(other["loss"]).all()
