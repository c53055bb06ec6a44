"""The two builds of the column-major view (the column softmax of Eq. 2 and
the column half-sweeps of Eq. 4 read the plan through it): per sample in LDS,
in column ranges, against slots taken through global counters. Both order a
column's entries by row, so the loss, both gradients and the exported plan
must agree bit for bit."""
import numpy as np
import pytest
import torch

import paper_2512_19743_amd as apml
from workloads import batch, config, custom

from ._parity import note, run_gpu

pytestmark = pytest.mark.gpu

CASES = {
    "ragged_b3": lambda: custom(41, 3, 300, 517, reference="sphere", prediction="uniform_cube"),
    "odd_m3": lambda: custom(42, 1, 65, 3, reference="sphere", prediction="uniform_cube"),
    "unequal_b2": lambda: custom(43, 2, 700, 2100, reference="primitives", prediction="uniform_cube"),
    "shape_completion_b32_n2048": lambda: batch(config(2)),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    apml.load()


def _run(X, Y, mode, monkeypatch):
    if mode is None:
        monkeypatch.delenv("APML_CSC", raising=False)
    else:
        monkeypatch.setenv("APML_CSC", mode)
    g = run_gpu(X, Y, n_iter=10)
    g["nnz"] = g["plan"].nnz()
    g["export"] = [g["plan"].export(b) for b in range(X.shape[0])]
    g["plan"].close()
    return g


@pytest.mark.parametrize("case", list(CASES))
def test_lds_and_global_column_views_agree(case, monkeypatch):
    X, Y = CASES[case]()
    note(f"column-major view builds: {case} B={X.shape[0]} N={X.shape[1]} M={Y.shape[1]}")
    lds = _run(X, Y, None, monkeypatch)
    glob = _run(X, Y, "global", monkeypatch)
    np.testing.assert_array_equal(glob["nnz"], lds["nnz"])
    np.testing.assert_array_equal(glob["loss"], lds["loss"])
    np.testing.assert_array_equal(glob["gx"], lds["gx"])
    np.testing.assert_array_equal(glob["gy"], lds["gy"])
    for eg, el in zip(glob["export"], lds["export"]):
        assert eg.keys() == el.keys()
        for k in el:
            np.testing.assert_array_equal(eg[k], el[k], err_msg=k)
