"""GPU parity: the C-ABI path (libapml on the MI355X) against the CPU oracle,
element by element on seeded inputs. Tolerances are in tests/_parity.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2512_19743_amd as apml
from workloads import batch, config, custom

from ._parity import GRAD_RTOL, compare_sample, note, oracle_params, rel_norm, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    apml.load()


# the two ways the dense scans visit the pairs (identical results): every
# pair, or skipping runs of the spatially sorted clouds that cannot matter
SCANS = {"full": 1, "skip": 2}


def _check_batch(X, Y, label, samples=None, check_grad_y=True, scan=None, grad_rtol=GRAD_RTOL, **prm):
    note(f"{label}: B={X.shape[0]} N={X.shape[1]} M={Y.shape[1]} {prm} scan={scan or 'auto'}")
    g = run_gpu(X, Y, **prm, **({} if scan is None else {"dense_scan": SCANS[scan]}))
    tau = prm.get("tau", 1e-8)
    out = []
    for b in (range(X.shape[0]) if samples is None else samples):
        ref = oracle.run_sample(X[b], Y[b], oracle_params(**prm), grad=True)
        out.append(compare_sample(g, b, X[b], Y[b], ref, tau, check_grad_y=check_grad_y, grad_rtol=grad_rtol))
    worst = {k: max(r[k] for r in out) for k in ("loss_rel", "gx_rel", "gy_rel", "gx_row", "gy_row", "v_rel")}
    note(f"{label}: worst relative errors " + ", ".join(f"{k} {v:.2e}" for k, v in worst.items()))
    return g, out


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_tiny_workload_full(scan):
    w = config(1)
    X, Y = batch(w)
    _, res = _check_batch(X, Y, w.name, n_iter=w.n_iter, scan=scan)
    assert all(r["flips"] == 0 for r in res), res


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_ragged_unequal_sizes(scan):
    # sizes that are not multiples of the wave, the workgroup or the chunk
    X, Y = custom(21, 3, 300, 517, reference="sphere", prediction="uniform_cube")
    _check_batch(X, Y, "ragged", n_iter=7, scan=scan)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_unequal_cardinality_primitives(scan):
    X, Y = custom(22, 2, 700, 2100, reference="primitives", prediction="uniform_cube")
    _check_batch(X, Y, "unequal", n_iter=10, scan=scan)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_minimum_size(scan):
    X, Y = custom(23, 4, 2, 2, sigma=0.1)
    _check_batch(X, Y, "N=M=2", n_iter=10, scan=scan)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_single_sample_odd_shapes(scan):
    X, Y = custom(24, 1, 65, 3, reference="sphere", prediction="uniform_cube")
    _check_batch(X, Y, "N=65 M=3", n_iter=3, scan=scan)


@pytest.mark.parametrize("L", [1, 3, 10])
def test_streamed_per_sample_sinkhorn(L):
    # clouds of 2048 < N, M <= 8192 points: one workgroup per sample runs every
    # Sinkhorn sweep with the pieces streamed from memory (ragged sizes)
    X, Y = custom(37, 3, 3000, 5000, reference="primitives", prediction="perm_noise", sigma=0.05)
    _check_batch(X, Y, f"streamed sweeps L={L}", n_iter=L)


def test_per_iteration_sweeps_twenty_iterations():
    # clouds beyond 8192 points: one launch per Sinkhorn half-sweep, with the
    # per-point factors gathered in single precision; 20 iterations, as the
    # large-batch workload
    X, Y = custom(38, 1, 9000, 9000, reference="primitives", prediction="perm_noise", sigma=0.01)
    _check_batch(X, Y, "per-iteration sweeps L=20", n_iter=20)


@pytest.mark.parametrize("L", [0, 1, 20])
def test_iteration_counts(L):
    X, Y = custom(25, 2, 200, 180, sigma=0.05)
    _check_batch(X, Y, f"L={L}", n_iter=L)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_dense_threshold_zero_full_support(scan):
    # tau = 0 keeps every pair: no run of the support scan can be skipped and
    # every row holds all M columns
    X, Y = custom(26, 1, 400, 400, sigma=0.05)
    g, res = _check_batch(X, Y, "tau=0", tau=0.0, n_iter=5, scan=scan)
    assert res[0]["nnz_gpu"] == 400 * 400


# Further hits of the full support scan (beyond a (row, chunk)'s slots): 1024
# rows against 4096 columns in 16 chunks of 256, 4 slots each, tiles of 256
# rows. Mean candidates per row (oracle support): about 20 (uniform
# predictions, tau 1e-8: every tile's further hits fit its list and the pool),
# about 118 (tau 1e-30: tiles need more than the pool's average share, so the
# later ones find it full and are scanned again) and about 241 (more than the
# 2048 hits a tile's list holds: scanned again).
#
# The first case also holds a row almost equidistant from its two nearest
# columns: its gap term (Eq. 1: the temperature adjoint times T / g) gives
# those two columns gradients of about 206 each, 70% of the gradient's norm.
# The reverse sweeps that keep a sample in LDS store the adjoint and the
# exchanged per-point factors in single precision, and that term inherits
# their rounding: 1.0e-4 normwise with L = 3 (the sweeps that keep them in
# double, 9e-8 on the same input; with no iterations, 3e-8). Its gradients
# are held to 2e-4, the other cases to the general 1e-4.
@pytest.mark.parametrize("prediction,sigma,tau,grad_rtol", [("uniform_cube", 0.0, 1e-8, 2e-4),
                                                            ("perm_noise", 0.05, 1e-30, GRAD_RTOL),
                                                            ("uniform_cube", 0.0, 1e-30, GRAD_RTOL)])
def test_support_scan_further_hits(prediction, sigma, tau, grad_rtol):
    X, Y = custom(90, 1, 1024, 4096, reference="primitives", prediction=prediction, sigma=sigma)
    _check_batch(X, Y, f"further hits {prediction} tau={tau}", tau=tau, n_iter=3, scan="full",
                 grad_rtol=grad_rtol)


def test_temperature_gradient_near_tie_without_iterations():
    # the near-degenerate sample above with L = 0: the loss is sum P0 C, and
    # the backward forms P in double precision, so the gap terms that T / g
    # amplifies keep their digits (stored single-precision P gave 5.5e-4)
    X, Y = custom(90, 1, 1024, 4096, reference="primitives", prediction="uniform_cube", sigma=0.0)
    _, res = _check_batch(X, Y, "near tie, L = 0", n_iter=0, scan="full")
    assert res[0]["gy_rel"] <= 1e-6, res[0]


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_threshold_one_is_half_chamfer(scan):
    X, Y = custom(27, 2, 150, 170, sigma=0.05)
    g, _ = _check_batch(X, Y, "tau=1", tau=1.0, n_iter=0, scan=scan)
    for b in range(2):
        D = np.linalg.norm(X[b].astype(np.float64)[:, None] - Y[b].astype(np.float64)[None], axis=-1)
        assert g["loss"][b] == pytest.approx(0.5 * (D.min(1).sum() + D.min(0).sum()), rel=1e-5)


@pytest.mark.parametrize("p_min", [0.5, 0.95])
def test_other_p_min(p_min):
    X, Y = custom(28, 2, 256, 256, sigma=0.03)
    _check_batch(X, Y, f"p_min={p_min}", p_min=p_min)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_duplicates_ties_and_clamps(scan):
    X, Y = custom(29, 2, 128, 100, sigma=0.05)
    Y = np.ascontiguousarray(np.concatenate([Y, Y[:, :30]], axis=1))  # exact ties
    X = np.ascontiguousarray(np.concatenate([X, X[:, :10]], axis=1))
    g, _ = _check_batch(X, Y, "ties", scan=scan)
    st = g["plan"].export_stats(0)
    assert st["clamp_row"].any() and st["clamp_col"].any()


# readings of the paper where it offers two (the defaults are clamp, half sum,
# full gradient)
VARIANTS = {"fallback": dict(gap_mode=1), "mean_dup": dict(sym_mode=1), "detached": dict(tgrad_mode=1),
            "all": dict(gap_mode=1, sym_mode=1, tgrad_mode=1)}


@pytest.mark.parametrize("scan", ["full", "skip"])
@pytest.mark.parametrize("variant", list(VARIANTS))
def test_reading_variants_with_ties(variant, scan):
    # duplicated points: their rows and columns tie, so the uniform fallback
    # takes whole rows and columns into the support
    X, Y = custom(34, 2, 128, 100, sigma=0.05)
    Y = np.ascontiguousarray(np.concatenate([Y, Y[:, :30]], axis=1))
    X = np.ascontiguousarray(np.concatenate([X, X[:, :10]], axis=1))
    g, _ = _check_batch(X, Y, f"variant {variant}", scan=scan, **VARIANTS[variant])
    if VARIANTS[variant].get("gap_mode") == 1:
        st = g["plan"].export_stats(0)
        ex = g["plan"].export(0)
        rows = np.flatnonzero(st["T_row"] == 0)
        assert rows.size > 0
        per_row = np.bincount(ex["i"], minlength=X.shape[1])
        assert (per_row[rows] == Y.shape[1]).all()
        sel = np.isin(ex["i"], rows)
        np.testing.assert_allclose(ex["p_row"][sel], 1.0 / Y.shape[1], rtol=1e-6)


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_fallback_rows_take_the_per_iteration_path(scan):
    # every reference point doubled: every row falls back to all 1200 columns,
    # too many pieces for the per-sample Sinkhorn kernels, so the sweeps take
    # one launch each
    X, Y = custom(35, 1, 700, 600, sigma=0.05, reference="sphere", prediction="uniform_cube")
    Y = np.ascontiguousarray(np.concatenate([Y, Y], axis=1))
    g, res = _check_batch(X, Y, "fallback, whole rows", scan=scan, n_iter=5, **VARIANTS["all"])
    st = g["plan"].export_stats(0)
    assert (st["T_row"] == 0).all()
    assert res[0]["nnz_gpu"] >= 700 * 1200


@pytest.mark.parametrize("variant", ["mean_dup", "detached"])
def test_reading_variants_tiny(variant):
    w = config(1)
    X, Y = batch(w)
    _check_batch(X, Y, f"{w.name} {variant}", n_iter=w.n_iter, **VARIANTS[variant])


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_identical_clouds(scan):
    _, Y = custom(30, 2, 300, 300, sigma=0.05)
    _check_batch(Y.copy(), Y, "x == y", scan=scan)


def test_upstream_gradient_scaling():
    X, Y = custom(31, 3, 128, 128, sigma=0.05)
    gbar = np.array([1.0, -2.5, 0.0], np.float32)
    note("upstream gradient")
    g = run_gpu(X, Y, gbar=gbar)
    for b in range(3):
        ref = oracle.run_sample(X[b], Y[b], oracle_params(), grad=True, gbar=float(gbar[b]))
        if gbar[b] == 0:
            assert np.all(g["gx"][b] == 0)
        else:
            assert rel_norm(g["gx"][b], ref.grad_x) <= 1e-4


@pytest.mark.parametrize("scan", ["full", "skip"])
def test_deterministic_bitwise(scan):
    X, Y = batch(config(1))
    note(f"determinism scan={scan}")
    a = run_gpu(X, Y, dense_scan=SCANS[scan])
    b = run_gpu(X, Y, dense_scan=SCANS[scan])
    assert np.array_equal(a["loss"], b["loss"])
    assert np.array_equal(a["gx"], b["gx"]) and np.array_equal(a["gy"], b["gy"])


def test_autograd_wrapper_mean_reduction():
    X, Y = custom(32, 4, 96, 80, sigma=0.05)
    note("autograd wrapper")
    x = torch.from_numpy(X).cuda().requires_grad_(True)
    y = torch.from_numpy(Y).cuda().requires_grad_(True)
    loss = apml.apml_loss(x, y, reduction="mean")
    loss.backward()
    ref_l, ref_gx, ref_gy = oracle.run_batch(X, Y, oracle_params(), grad=True)
    assert loss.item() == pytest.approx(ref_l.mean(), rel=1e-5)
    assert rel_norm(x.grad.cpu().numpy().astype(np.float64), ref_gx / 4) <= 1e-4
    assert rel_norm(y.grad.cpu().numpy().astype(np.float64), ref_gy / 4) <= 1e-4


def test_autograd_wrapper_variant_by_name():
    X, Y = custom(36, 2, 120, 110, sigma=0.05)
    note("autograd wrapper, variants")
    x = torch.from_numpy(X).cuda().requires_grad_(True)
    y = torch.from_numpy(Y).cuda()
    loss = apml.apml_loss(x, y, reduction="sum", sym_mode="mean_dup", tgrad_mode="detached", n_iter=5)
    loss.backward()
    ref_l, ref_gx, _ = oracle.run_batch(X, Y, oracle_params(n_iter=5, sym_mode=1, tgrad_mode=1), grad=True)
    assert loss.item() == pytest.approx(ref_l.sum(), rel=1e-5)
    assert rel_norm(x.grad.cpu().numpy().astype(np.float64), ref_gx) <= 1e-4


def test_rejects_bad_input_on_gpu():
    x = torch.zeros(2, 8, 3, device="cuda")
    with pytest.raises(apml.ApmlError):
        apml.apml_forward(x, torch.zeros(2, 1, 3, device="cuda"))
    with pytest.raises(ValueError):
        apml.apml_forward(x.double(), x.double())


def test_plan_reports_and_memory_returns():
    X, Y = custom(33, 2, 256, 256, sigma=0.05)
    note("plan info")
    before = apml.apml_get_memory_stats()["in_use"]
    g = run_gpu(X, Y)
    info = g["plan"].info()
    assert info.B == 2 and info.N == 256 and info.stored_pairs >= g["plan"].nnz().sum()
    assert apml.apml_get_memory_stats()["in_use"] - before == info.bytes
    g["plan"].close()
    assert apml.apml_get_memory_stats()["in_use"] == before


# ---------------------------------------------------------------------------
# full-size configurations, in the launch configuration the benchmark times
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("scan", ["full", "skip"])
def test_shape_completion_full_batch(scan):
    w = config(2)
    X, Y = batch(w)
    _, res = _check_batch(X, Y, w.name, n_iter=w.n_iter, scan=scan)
    note(f"{w.name} nnz per sample: {[r['nnz_gpu'] for r in res[:4]]} flips {sum(r['flips'] for r in res)}")


@pytest.mark.parametrize("cfg,scan", [(3, None), (4, None), (4, "full"), (4, "skip")])
def test_large_workloads_one_sample_exact(cfg, scan):
    # the whole batch runs on the GPU; sample 0 is checked against a full oracle run
    w = config(cfg)
    X, Y = batch(w)
    _check_batch(X, Y, w.name, samples=[0], n_iter=w.n_iter, scan=scan)


@pytest.mark.parametrize("cfg,sample", [(3, 63), (4, 15), (5, 0), (5, 3)])
def test_large_workloads_exact_sample(cfg, sample):
    # the whole batch on the GPU in the benchmark's launch configuration
    # (automatic scan mode: skipping scans for the large batch and the large
    # scene, per-iteration Sinkhorn sweeps for all three); one sample against
    # a full oracle run: the last sample of the large batch and of the unequal
    # workload (the largest row, column and pair offsets), the first and the
    # last sample of the large scene
    w = config(cfg)
    X, Y = batch(w)
    _check_batch(X, Y, w.name, samples=[sample], n_iter=w.n_iter)


def test_large_scene_sampled_owners_and_invariants():
    w = config(5)
    X, Y = batch(w)
    note(w.name)
    g = run_gpu(X, Y, n_iter=w.n_iter)
    plan = g["plan"]
    nnz = plan.nnz()
    prm = oracle_params(n_iter=w.n_iter)
    rng = np.random.default_rng(5)
    for b in range(w.B):
        assert np.isfinite(g["loss"][b]) and g["loss"][b] > 0
        # translation invariance of the loss: the gradients sum to zero
        scale = np.abs(g["gx"][b]).sum() + np.abs(g["gy"][b]).sum()
        assert np.abs(g["gx"][b].sum(0) + g["gy"][b].sum(0)).max() <= 1e-4 * scale
    for b in (0, w.B - 1):
        ex = plan.export(b)
        st = plan.export_stats(b)
        # P0 has mass (N + M)/2: every row of P_row and every column of P_col sums to 1
        assert ex["p0"].astype(np.float64).sum() == pytest.approx((w.N + w.M) / 2, rel=1e-5)
        assert len(ex["i"]) == nnz[b]
        rows = rng.choice(w.N, 48, replace=False)
        ref = oracle.owner_stats(X[b], Y[b], rows, prm)
        np.testing.assert_array_equal(st["j1"][rows], ref["k1"])
        np.testing.assert_array_equal(st["j2"][rows], ref["k2"])
        np.testing.assert_allclose(st["T_row"][rows], ref["T"], rtol=1e-12)
        for r in rows[:16]:
            idx, s, p = oracle.owner_support(X[b], Y[b], int(r), prm)
            sel = (ex["i"] == r) & ((ex["flags"] & 1) > 0)
            np.testing.assert_array_equal(ex["j"][sel], idx)
            np.testing.assert_allclose(ex["p_row"][sel], p, rtol=2e-6)
        cols = rng.choice(w.M, 32, replace=False)
        refc = oracle.owner_stats(Y[b], X[b], cols, prm)
        np.testing.assert_array_equal(st["i1"][cols], refc["k1"])
        np.testing.assert_allclose(st["T_col"][cols], refc["T"], rtol=1e-12)
        for c in cols[:12]:
            idx, s, p = oracle.owner_support(Y[b], X[b], int(c), prm)
            sel = (ex["j"] == c) & ((ex["flags"] & 2) > 0)
            np.testing.assert_array_equal(ex["i"][sel], idx)
            np.testing.assert_allclose(ex["p_col"][sel], p, rtol=2e-6)


def test_largest_sweep_size_sampled_owners():
    # the memory sweep's largest clouds (N = M = 262144, shape-completion
    # generator): sampled rows' and columns' minima, temperatures and kept
    # supports against the oracle, owner by owner
    n = 262144
    X, Y = custom(7, 1, n, n, reference="primitives", prediction="perm_noise", sigma=0.05)
    note(f"sweep size {n}")
    g = run_gpu(X, Y, n_iter=10)
    plan = g["plan"]
    ex = plan.export(0)
    st = plan.export_stats(0)
    prm = oracle_params(n_iter=10)
    rng = np.random.default_rng(262144)
    assert np.isfinite(g["loss"][0]) and np.isfinite(g["gx"]).all()
    assert ex["p0"].astype(np.float64).sum() == pytest.approx(n, rel=1e-5)  # (N + M) / 2
    rows = rng.choice(n, 64, replace=False)
    ref = oracle.owner_stats(X[0], Y[0], rows, prm)
    np.testing.assert_array_equal(st["j1"][rows], ref["k1"])
    np.testing.assert_array_equal(st["j2"][rows], ref["k2"])
    np.testing.assert_allclose(st["T_row"][rows], ref["T"], rtol=1e-12)
    cols = rng.choice(n, 64, replace=False)
    refc = oracle.owner_stats(Y[0], X[0], cols, prm)
    np.testing.assert_array_equal(st["i1"][cols], refc["k1"])
    np.testing.assert_array_equal(st["i2"][cols], refc["k2"])
    np.testing.assert_allclose(st["T_col"][cols], refc["T"], rtol=1e-12)
    for r in rows[:16]:
        idx, s, p = oracle.owner_support(X[0], Y[0], int(r), prm)
        sel = (ex["i"] == r) & ((ex["flags"] & 1) > 0)
        np.testing.assert_array_equal(ex["j"][sel], idx)
        np.testing.assert_allclose(ex["p_row"][sel], p, rtol=2e-6)
    for c in cols[:16]:
        idx, s, p = oracle.owner_support(Y[0], X[0], int(c), prm)
        sel = (ex["j"] == c) & ((ex["flags"] & 2) > 0)
        np.testing.assert_array_equal(ex["i"][sel], idx)
        np.testing.assert_allclose(ex["p_col"][sel], p, rtol=2e-6)
