"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: every expected value is a
closed form, an exact rational computation, a brute-force textbook quantity,
an invariance of the definition, PyTorch autograd of an independent dense
formulation, or a finite difference.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle.dense import dense_apml
from workloads import custom

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _cloud(seed, N, M, sigma=0.05):
    X, Y = custom(seed, 1, N, M, sigma=sigma)
    return X[0], Y[0]


# ---------------------------------------------------------------------------
# Worked example: K = 2 makes Eq. 1 exact, so P_row = (p, 1-p) and the whole
# forward pass is a rational computation (Eq. 1, Eq. 2, initial plan, Eq. 3-4).
# ---------------------------------------------------------------------------

EX_X = np.array([[0.0, 0, 0], [0.375, 0, 0]], np.float32)
EX_Y = np.array([[0.125, 0, 0], [1.0, 0, 0]], np.float32)
EX_C = [[Fraction(1, 8), Fraction(1)], [Fraction(1, 4), Fraction(5, 8)]]


def _exact_sinkhorn_loss(P, L):
    P = [row[:] for row in P]
    for _ in range(L):
        for j in range(2):
            s = P[0][j] + P[1][j]
            P[0][j] /= s
            P[1][j] /= s
        for i in range(2):
            s = P[i][0] + P[i][1]
            P[i][0] /= s
            P[i][1] /= s
    return sum(P[i][j] * EX_C[i][j] for i in range(2) for j in range(2))


@pytest.mark.parametrize("p_min", [0.6, 0.8, 0.95])
def test_worked_example_exact(p_min):
    p = Fraction(p_min).limit_denominator(1000)
    q = 1 - p
    # rows: both minima at j=0; columns: minimum of col 0 at i=0, of col 1 at i=1
    P_row = [[p, q], [p, q]]
    P_col = [[p, q], [q, p]]
    P0 = [[(P_row[i][j] + P_col[i][j]) / 2 for j in range(2)] for i in range(2)]
    for L in (0, 1, 2, 10):
        prm = oracle.params(p_min=p_min, delta=0.0, eps_stab=0.0, n_iter=L)
        r = oracle.run_sample(EX_X, EX_Y, prm, grad=False)
        assert r.nnz == 4
        want = float(_exact_sinkhorn_loss(P0, L))
        assert r.loss == pytest.approx(want, rel=1e-13, abs=0)
    r = oracle.run_sample(EX_X, EX_Y, oracle.params(p_min=p_min, delta=0.0, eps_stab=0.0, n_iter=0), grad=False)
    np.testing.assert_allclose(r.p_row, [float(v) for v in (p, q, p, q)], rtol=1e-14)
    np.testing.assert_allclose(r.p_col, [float(v) for v in (p, q, q, p)], rtol=1e-14)
    # Eq. 1 with K = 2: T = log(p / (1 - p)) / gap
    lk = math.log(p_min / (1 - p_min))
    np.testing.assert_allclose(r.row["T"], [lk / 0.875, lk / 0.375], rtol=1e-14)
    np.testing.assert_allclose(r.col["T"], [lk / 0.125, lk / 0.375], rtol=1e-14)


def test_worked_example_sinkhorn_limit():
    # P0 = [[.8,.2],[.5,.5]] has cross-ratio 4, so the doubly stochastic limit is
    # [[a,1-a],[1-a,a]] with (a/(1-a))^2 = 4: a = 2/3 and loss -> 11/12.
    r = oracle.run_sample(EX_X, EX_Y, oracle.params(delta=0.0, eps_stab=0.0, n_iter=200), grad=False)
    assert r.loss == pytest.approx(11.0 / 12.0, rel=1e-12)


# ---------------------------------------------------------------------------
# Eq. 1: with every non-minimal entry at the same gap g above the minimum, the
# nearest entry gets probability exactly p_min, for any K.
# ---------------------------------------------------------------------------

def _equal_gap_cloud(r=0.25, R=5.0 / 8.0):
    # 30 points at distance exactly 5/8 from the origin: permutations of (0, +-3, +-4)/8
    # and the six axis points +-5/8; plus one point at distance 1/4.
    pts = []
    for a, b in ((3, 4), (4, 3)):
        for sa in (1, -1):
            for sb in (1, -1):
                pts += [(0, sa * a, sb * b), (sa * a, 0, sb * b), (sa * a, sb * b, 0)]
    pts = [tuple(v / 8 for v in p) for p in pts]
    for k in range(3):
        for s in (1, -1):
            e = [0.0, 0.0, 0.0]
            e[k] = s * R
            pts.append(tuple(e))
    Y = np.array([(0.0, 0.0, r)] + pts, np.float32)
    X = np.array([(0.0, 0.0, 0.0), (9.0, 9.0, 9.0), (-9.0, -9.0, -9.0)], np.float32)
    assert np.allclose(np.linalg.norm(Y[1:].astype(np.float64), axis=1), R, rtol=0, atol=0)
    return X, Y


@pytest.mark.parametrize("p_min", [0.5, 0.8, 0.95])
def test_eq1_min_probability_equal_gaps(p_min):
    X, Y = _equal_gap_cloud()
    r = oracle.run_sample(X, Y, oracle.params(p_min=p_min, delta=0.0, tau=0.0, n_iter=0), grad=False)
    sel = (r.i == 0) & (r.j == 0)
    assert r.row["k1"][0] == 0
    assert r.p_row[sel][0] == pytest.approx(p_min, rel=1e-14)
    K = Y.shape[0]
    assert r.row["T"][0] == pytest.approx(math.log((K - 1) * p_min / (1 - p_min)) / (5 / 8 - 1 / 4), rel=1e-14)


# ---------------------------------------------------------------------------
# Threshold: tau = 1 keeps only the argmin entries, so with L = 0 the loss is
# half the (unsquared) Chamfer sum, computed here by brute-force nearest neighbours.
# ---------------------------------------------------------------------------

def test_tau_one_is_half_chamfer():
    x, y = _cloud(1, 40, 33)
    r = oracle.run_sample(x, y, oracle.params(tau=1.0, n_iter=0), grad=False)
    D = np.linalg.norm(x.astype(np.float64)[:, None] - y.astype(np.float64)[None], axis=-1)
    want = 0.5 * (D.min(1).sum() + D.min(0).sum())
    assert r.loss == pytest.approx(want, rel=1e-13)
    assert r.nnz <= 40 + 33
    np.testing.assert_array_equal(r.row["k1"], D.argmin(1))
    np.testing.assert_array_equal(r.col["k1"], D.argmin(0))


def test_radius_identity():
    # s >= tau  <=>  C <= C1 + log(1/tau)/T : the kept set of a row is a ball.
    x, y = _cloud(2, 30, 50)
    prm = oracle.params(tau=1e-3)
    r = oracle.run_sample(x, y, prm, grad=False)
    D = np.linalg.norm(x.astype(np.float64)[:, None] - y.astype(np.float64)[None], axis=-1)
    R = r.row["c1"] + math.log(1 / 1e-3) / r.row["T"]
    ball = D <= R[:, None]
    kept = np.zeros_like(ball)
    kept[r.i[(r.flags & 1) > 0], r.j[(r.flags & 1) > 0]] = True
    np.testing.assert_array_equal(kept, ball)


# ---------------------------------------------------------------------------
# Mass and normalisation invariants of the sparse initial plan.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("tau", [0.0, 1e-8, 1e-3, 1.0])
def test_initial_plan_mass(tau):
    x, y = _cloud(3, 37, 29)
    r = oracle.run_sample(x, y, oracle.params(tau=tau), grad=False)
    rows = np.bincount(r.i, weights=r.p_row, minlength=37)
    cols = np.bincount(r.j, weights=r.p_col, minlength=29)
    np.testing.assert_allclose(rows, 1.0, rtol=1e-14)
    np.testing.assert_allclose(cols, 1.0, rtol=1e-14)
    assert r.p0.sum() == pytest.approx((37 + 29) / 2, rel=1e-14)
    # a positive probability needs the flag; with tau > 0 every flagged entry is positive
    # (with tau = 0 far entries underflow to exactly zero in double precision)
    assert not np.any((r.p_row > 0) & ((r.flags & 1) == 0))
    assert not np.any((r.p_col > 0) & ((r.flags & 2) == 0))
    if tau > 0:
        assert np.all(r.p_row[(r.flags & 1) > 0] > 0) and np.all(r.p_col[(r.flags & 2) > 0] > 0)
    # entries sorted by (i, j), each pair once
    key = r.i.astype(np.int64) * 29 + r.j
    assert np.all(np.diff(key) > 0)


# ---------------------------------------------------------------------------
# Dense formulation (independent matrix code): tau = 0 must be identical.
# ---------------------------------------------------------------------------

def _dense_from_oracle(x, y, r, **kw):
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    yt = torch.tensor(y, dtype=torch.float64, requires_grad=True)
    loss, mats = dense_apml(xt, yt, row_argmins=(r.row["k1"], r.row["k2"]),
                            col_argmins=(r.col["k1"], r.col["k2"]), **kw)
    loss.backward()
    return loss.item(), xt.grad.numpy(), yt.grad.numpy(), mats


@pytest.mark.parametrize("tau", [0.0, 1e-8, 1e-2])
def test_matches_dense_formulation(tau):
    x, y = _cloud(4, 23, 31, sigma=0.1)
    kw = dict(p_min=0.8, tau=tau, n_iter=7, eps_stab=1e-8, delta=1e-8, eps_gap=1e-6)
    r = oracle.run_sample(x, y, oracle.params(**kw), grad=True)
    loss, gx, gy, mats = _dense_from_oracle(x, y, r, **kw)
    if tau == 0.0:
        assert r.nnz == 23 * 31
    assert r.loss == pytest.approx(loss, rel=1e-12)
    # autograd of the dense formulation pins the hand-written reverse mode
    np.testing.assert_allclose(r.grad_x, gx, rtol=1e-9, atol=1e-12 * np.abs(gx).max())
    np.testing.assert_allclose(r.grad_y, gy, rtol=1e-9, atol=1e-12 * np.abs(gy).max())
    np.testing.assert_allclose(r.p0, mats["P0"].detach().numpy()[r.i, r.j], rtol=1e-12)
    np.testing.assert_allclose(r.v, mats["P"].detach().numpy()[r.i, r.j], rtol=1e-11)
    # the support is exactly the union of the dense masks
    union = (mats["keep_row"] | mats["keep_col"]).numpy()
    assert r.nnz == union.sum()
    assert union[r.i, r.j].all()


def test_argmins_match_double_precision_decision():
    # on generic data the single-precision decision equals the double one
    x, y = _cloud(5, 64, 64)
    r = oracle.run_sample(x, y, oracle.params(), grad=False)
    D = np.linalg.norm(x.astype(np.float64)[:, None] - y.astype(np.float64)[None], axis=-1)
    o = np.argsort(D, axis=1, kind="stable")
    np.testing.assert_array_equal(r.row["k1"], o[:, 0])
    np.testing.assert_array_equal(r.row["k2"], o[:, 1])
    oc = np.argsort(D, axis=0, kind="stable")
    np.testing.assert_array_equal(r.col["k1"], oc[0])
    np.testing.assert_array_equal(r.col["k2"], oc[1])


def test_sparse_close_to_dense_apml():
    # the paper's claim: thresholding at tau = 1e-8 keeps the loss of dense APML
    x, y = _cloud(6, 128, 128)
    dense = oracle.run_sample(x, y, oracle.params(tau=0.0), grad=True)
    sparse = oracle.run_sample(x, y, oracle.params(tau=1e-8), grad=True)
    assert sparse.nnz < 0.2 * dense.nnz
    assert sparse.loss == pytest.approx(dense.loss, rel=1e-5)
    err = np.linalg.norm(sparse.grad_x - dense.grad_x) / np.linalg.norm(dense.grad_x)
    assert err < 1e-3


# ---------------------------------------------------------------------------
# Backward: finite differences in double precision.
# ---------------------------------------------------------------------------

def test_finite_differences():
    x, y = _cloud(7, 14, 17, sigma=0.15)
    prm = oracle.params(n_iter=5)
    r = oracle.run_sample(x, y, prm, grad=True)
    x64, y64 = x.astype(np.float64), y.astype(np.float64)
    h = 1e-6
    rng = np.random.default_rng(0)
    checked = 0
    for which, base, g in (("x", x64, r.grad_x), ("y", y64, r.grad_y)):
        for _ in range(12):
            a, k = int(rng.integers(base.shape[0])), int(rng.integers(3))
            vals = []
            for sgn in (1, -1):
                pert = base.copy()
                pert[a, k] += sgn * h
                rr = oracle.run_sample(pert if which == "x" else x64, y64 if which == "x" else pert, prm, grad=False)
                vals.append(rr)
            if vals[0].nnz != r.nnz or vals[1].nnz != r.nnz or not (
                    np.array_equal(vals[0].flags, r.flags) and np.array_equal(vals[1].flags, r.flags)):
                continue  # the support moved: not differentiable there
            fd = (vals[0].loss - vals[1].loss) / (2 * h)
            assert fd == pytest.approx(g[a, k], rel=2e-5, abs=2e-6 * np.abs(g).max())
            checked += 1
    assert checked >= 18


# ---------------------------------------------------------------------------
# Invariances of the definition (exact transformations in float32).
# ---------------------------------------------------------------------------

def test_permutation_invariance():
    x, y = _cloud(8, 50, 45)
    r = oracle.run_sample(x, y, oracle.params(), grad=True)
    rng = np.random.default_rng(1)
    px, py = rng.permutation(50), rng.permutation(45)
    rp = oracle.run_sample(x[px], y[py], oracle.params(), grad=True)
    assert rp.loss == pytest.approx(r.loss, rel=1e-12)
    assert rp.nnz == r.nnz
    np.testing.assert_allclose(rp.grad_x, r.grad_x[px], rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(rp.grad_y, r.grad_y[py], rtol=1e-9, atol=1e-12)


def test_rigid_invariance():
    # dyadic coordinates make the translation and the 90-degree rotation exact
    rng = np.random.default_rng(9)
    x = (rng.integers(-2 ** 12, 2 ** 12, size=(40, 3)) / 2 ** 13).astype(np.float32)
    y = (rng.integers(-2 ** 12, 2 ** 12, size=(36, 3)) / 2 ** 13).astype(np.float32)
    r = oracle.run_sample(x, y, oracle.params(), grad=True)
    t = np.array([0.5, -0.25, 0.125], np.float32)
    rt = oracle.run_sample(x + t, y + t, oracle.params(), grad=True)
    assert rt.loss == pytest.approx(r.loss, rel=1e-12)
    np.testing.assert_allclose(rt.grad_x, r.grad_x, rtol=1e-8, atol=1e-11)
    rot = np.array([[0, -1, 0], [1, 0, 0], [0, 0, 1]], np.float32)
    rr = oracle.run_sample(x @ rot.T, y @ rot.T, oracle.params(), grad=True)
    assert rr.loss == pytest.approx(r.loss, rel=1e-12)
    np.testing.assert_allclose(rr.grad_x, r.grad_x @ rot.T, rtol=1e-8, atol=1e-11)


def test_scale_covariance_exact():
    # doubling all coordinates, delta and eps_g leaves every exponent unchanged
    x, y = _cloud(10, 33, 41)
    kw = dict(delta=1e-8, eps_gap=1e-6, eps_dist=0.0)
    r = oracle.run_sample(x, y, oracle.params(**kw), grad=True)
    kw2 = dict(delta=2e-8, eps_gap=2e-6, eps_dist=0.0)
    r2 = oracle.run_sample(2 * x, 2 * y, oracle.params(**kw2), grad=True)
    assert r2.loss == 2 * r.loss
    np.testing.assert_array_equal(r2.grad_x, r.grad_x)


def test_gradient_identities():
    x, y = _cloud(11, 60, 52, sigma=0.08)
    r = oracle.run_sample(x, y, oracle.params(delta=0.0, eps_dist=0.0), grad=True)
    x64, y64 = x.astype(np.float64), y.astype(np.float64)
    scale = np.abs(r.grad_x).sum()
    # translation: sum of all point gradients vanishes
    np.testing.assert_allclose(r.grad_x.sum(0) + r.grad_y.sum(0), 0.0, atol=1e-12 * scale)
    # rotation: total torque vanishes
    torque = np.cross(x64, r.grad_x).sum(0) + np.cross(y64, r.grad_y).sum(0)
    np.testing.assert_allclose(torque, 0.0, atol=1e-12 * scale)
    # Euler: the loss is homogeneous of degree 1 when delta = 0 and no gap is clamped
    assert not r.row["clamped"].any() and not r.col["clamped"].any()
    euler = (x64 * r.grad_x).sum() + (y64 * r.grad_y).sum()
    assert euler == pytest.approx(r.loss, rel=1e-10)


# ---------------------------------------------------------------------------
# Sinkhorn (Eq. 3, Eq. 4)
# ---------------------------------------------------------------------------

def test_sinkhorn_marginals_converge():
    # N = M, full support: the column marginals approach the uniform target
    x, y = _cloud(12, 24, 24, sigma=0.3)
    dev = []
    for L in (10, 100, 1000):
        r = oracle.run_sample(x, y, oracle.params(tau=0.0, n_iter=L, eps_stab=0.0), grad=False)
        np.testing.assert_allclose(np.bincount(r.i, weights=r.v, minlength=24), 1.0, rtol=1e-12)
        dev.append(np.abs(np.bincount(r.j, weights=r.v, minlength=24) - 1.0).max())
    assert dev[0] > dev[1] > dev[2] and dev[2] < 1e-10


def test_sinkhorn_row_sums_and_cross_ratios():
    x, y = _cloud(13, 40, 40, sigma=0.05)
    eps = 1e-3
    r = oracle.run_sample(x, y, oracle.params(n_iter=4, eps_stab=eps), grad=False)
    rows = np.bincount(r.i, weights=r.v, minlength=40)
    np.testing.assert_allclose(rows, r.rowsum_last / (r.rowsum_last + eps), rtol=1e-13)
    # scaling by row and column factors preserves every 2x2 cross-ratio inside the support
    pos = {(a, b): t for t, (a, b) in enumerate(zip(r.i, r.j))}
    n = 0
    for (a, b), t in pos.items():
        for (c, d), u in pos.items():
            if c <= a or d == b or (a, d) not in pos or (c, b) not in pos:
                continue
            ad, cb = pos[(a, d)], pos[(c, b)]
            want = r.p0[t] * r.p0[u] / (r.p0[ad] * r.p0[cb])
            got = r.v[t] * r.v[u] / (r.v[ad] * r.v[cb])
            assert got == pytest.approx(want, rel=1e-11)
            n += 1
    assert n > 10


def test_identical_clouds_small_loss():
    x, y = _cloud(14, 200, 200, sigma=0.03)
    noisy = oracle.run_sample(x, y, oracle.params(), grad=False).loss
    prev = None
    for p in (0.8, 0.95, 0.995):
        same = oracle.run_sample(y, y, oracle.params(p_min=p), grad=False).loss
        assert same < 0.1 * noisy
        if prev is not None:
            assert same < prev
        prev = same


def test_ties_clamp_and_index_order():
    # duplicated reference points: the two smallest costs tie, the gap clamps to
    # eps_g, and the argmins are the two smallest indices attaining the tie
    x, y = _cloud(15, 20, 20)
    y = np.concatenate([y, y[:5]])  # points 20..24 duplicate 0..4
    r = oracle.run_sample(x, y, oracle.params(), grad=True)
    dup = np.isin(r.row["k1"], np.arange(5))
    assert dup.any()
    np.testing.assert_array_equal(r.row["k2"][dup], r.row["k1"][dup] + 20)
    assert r.row["clamped"][dup].all()
    np.testing.assert_allclose(r.row["g"][dup], 1e-6)
    lk = math.log((25 - 1) * 0.8 / 0.2)
    np.testing.assert_allclose(r.row["T"][dup], lk / 1e-6, rtol=1e-14)
    # clamped rows have no temperature gradient: the identities still hold
    scale = np.abs(r.grad_x).sum()
    np.testing.assert_allclose(r.grad_x.sum(0) + r.grad_y.sum(0), 0.0, atol=1e-11 * scale)


# ---------------------------------------------------------------------------
# Reading variants: uniform fallback, literal duplicate averaging, detached
# temperature. Each is pinned by a closed form and by autograd of the dense
# formulation.
# ---------------------------------------------------------------------------

def _nn_pairs(D):
    """Union of the row and column argmin pairs (brute force), as a set."""
    rows = {(i, int(j)) for i, j in enumerate(D.argmin(1))}
    cols = {(int(i), j) for j, i in enumerate(D.argmin(0))}
    return rows, cols


def test_mean_dup_tau_one_closed_form():
    # tau = 1 keeps only argmin entries with probability 1 in their direction:
    # averaging duplicates literally gives P0 = 1 on the union of the argmin
    # pairs, so with L = 0 the loss is the sum of C over that union
    x, y = _cloud(18, 40, 33)
    D = np.linalg.norm(x.astype(np.float64)[:, None] - y.astype(np.float64)[None], axis=-1)
    rows, cols = _nn_pairs(D)
    union = rows | cols
    want = sum(D[i, j] for i, j in union)
    r = oracle.run_sample(x, y, oracle.params(tau=1.0, n_iter=0, sym_mode=1), grad=False)
    assert r.nnz == len(union)
    assert r.loss == pytest.approx(want, rel=1e-13)
    np.testing.assert_allclose(r.p0, 1.0, rtol=0)
    # the half sum differs exactly on the pairs one direction keeps alone
    h = oracle.run_sample(x, y, oracle.params(tau=1.0, n_iter=0), grad=False)
    single = sum(D[i, j] for i, j in union - (rows & cols))
    assert r.loss - h.loss == pytest.approx(0.5 * single, rel=1e-12)


def test_mean_dup_full_support_equals_half_sum():
    # tau = 0 keeps every pair in both directions: nothing is a singleton
    x, y = _cloud(19, 17, 21)
    a = oracle.run_sample(x, y, oracle.params(tau=0.0, sym_mode=1), grad=True)
    b = oracle.run_sample(x, y, oracle.params(tau=0.0), grad=True)
    assert a.loss == b.loss
    np.testing.assert_array_equal(a.grad_x, b.grad_x)


def _tie_cloud(seed):
    # every reference point doubled: each row's two smallest costs tie
    x, y = _cloud(seed, 12, 10, sigma=0.1)
    return x, np.concatenate([y, y])


def test_fallback_tau_one_closed_form():
    # with all references doubled, every row falls back to 1/M over all M
    # entries; columns (distinct x) keep their argmin. tau = 1, L = 0:
    # loss = (sum_i mean_j C_ij + sum_j min_i C_ij) / 2
    x, y = _tie_cloud(20)
    N, M = x.shape[0], y.shape[0]
    D = np.linalg.norm(x.astype(np.float64)[:, None] - y.astype(np.float64)[None], axis=-1)
    r = oracle.run_sample(x, y, oracle.params(tau=1.0, n_iter=0, gap_mode=1), grad=True)
    assert (r.row["T"] == 0).all() and r.row["clamped"].all()
    assert r.nnz == N * M
    want = 0.5 * (D.mean(1).sum() + D.min(0).sum())
    assert r.loss == pytest.approx(want, rel=1e-13)
    np.testing.assert_allclose(r.p_row, 1.0 / M, rtol=1e-15)
    # the fallback is a constant: only the column softmaxes and the costs carry gradient,
    # and at tau = 1 the column direction is a plain nearest neighbour
    gx = np.zeros_like(D[:, :1].repeat(3, 1))
    diff = x.astype(np.float64)[:, None] - y.astype(np.float64)[None]
    gx += 0.5 * (diff / D[..., None]).sum(1) / M
    i1 = D.argmin(0)
    for j in range(M):
        gx[i1[j]] += 0.5 * diff[i1[j], j] / D[i1[j], j]
    np.testing.assert_allclose(r.grad_x, gx, rtol=1e-10, atol=1e-14)


def test_fallback_only_below_eps_gap():
    # generic data: no gap is below eps_g, so the fallback changes nothing
    x, y = _cloud(21, 30, 30)
    a = oracle.run_sample(x, y, oracle.params(gap_mode=1), grad=True)
    b = oracle.run_sample(x, y, oracle.params(), grad=True)
    assert a.loss == b.loss and a.nnz == b.nnz
    np.testing.assert_array_equal(a.grad_x, b.grad_x)


def test_detached_temperature_drops_gap_term():
    # with the temperature a constant, the gradient is the full one minus the
    # gap term; finite differences of a loss at fixed T are not available from
    # the oracle, so the dense formulation's autograd (T detached) pins it
    x, y = _cloud(22, 19, 23, sigma=0.1)
    kw = dict(p_min=0.8, tau=1e-2, n_iter=6, eps_stab=1e-8, delta=1e-8, eps_gap=1e-6)
    r = oracle.run_sample(x, y, oracle.params(tgrad_mode=1, **kw), grad=True)
    full = oracle.run_sample(x, y, oracle.params(**kw), grad=True)
    assert r.loss == full.loss
    assert np.abs(r.grad_x - full.grad_x).max() > 1e-3 * np.abs(full.grad_x).max()
    loss, gx, gy, _ = _dense_from_oracle(x, y, r, tgrad_mode=1, **kw)
    assert r.loss == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(r.grad_x, gx, rtol=1e-9, atol=1e-12 * np.abs(gx).max())
    np.testing.assert_allclose(r.grad_y, gy, rtol=1e-9, atol=1e-12 * np.abs(gy).max())


def test_mean_dup_finite_differences():
    # literal duplicate averaging is still a differentiable function of the
    # points away from support changes: its hand-written gradient against
    # central differences of its own loss
    x, y = _cloud(24, 13, 16, sigma=0.15)
    prm = oracle.params(n_iter=4, sym_mode=1)
    r = oracle.run_sample(x, y, prm, grad=True)
    assert ((r.flags == 1) | (r.flags == 2)).any()  # singletons exist, so the variant differs
    x64, y64 = x.astype(np.float64), y.astype(np.float64)
    h = 1e-6
    rng = np.random.default_rng(3)
    checked = 0
    for which, base, g in (("x", x64, r.grad_x), ("y", y64, r.grad_y)):
        for _ in range(10):
            a, k = int(rng.integers(base.shape[0])), int(rng.integers(3))
            vals = []
            for sgn in (1, -1):
                pert = base.copy()
                pert[a, k] += sgn * h
                vals.append(oracle.run_sample(pert if which == "x" else x64, y64 if which == "x" else pert, prm,
                                              grad=False))
            if any(v.nnz != r.nnz or not np.array_equal(v.flags, r.flags) for v in vals):
                continue
            fd = (vals[0].loss - vals[1].loss) / (2 * h)
            assert fd == pytest.approx(g[a, k], rel=2e-5, abs=2e-6 * np.abs(g).max())
            checked += 1
    assert checked >= 14


@pytest.mark.parametrize("mode", [dict(sym_mode=1), dict(gap_mode=1), dict(gap_mode=1, sym_mode=1, tgrad_mode=1)])
def test_variants_match_dense_formulation(mode):
    x, y = _tie_cloud(23) if mode.get("gap_mode") else _cloud(23, 21, 26, sigma=0.1)
    kw = dict(p_min=0.8, tau=1e-3, n_iter=5, eps_stab=1e-8, delta=1e-8, eps_gap=1e-6)
    r = oracle.run_sample(x, y, oracle.params(**kw, **mode), grad=True)
    loss, gx, gy, mats = _dense_from_oracle(x, y, r, **kw, **mode)
    assert r.loss == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(r.grad_x, gx, rtol=1e-9, atol=1e-12 * np.abs(gx).max())
    np.testing.assert_allclose(r.grad_y, gy, rtol=1e-9, atol=1e-12 * np.abs(gy).max())
    np.testing.assert_allclose(r.p0, mats["P0"].detach().numpy()[r.i, r.j], rtol=1e-12)
    union = (mats["keep_row"] | mats["keep_col"]).numpy()
    assert r.nnz == union.sum()


def test_owner_sampling_matches_full_run():
    x, y = _cloud(16, 70, 90)
    prm = oracle.params()
    r = oracle.run_sample(x, y, prm, grad=False)
    rows = np.array([0, 5, 69, 33])
    st = oracle.owner_stats(x, y, rows, prm)
    np.testing.assert_array_equal(st["T"], r.row["T"][rows])
    np.testing.assert_array_equal(st["k2"], r.row["k2"][rows])
    cnt = np.bincount(r.i[(r.flags & 1) > 0], minlength=70)
    np.testing.assert_array_equal(st["count"], cnt[rows])
    idx, s, p = oracle.owner_support(y, x, 7, prm)
    sel = (r.j == 7) & ((r.flags & 2) > 0)
    np.testing.assert_array_equal(idx, r.i[sel])
    np.testing.assert_array_equal(p, r.p_col[sel])


def test_rejects_invalid_arguments():
    x, y = _cloud(17, 8, 8)
    for bad in (dict(p_min=1.0), dict(p_min=0.1), dict(tau=2.0), dict(n_iter=-1), dict(eps_gap=0.0),
                dict(gap_mode=2), dict(sym_mode=-1), dict(tgrad_mode=3)):
        with pytest.raises(ValueError):
            oracle.run_sample(x, y, oracle.params(**bad))
    with pytest.raises(ValueError):
        oracle.run_sample(x[:1], y, oracle.params())
