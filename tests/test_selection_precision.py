"""Reading R2 measured on the benchmark workloads (CPU only).

The paper defines the minimum and second minimum of a row or column on the
cost C (Sec. III-A, Eq. 1). The oracle, like the GPU path, decides them on the
single-precision squared distance (reading R2). These tests count, on the
seeded inputs of all five workloads, the owners whose (argmin, second argmin)
would change if the decision were taken on C in double precision, and check
that the loss and gradient of every sample holding such an owner stay within
the parity tolerances (loss 1e-5, gradient 1e-4 relative) under the double
decision.
"""
import numpy as np
import pytest

import oracle
from workloads import batch, config, custom

LOSS_RTOL = 1e-5
GRAD_RTOL = 1e-4


def _rel(a, b):
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def _sq32(a, b):
    d = (a.astype(np.float32) - b.astype(np.float32)).astype(np.float32)
    s = np.float32(d[0] * d[0])
    s = np.float32(np.float64(d[1]) * np.float64(d[1]) + np.float64(s))  # fma, one rounding
    return np.float32(np.float64(d[2]) * np.float64(d[2]) + np.float64(s))


def _near_tie(rng):
    """x, y0, y1 in float32 with equal single-precision squared distances
    while y0 is strictly farther from x than y1 in exact arithmetic."""
    while True:
        x = rng.uniform(-1, 1, 3).astype(np.float32)
        y1 = rng.uniform(-1, 1, 3).astype(np.float32)
        y0 = y1.copy()
        k = rng.integers(3)
        y0[k] = np.nextafter(y1[k], np.float32(np.inf if y1[k] > x[k] else -np.inf))
        d0 = np.linalg.norm(x.astype(np.float64) - y0.astype(np.float64))
        d1 = np.linalg.norm(x.astype(np.float64) - y1.astype(np.float64))
        if _sq32(x, y0) == _sq32(x, y1) and d0 > d1:
            return x, y0, y1


def test_double_decision_is_brute_force_argsort():
    # a near-tie below single-precision resolution: y0 and y1 are one ulp
    # apart, y0 (the smaller index) farther from x; the double decision must
    # follow the exact order, the single one sees a tie and keeps the smaller
    # index
    x, y0, y1 = _near_tie(np.random.default_rng(7))
    x2 = np.stack([x, y1 + 9.5]).astype(np.float32)
    y2 = np.stack([y0, y1, y1 + 10.0, y1 - 10.0]).astype(np.float32)
    prm = oracle.params(select_mode=1, n_iter=0)
    st = oracle.owner_stats(x2, y2, np.arange(2), prm)
    single = oracle.owner_stats(x2, y2, np.arange(2), oracle.params(n_iter=0))
    assert (single["k1"][0], single["k2"][0]) == (0, 1), "the case must tie in single precision"
    assert (st["k1"][0], st["k2"][0]) == (1, 0)
    D = np.linalg.norm(x2.astype(np.float64)[:, None] - y2.astype(np.float64)[None], axis=-1)
    o = np.argsort(D, axis=1, kind="stable")
    np.testing.assert_array_equal(st["k1"], o[:, 0])
    np.testing.assert_array_equal(st["k2"], o[:, 1])
    np.testing.assert_allclose(st["c1"], D[np.arange(2), o[:, 0]], rtol=0, atol=0)
    # random clouds with exact duplicates: ties go to the smaller index
    X, Y = custom(41, 1, 90, 70, sigma=0.05)
    Y = np.concatenate([Y[0], Y[0, :20]])
    for P, Q in ((X[0], Y), (Y, X[0])):
        st = oracle.owner_stats(P, Q, np.arange(P.shape[0]), prm)
        D = np.linalg.norm(P.astype(np.float64)[:, None] - Q.astype(np.float64)[None], axis=-1)
        o = np.argsort(D, axis=1, kind="stable")
        np.testing.assert_array_equal(st["k1"], o[:, 0])
        np.testing.assert_array_equal(st["k2"], o[:, 1])


# owners examined per workload: every owner of every sample of the two small
# workloads, every owner of samples 0-3 and of the last sample of the large
# batch and the unequal workload, and 4096 seeded owners per direction in the
# first and the last sample of the large scene
def _owners(cfg, n, rng):
    if cfg != 5:
        return np.arange(n, dtype=np.int32)
    return np.sort(rng.choice(n, 4096, replace=False)).astype(np.int32)


def _samples(w):
    if w.N <= 2048:
        return list(range(w.B))
    return [0, w.B - 1] if w.N > 16384 else [0, 1, 2, 3, w.B - 1]


@pytest.mark.slow
@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_single_precision_decision_on_the_workloads(cfg):
    w = config(cfg)
    X, Y = batch(w)
    rng = np.random.default_rng(1000 + cfg)
    p32 = oracle.params(n_iter=w.n_iter)
    p64 = oracle.params(n_iter=w.n_iter, select_mode=1)
    owners = differing = 0
    affected = set()
    for b in _samples(w):
        for P, Q in ((X[b], Y[b]), (Y[b], X[b])):
            own = _owners(cfg, P.shape[0], rng)
            a = oracle.owner_stats(P, Q, own, p32)
            c = oracle.owner_stats(P, Q, own, p64)
            d = (a["k1"] != c["k1"]) | (a["k2"] != c["k2"])
            owners += own.size
            differing += int(d.sum())
            if d.any():
                affected.add(b)
    print(f"\n{w.name}: {differing} of {owners} owners change their (argmin, second argmin) "
          f"under the double decision; samples {sorted(affected)}")
    # the whole-sample consequence, where a sample is cheap enough to run twice
    for b in sorted(affected):
        if w.N * w.M > 4096 * 16384:
            continue
        r32 = oracle.run_sample(X[b], Y[b], p32, grad=True)
        r64 = oracle.run_sample(X[b], Y[b], p64, grad=True)
        dl = abs(r32.loss - r64.loss) / abs(r64.loss)
        dgx, dgy = _rel(r32.grad_x, r64.grad_x), _rel(r32.grad_y, r64.grad_y)
        print(f"  sample {b}: loss rel {dl:.2e}, grad_x rel {dgx:.2e}, grad_y rel {dgy:.2e}, "
              f"stored pairs {r32.nnz} vs {r64.nnz}")
        assert dl <= LOSS_RTOL and dgx <= GRAD_RTOL and dgy <= GRAD_RTOL
