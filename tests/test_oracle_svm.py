"""Pins of the oracle's hinge-loss SVM dual solver (box-constrained coordinate ascent).

  P(w) = (1/N) sum_i max(0, 1 - y_i x_i.w) + lambda/2 |w|^2
  D(a) = (1/N) sum_i a_i - lambda/2 |w(a)|^2,  w(a) = sum_i a_i y_i x_i / (lambda N),  0 <= a <= 1

Pinned by: active-set brute force of the dual QP's KKT system on tiny problems (w* and P*
are unique because P is strongly convex), bounded 1-D library maximisation of D along the
visited coordinate, the N = 1 closed case, box constraints, per-step monotone D, weak
duality, gap -> 0 and the invariant w = w(alpha).
"""
import itertools

import numpy as np
import pytest
from scipy.optimize import minimize_scalar

from tests._helpers import rel_inf, segments


def _P(X, y, lam, w):
    return np.maximum(0.0, 1.0 - y * (X @ w)).mean() + lam / 2 * w @ w


def _D(X, y, lam, a):
    N = X.shape[0]
    w = X.T @ (a * y) / (lam * N)
    return a.mean() - lam / 2 * w @ w


def _brute_force(X, y, lam):
    """Enumerate every {0, free, 1} pattern of the dual QP; keep the KKT-feasible one."""
    N = X.shape[0]
    Q = (y[:, None] * X) @ (y[:, None] * X).T
    best = None
    for pat in itertools.product((0, 1, 2), repeat=N):
        pat = np.array(pat)
        a = np.where(pat == 1, 1.0, 0.0)
        F = np.nonzero(pat == 2)[0]
        if F.size:
            # Free coordinates: 1 - y_i x_i.w = 0  <=>  Q_FF a_F = lam N - Q_F,rest a_rest.
            rhs = lam * N - Q[np.ix_(F, np.setdiff1d(np.arange(N), F))] @ a[np.setdiff1d(np.arange(N), F)]
            sol, *_ = np.linalg.lstsq(Q[np.ix_(F, F)], rhs, rcond=None)
            if not np.allclose(Q[np.ix_(F, F)] @ sol, rhs, atol=1e-10):
                continue
            a[F] = sol
        if np.any(a < -1e-12) or np.any(a > 1 + 1e-12):
            continue
        w = X.T @ (a * y) / (lam * N)
        m = 1.0 - y * (X @ w)
        tol = 1e-9
        ok = (np.all(m[pat == 0] <= tol) and np.all(m[pat == 1] >= -tol) and np.all(np.abs(m[F]) <= tol))
        if ok:
            val = _D(X, y, lam, np.clip(a, 0, 1))
            if best is None or val > best[0]:
                best = (val, w, np.clip(a, 0, 1))
    return best


def _tiny(seed, N, M, density=1.0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((N, M)).astype(np.float32)
    if density < 1.0:
        X *= rng.random((N, M)) < density
    y = np.where(rng.random(N) < 0.5, -1.0, 1.0).astype(np.float32)
    return X.astype(np.float64), y


@pytest.mark.parametrize("seed,N,M,lam", [(0, 5, 3, 0.1), (1, 7, 4, 0.05), (2, 8, 2, 0.2), (3, 6, 10, 0.01),
                                          (4, 8, 5, 1.0)])
def test_converges_to_active_set_brute_force(oracle, seed, N, M, lam):
    X, y = _tiny(seed, N, M)
    Dstar, wstar, _ = _brute_force(X, y.astype(np.float64), lam)
    ptr, idx, val = segments(X, "csr")
    a = np.zeros(N)
    w = np.zeros(M)
    oracle.epochs("svm_dual", N, M, ptr, idx, val, y, lam, 0, 0, 3000, a, w)
    assert np.all(a >= 0) and np.all(a <= 1)
    fresh = oracle.fresh_shared("svm_dual", N, M, ptr, idx, val, y, lam, a)
    assert rel_inf(fresh, wstar) <= 1e-9
    P, D, G = oracle.objectives("svm_dual", N, M, ptr, idx, val, y, lam, a)
    Pstar = _P(X, y, lam, wstar)
    assert abs(P - Pstar) <= 1e-9 * abs(Pstar)
    assert abs(D - Dstar) <= 1e-9 * abs(Pstar)
    assert G <= 1e-9


def test_step_is_bounded_1d_maximiser(oracle):
    X, y = _tiny(10, 9, 6, 0.7)
    N, M = X.shape
    lam = 0.05
    ptr, idx, val = segments(X, "csr")
    rng = np.random.default_rng(2)
    a = rng.random(N)
    w = X.T @ (a * y) / (lam * N)
    clipped = interior = 0
    for i in [0, 4, 8, 2, 6, 1, 3]:
        before = a.copy()
        oracle.visit("svm_dual", N, M, ptr, idx, val, y, lam, [i], a, w)
        e = np.zeros(N)
        e[i] = 1.0
        res = minimize_scalar(lambda t: -_D(X, y, lam, before + (t - before[i]) * e), bounds=(0.0, 1.0),
                              method="bounded", options={"xatol": 1e-12})
        assert abs(a[i] - res.x) <= 1e-5
        clipped += a[i] in (0.0, 1.0)
        interior += 0.0 < a[i] < 1.0
        np.testing.assert_allclose(w, X.T @ (a * y) / (lam * N), rtol=0, atol=1e-12)
    assert clipped and interior  # both branches exercised


def test_single_example_closed_case(oracle):
    x = np.array([[0.3, -1.2, 2.0]])
    for yv, lam in [(1.0, 0.5), (-1.0, 0.5), (1.0, 100.0)]:
        ptr, idx, val = segments(x, "csr")
        s = float((val.astype(np.float64) ** 2).sum())
        a = np.zeros(1)
        w = np.zeros(3)
        y = np.array([yv], dtype=np.float32)
        oracle.visit("svm_dual", 1, 3, ptr, idx, val, y, lam, [0], a, w)
        assert a[0] == pytest.approx(min(1.0, lam / s), rel=1e-15)
        if lam / s < 1.0:  # unclipped: the margin lands exactly on 1
            assert yv * float(val.astype(np.float64) @ w[idx]) == pytest.approx(1.0, rel=1e-14)


def test_monotone_dual_box_and_weak_duality(oracle, synth):
    p = synth.make("click_svm", n_rows=400, n_cols=600, row_nnz=8)
    X = np.zeros((p.n_rows, p.n_cols))
    for i in range(p.n_rows):
        X[i, p.idx[p.ptr[i]:p.ptr[i + 1]]] = p.val[p.ptr[i]:p.ptr[i + 1]]
    y = p.y.astype(np.float64)
    a = np.zeros(p.n_rows)
    w = np.zeros(p.n_cols)
    last = _D(X, y, p.lam, a)
    for i in oracle.permutation(0, 0, p.n_rows).tolist():
        oracle.visit("svm_dual", p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, [i], a, w)
        now = _D(X, y, p.lam, a)
        assert now >= last - 1e-13
        last = now
    assert np.all((a >= 0) & (a <= 1))
    rng = np.random.default_rng(0)
    for _ in range(5):
        r = rng.random(p.n_rows)
        P, D, G = oracle.objectives("svm_dual", p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, r)
        assert G >= 0.0 and abs(P - _P(X, y, p.lam, X.T @ (r * y) / (p.lam * p.n_rows))) <= 1e-12 * max(1, P)


def test_gap_to_zero_and_invariant(oracle, synth):
    p = synth.make("text_svm", n_rows=300, n_cols=4000, row_nnz=40)
    a = np.zeros(p.C)
    w = np.zeros(p.L)
    gaps = []
    for e in range(40):
        oracle.epochs(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 5, e, 1, a, w)
        gaps.append(oracle.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, a)[2])
    assert gaps[0] > 1e-2 and gaps[-1] < 1e-7
    fresh = oracle.fresh_shared(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, a)
    assert rel_inf(w, fresh) <= 1e-12


def test_empty_row_goes_to_upper_bound(oracle):
    X = np.array([[1.0, 0.0], [0.0, 0.0], [0.5, 2.0]])
    y = np.array([1, -1, 1], dtype=np.float32)
    ptr, idx, val = segments(X, "csr")
    a = np.array([0.2, 0.3, 0.0])
    w = X.T @ (a * y) / (0.1 * 3)
    w0 = w.copy()
    oracle.visit("svm_dual", 3, 2, ptr, idx, val, y, 0.1, [1], a, w)
    assert a[1] == 1.0 and np.array_equal(w, w0)


def test_resume_is_bit_exact(oracle, synth):
    p = synth.make("click_svm", n_rows=3000, n_cols=5000, row_nnz=12)
    args = (p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 9)
    a1, w1 = np.zeros(p.C), np.zeros(p.L)
    oracle.epochs(*args, 0, 6, a1, w1)
    a2, w2 = np.zeros(p.C), np.zeros(p.L)
    oracle.epochs(*args, 0, 2, a2, w2)
    oracle.epochs(*args, 2, 4, a2, w2)
    assert np.array_equal(a1, a2) and np.array_equal(w1, w2)
