"""Pins of the oracle's ridge-regression solvers (Sec. II, Alg. 1).

Primal: closed-form minimiser (A^T A + N lambda I)^-1 A^T y (normal equations of
eq. primal_obj), strong duality P(beta*) = D(alpha*) with alpha* = (y - A beta*)/N
(eqs. duality-1/2), 1-D library minimisation of P along the visited coordinate,
per-step monotonicity, shared-vector invariant w = A beta, gap -> 0, resume determinism.
Dual: alpha* = (y - A beta*)/N and beta* = A^T alpha*/lambda at convergence, 1-D
library maximisation of D, gap -> 0.
"""
import numpy as np
import pytest
from scipy.optimize import minimize_scalar

from tests._helpers import rel_inf, segments


def _closed_form(A, y, lam):
    N, M = A.shape
    return np.linalg.solve(A.T @ A + N * lam * np.eye(M), A.T @ y)


def _P(A, y, lam, beta):  # eq. primal_obj evaluated densely
    N = A.shape[0]
    r = A @ beta - y
    return r @ r / (2 * N) + lam / 2 * beta @ beta


def _D(A, y, lam, alpha):  # eq. dual_obj evaluated densely
    N = A.shape[0]
    v = A.T @ alpha
    return -N / 2 * alpha @ alpha - v @ v / (2 * lam) + alpha @ y


def _tiny(seed, N, M, density=1.0):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, M)).astype(np.float32)
    if density < 1.0:
        A *= rng.random((N, M)) < density
    y = (A @ rng.standard_normal(M) + 0.1 * rng.standard_normal(N)).astype(np.float32)
    return A.astype(np.float64), y


def _run_primal(oracle, A, y, lam, n_epochs, seed=0):
    N, M = A.shape
    ptr, idx, val = segments(A, "csc")
    beta = np.zeros(M)
    w = np.zeros(N)
    oracle.epochs("ridge_primal", N, M, ptr, idx, val, y, lam, seed, 0, n_epochs, beta, w)
    return beta, w, (ptr, idx, val)


@pytest.mark.parametrize("seed,N,M,density,lam", [(0, 20, 5, 1.0, 1e-2), (1, 50, 10, 0.5, 1e-3),
                                                  (2, 7, 10, 1.0, 1e-1), (3, 40, 8, 0.3, 1.0)])
def test_primal_reaches_closed_form(oracle, seed, N, M, density, lam):
    A, y = _tiny(seed, N, M, density)
    beta, w, _ = _run_primal(oracle, A, y, lam, 400)
    star = _closed_form(A, y.astype(np.float64), lam)
    assert rel_inf(beta, star) <= 1e-10


def test_primal_dense_ridge_workload_matches_normal_equations(oracle, synth):
    p = synth.make("dense_ridge")
    A = np.zeros((p.n_rows, p.n_cols))
    for m in range(p.n_cols):
        A[p.idx[p.ptr[m]:p.ptr[m + 1]], m] = p.val[p.ptr[m]:p.ptr[m + 1]]
    beta = np.zeros(p.n_cols)
    w = np.zeros(p.n_rows)
    oracle.epochs("ridge_primal", p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 0, 0, 50, beta, w)
    star = _closed_form(A, p.y.astype(np.float64), p.lam)
    assert rel_inf(beta, star) <= 1e-9
    P, D, G = oracle.objectives("ridge_primal", p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, beta)
    assert G <= 1e-9 * abs(P)


def test_strong_duality_at_closed_form(oracle):
    A, y = _tiny(4, 60, 12, 0.6)
    lam = 3e-2
    star = _closed_form(A, y.astype(np.float64), lam)
    ptr, idx, val = segments(A, "csc")
    P, D, G = oracle.objectives("ridge_primal", 60, 12, ptr, idx, val, y, lam, star)
    assert abs(P - _P(A, y, lam, star)) <= 1e-12 * abs(P)
    assert abs(D - _D(A, y, lam, (y - A @ star) / 60)) <= 1e-12 * abs(P)
    assert G <= 1e-12 * abs(P)
    # Away from the optimum the gap is clearly positive.
    _, _, G1 = oracle.objectives("ridge_primal", 60, 12, ptr, idx, val, y, lam, star * 0.9)
    assert G1 > 1e-6


def test_primal_step_is_exact_1d_minimiser(oracle):
    A, y = _tiny(5, 30, 6, 0.7)
    N, M = A.shape
    lam = 5e-2
    ptr, idx, val = segments(A, "csc")
    rng = np.random.default_rng(0)
    beta = rng.standard_normal(M)
    w = A @ beta
    for m in [0, 3, 5, 2]:
        before = beta.copy()
        oracle.visit("ridge_primal", N, M, ptr, idx, val, y, lam, [m], beta, w)
        e = np.zeros(M)
        e[m] = 1.0
        res = minimize_scalar(lambda t: _P(A, y, lam, before + t * e), bracket=(-1, 1), tol=1e-12)
        assert abs((beta[m] - before[m]) - res.x) <= 1e-6 * max(1.0, abs(res.x))
        assert np.array_equal(np.delete(beta, m), np.delete(before, m))
        np.testing.assert_allclose(w, A @ beta, rtol=0, atol=1e-12 * max(1.0, np.abs(w).max()))


def test_primal_monotone_and_gap_to_zero(oracle):
    A, y = _tiny(6, 40, 15, 0.4)
    N, M = A.shape
    lam = 1e-2
    ptr, idx, val = segments(A, "csc")
    beta = np.zeros(M)
    w = np.zeros(N)
    last = _P(A, y, lam, beta)
    for m in oracle.permutation(0, 0, M).tolist() * 3:
        oracle.visit("ridge_primal", N, M, ptr, idx, val, y, lam, [m], beta, w)
        now = _P(A, y, lam, beta)
        assert now <= last + 1e-14 * abs(last)
        last = now
    gaps = []
    beta = np.zeros(M)
    w = np.zeros(N)
    for e in range(60):
        oracle.epochs("ridge_primal", N, M, ptr, idx, val, y, lam, 0, e, 1, beta, w)
        gaps.append(oracle.objectives("ridge_primal", N, M, ptr, idx, val, y, lam, beta)[2])
    assert gaps[-1] < 1e-11 and gaps[-1] < gaps[0] * 1e-8


def test_shared_vector_invariant(oracle, synth):
    p = synth.make("sparse_ridge", n_rows=3000, n_cols=1500, density=0.01)
    beta = np.zeros(p.C)
    w = np.zeros(p.L)
    oracle.epochs(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 0, 0, 3, beta, w)
    fresh = oracle.fresh_shared(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, beta)
    assert rel_inf(w, fresh) <= 1e-12


def test_resume_is_bit_exact(oracle, synth):
    p = synth.make("sparse_ridge", n_rows=2000, n_cols=1000, density=0.01)
    args = (p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 77)
    b1, w1 = np.zeros(p.C), np.zeros(p.L)
    oracle.epochs(*args, 0, 10, b1, w1)
    b2, w2 = np.zeros(p.C), np.zeros(p.L)
    oracle.epochs(*args, 0, 5, b2, w2)
    oracle.epochs(*args, 5, 5, b2, w2)
    assert np.array_equal(b1, b2) and np.array_equal(w1, w2)


def test_empty_column_stays_zero(oracle):
    A, y = _tiny(7, 10, 4)
    A[:, 2] = 0.0
    ptr, idx, val = segments(A, "csc")
    assert ptr[3] == ptr[2]
    beta = np.array([0.0, 0.0, 5.0, 0.0])  # a nonzero weight on an empty column is pulled to 0
    w = A @ beta
    oracle.visit("ridge_primal", 10, 4, ptr, idx, val, y, 0.1, [2], beta, w)
    assert beta[2] == 0.0


def test_dual_reaches_optimality_conditions(oracle):
    A, y = _tiny(8, 25, 10, 0.6)
    N, M = A.shape
    lam = 2e-2
    ptr, idx, val = segments(A, "csr")
    alpha = np.zeros(N)
    wbar = np.zeros(M)
    oracle.epochs("ridge_dual", N, M, ptr, idx, val, y, lam, 0, 0, 600, alpha, wbar)
    star = _closed_form(A, y.astype(np.float64), lam)
    assert rel_inf(alpha, (y - A @ star) / N) <= 1e-9     # eq. duality-2
    assert rel_inf(wbar / lam, star) <= 1e-9              # eq. duality-1
    P, D, G = oracle.objectives("ridge_dual", N, M, ptr, idx, val, y, lam, alpha)
    assert abs(P - _P(A, y, lam, star)) <= 1e-10 * abs(P)
    assert G <= 1e-10 * abs(P)


def test_dual_step_is_exact_1d_maximiser(oracle):
    A, y = _tiny(9, 12, 20, 0.5)
    N, M = A.shape
    lam = 1e-1
    ptr, idx, val = segments(A, "csr")
    rng = np.random.default_rng(1)
    alpha = 0.1 * rng.standard_normal(N)
    wbar = A.T @ alpha
    for n in [0, 7, 11]:
        before = alpha.copy()
        oracle.visit("ridge_dual", N, M, ptr, idx, val, y, lam, [n], alpha, wbar)
        e = np.zeros(N)
        e[n] = 1.0
        res = minimize_scalar(lambda t: -_D(A, y, lam, before + t * e), bracket=(-1, 1), tol=1e-12)
        assert abs((alpha[n] - before[n]) - res.x) <= 1e-6 * max(1.0, abs(res.x))
        np.testing.assert_allclose(wbar, A.T @ alpha, rtol=0, atol=1e-12)


def test_gather_dots_and_norms_match_sparse_library(oracle, synth):
    # The per-coordinate inner products <a_c, u> are A^T u (CSC) or A u (CSR): scipy's sparse product.
    import scipy.sparse as sps
    p = synth.make("sparse_ridge", n_rows=4000, n_cols=3000, density=0.01)
    A = sps.csc_matrix((p.val.astype(np.float64), p.idx, p.ptr), shape=(p.n_rows, p.n_cols))
    u = np.random.default_rng(0).standard_normal(p.n_rows).astype(np.float32)
    d, cond = oracle.gather_dots(p.ptr, p.idx, p.val, u)
    np.testing.assert_allclose(d, A.T @ u.astype(np.float64), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(cond, abs(A).T @ np.abs(u.astype(np.float64)), rtol=1e-12)
    np.testing.assert_allclose(oracle.norms(p.ptr, p.val), np.asarray(A.multiply(A).sum(axis=0)).ravel(),
                               rtol=1e-12)
    q = synth.make("click_svm", n_rows=2000, n_cols=5000, row_nnz=10)
    X = sps.csr_matrix((q.val.astype(np.float64), q.idx, q.ptr), shape=(q.n_rows, q.n_cols))
    v = np.random.default_rng(1).standard_normal(q.n_cols).astype(np.float32)
    np.testing.assert_allclose(oracle.gather_dots(q.ptr, q.idx, q.val, v)[0], X @ v.astype(np.float64),
                               rtol=1e-12, atol=1e-12)
