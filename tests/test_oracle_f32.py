"""Pins of the single-precision copy of the oracle's epochs (the paper's CPU baseline
precision, used only for timing beside the fp64 oracle).

Ridge primal: the closed-form minimiser (A^T A + N lambda I)^-1 A^T y at fp32 accuracy.
Ridge dual: alpha* = (y - A beta*)/N (eqs. duality-1/2) at fp32 accuracy.
Hinge SVM dual: w* of the active-set brute force at fp32 accuracy.
All three: the visiting order and the steps of the fp64 oracle (one epoch from zero agrees to
fp32 rounding), and the shared vector equals the one recomputed from the model.
"""
import numpy as np
import pytest

from tests._helpers import rel_inf, segments
from tests.test_oracle_svm import _brute_force


def _dense(seed, N, M, labels=False):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, M)).astype(np.float32)
    if labels:
        y = np.where(rng.random(N) < 0.5, -1.0, 1.0).astype(np.float32)
    else:
        y = (A @ rng.standard_normal(M).astype(np.float32) + 0.1 * rng.standard_normal(N)).astype(np.float32)
    return A.astype(np.float64), y


def _run(oracle, form, A, y, lam, epochs, layout):
    N, M = A.shape
    ptr, idx, val = segments(A, layout)
    C, L = (M, N) if form == "ridge_primal" else (N, M)
    model = np.zeros(C, dtype=np.float32)
    shared = np.zeros(L, dtype=np.float32)
    oracle.epochs_f32(form, N, M, ptr, idx, val, y, lam, 0, 0, epochs, model, shared)
    fresh = oracle.fresh_shared(form, N, M, ptr, idx, val, y, lam, model.astype(np.float64))
    assert rel_inf(shared, fresh) <= 1e-4
    return model.astype(np.float64), (ptr, idx, val)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ridge_primal_reaches_closed_form(oracle, seed):
    A, y = _dense(seed, 40, 8)
    lam = 0.05
    beta, _ = _run(oracle, "ridge_primal", A, y, lam, 300, "csc")
    N, M = A.shape
    star = np.linalg.solve(A.T @ A + N * lam * np.eye(M), A.T @ y.astype(np.float64))
    assert rel_inf(beta, star) <= 1e-4


def test_ridge_dual_reaches_closed_form(oracle):
    A, y = _dense(3, 30, 10)
    lam = 0.05
    alpha, _ = _run(oracle, "ridge_dual", A, y, lam, 400, "csr")
    N, M = A.shape
    beta = np.linalg.solve(A.T @ A + N * lam * np.eye(M), A.T @ y.astype(np.float64))
    assert rel_inf(alpha, (y - A @ beta) / N) <= 1e-4


@pytest.mark.parametrize("seed,N,M,lam", [(0, 5, 3, 0.1), (1, 7, 4, 0.05), (4, 8, 5, 1.0)])
def test_svm_dual_reaches_brute_force(oracle, seed, N, M, lam):
    X, y = _dense(seed, N, M, labels=True)
    _, wstar, _ = _brute_force(X, y.astype(np.float64), lam)
    a, (ptr, idx, val) = _run(oracle, "svm_dual", X, y, lam, 3000, "csr")
    assert np.all(a >= 0) and np.all(a <= 1)
    w = oracle.fresh_shared("svm_dual", N, M, ptr, idx, val, y, lam, a)
    assert rel_inf(w, wstar) <= 1e-4


@pytest.mark.parametrize("form,layout", [("ridge_primal", "csc"), ("ridge_dual", "csr"), ("svm_dual", "csr")])
def test_one_epoch_matches_fp64_oracle(oracle, form, layout):
    A, y = _dense(5, 60, 25, labels=form == "svm_dual")
    lam = 0.02
    N, M = A.shape
    ptr, idx, val = segments(A, layout)
    C, L = (M, N) if form == "ridge_primal" else (N, M)
    m32, s32 = np.zeros(C, dtype=np.float32), np.zeros(L, dtype=np.float32)
    m64, s64 = np.zeros(C), np.zeros(L)
    oracle.epochs_f32(form, N, M, ptr, idx, val, y, lam, 7, 3, 1, m32, s32)
    oracle.epochs(form, N, M, ptr, idx, val, y, lam, 7, 3, 1, m64, s64)
    assert rel_inf(m32, m64) <= 1e-4
    assert rel_inf(s32, s64) <= 1e-4
