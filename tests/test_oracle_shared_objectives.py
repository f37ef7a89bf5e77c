"""Pins of the oracle's objective evaluation from a maintained shared vector.

The objective functions take an optional shared vector that stands in for the one defined by the
model: w = A beta for the ridge primal (Sec. II-A), wbar = A^T alpha for the ridge dual
(Sec. II-B), w(alpha) = sum_i alpha_i y_i x_i / (lambda N) for the hinge SVM dual.  The GPU path
maintains that vector by atomic scatters, and the parity tests evaluate the oracle's reference
gaps with it, so this branch needs pins of its own:

  * fed the shared vector that a library sparse product (scipy) computes from the model, it must
    reproduce the fresh evaluation (which strong duality and the closed forms pin) to 1e-14;
  * fed a vector that differs from the model's in one entry that no segment touches, P and D must
    move by the amounts the definitions give in closed form for that entry alone (the entry enters
    only through the squared norm or the residual, never through a gathered product), so a branch
    that silently recomputes the vector, or reads it at the wrong index, fails.
"""
import numpy as np
import pytest

from tests._helpers import segments, to_scipy


def _tiny(seed, N, M, empty_row, empty_col):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((N, M)) * (rng.random((N, M)) < 0.6)
    A[empty_row, :] = 0.0
    A[:, empty_col] = 0.0
    return A.astype(np.float32).astype(np.float64)


def _scipy_shared(form, A, y, lam, model):
    """The shared vector of the model by a library sparse product (independent of the oracle)."""
    N = A.shape[0]
    if form == "ridge_primal":
        return to_scipy(*A.shape, "csc", *segments(A, "csc")) @ model
    X = to_scipy(*A.shape, "csr", *segments(A, "csr"))
    if form == "ridge_dual":
        return X.T @ model
    return X.T @ (model * y.astype(np.float64) / (lam * N))


CASES = [("ridge_primal", 0, 1e-2), ("ridge_dual", 1, 3e-2), ("svm_dual", 2, 5e-2)]


@pytest.mark.parametrize("form,seed,lam", CASES)
def test_maintained_shared_vector_equals_fresh(oracle, form, seed, lam):
    N, M = 30, 12
    A = _tiny(seed, N, M, empty_row=4, empty_col=7)
    rng = np.random.default_rng(seed + 10)
    if form == "svm_dual":
        y = np.where(rng.random(N) < 0.5, -1.0, 1.0).astype(np.float32)
        model = rng.random(N)
    else:
        y = rng.standard_normal(N).astype(np.float32)
        model = 0.1 * rng.standard_normal(M if form == "ridge_primal" else N)
    layout = "csc" if form == "ridge_primal" else "csr"
    ptr, idx, val = segments(A, layout)
    shared = _scipy_shared(form, A, y, lam, model)
    fresh = oracle.fresh_shared(form, N, M, ptr, idx, val, y, lam, model)
    assert np.max(np.abs(fresh - shared)) <= 1e-13 * max(np.max(np.abs(shared)), 1e-300)
    P0, D0, G0 = oracle.objectives(form, N, M, ptr, idx, val, y, lam, model)
    P1, D1, G1 = oracle.objectives(form, N, M, ptr, idx, val, y, lam, model, shared)
    scale = max(abs(P0), abs(D0))
    assert abs(P1 - P0) <= 1e-14 * scale and abs(D1 - D0) <= 1e-14 * scale
    assert abs(G1 - G0) <= 1e-14 * scale


@pytest.mark.parametrize("form,seed,lam", CASES)
def test_maintained_shared_vector_is_the_one_read(oracle, form, seed, lam):
    N, M = 30, 12
    er, ec = 4, 7
    A = _tiny(seed, N, M, empty_row=er, empty_col=ec)
    rng = np.random.default_rng(seed + 20)
    if form == "svm_dual":
        y = np.where(rng.random(N) < 0.5, -1.0, 1.0).astype(np.float32)
        model = rng.random(N)
    else:
        y = rng.standard_normal(N).astype(np.float32)
        model = 0.1 * rng.standard_normal(M if form == "ridge_primal" else N)
    layout = "csc" if form == "ridge_primal" else "csr"
    ptr, idx, val = segments(A, layout)
    shared = _scipy_shared(form, A, y, lam, model)
    P0, D0, _ = oracle.objectives(form, N, M, ptr, idx, val, y, lam, model, shared)
    delta = 0.37
    moved = shared.copy()
    if form == "ridge_primal":
        # Row er is empty: w_er enters P only through the residual r_er = w_er - y_er, and D only
        # through alpha_er = (y_er - w_er)/N (no column gathers row er).
        k = er
        moved[k] += delta
        r0, r1 = shared[k] - y[k], moved[k] - y[k]
        a0, a1 = -r0 / N, -r1 / N
        dP = (r1 * r1 - r0 * r0) / (2 * N)
        dD = -N / 2 * (a1 * a1 - a0 * a0) + (a1 - a0) * float(y[k])
    else:
        # Column ec is empty: its shared entry enters only through the squared norm of the shared
        # vector (no row gathers it).
        k = ec
        moved[k] += delta
        dn = moved[k] ** 2 - shared[k] ** 2
        if form == "ridge_dual":
            dP, dD = dn / (2 * lam), -dn / (2 * lam)  # P(wbar/lambda) has lambda/2 |wbar/lambda|^2
        else:
            dP, dD = lam / 2 * dn, -lam / 2 * dn
    P1, D1, _ = oracle.objectives(form, N, M, ptr, idx, val, y, lam, model, moved)
    scale = max(abs(P0), abs(D0), 1.0)
    assert abs((P1 - P0) - dP) <= 1e-13 * scale, (P1 - P0, dP)
    assert abs((D1 - D0) - dD) <= 1e-13 * scale, (D1 - D0, dD)
    assert abs(dP) > 1e-6 and abs(dD) > 1e-6
