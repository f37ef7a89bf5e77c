"""The allocation-free entry point scd_objective_static against scd_objective through the C ABI.

For a state reached by asynchronous epochs, the handle-free evaluation must give the handle's
objectives (both fp64 reductions of fp32 data over the same state; they differ only in how
<a_c, y - w> is formed for the ridge primal -- from <y, a_c> computed at set-up, or gathered -- so
to 1e-9 relative, the tolerance for objectives of a given state).  Two calls in a row, the second
on a smaller input, check that the fixed scratch array keeps no state between calls.  Invalid
inputs are rejected by its validation pass without running the objective pass.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_1702_07005_amd import scd, synth  # noqa: E402

DEV = "cuda"


def _static(p, model, shared):
    ptr, idx, val, y = scd.upload(p, DEV)
    return scd.objective_static(p.n_rows, p.n_cols, ptr, idx, val, y, p.lam, p.form, model, shared)


def _case(p, epochs):
    s = scd.solver_for(p)
    assert s.info()["shared_fp64"] == 0  # the handle holds the same fp32 state that get_state returns
    s.epochs(0, epochs)
    P, D = s.objective()
    model, shared, _ = s.get_state()
    s.close()
    return P, D, model, shared


PROBLEMS = {
    "svm_click": lambda: (synth.make("click_svm", n_rows=50_000, n_cols=75_000),
                          synth.make("click_svm", n_rows=5_000, n_cols=9_000)),
    "ridge_primal": lambda: (synth.make("sparse_ridge", n_rows=20_000, n_cols=10_000, density=5e-3),
                             synth.make("sparse_ridge", n_rows=3_000, n_cols=800, density=2e-2)),
    "ridge_dual": lambda: (synth.as_ridge_dual(synth.make("sparse_ridge", n_rows=20_000, n_cols=10_000, density=5e-3)),
                           synth.as_ridge_dual(synth.make("dense_ridge", n_rows=600, n_cols=40))),
}


@pytest.mark.parametrize("name", sorted(PROBLEMS))
def test_static_objective_matches_handle(name):
    big, small = PROBLEMS[name]()
    for p, epochs in ((big, 3), (small, 2)):
        print(f"static objective {name}: {p.n_rows} x {p.n_cols}, {p.nnz} entries", flush=True)
        P, D, model, shared = _case(p, epochs)
        Ps, Ds = _static(p, model, shared)
        scale = max(abs(P), abs(D))
        assert abs(Ps - P) <= 1e-9 * scale and abs(Ds - D) <= 1e-9 * scale, (Ps, P, Ds, D)
        # and the oracle's evaluation of the same state, with the same maintained shared vector
        Pr, Dr, _ = orc.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam,
                                   model.cpu().numpy().astype(np.float64), shared.cpu().numpy().astype(np.float64))
        assert abs(Ps - Pr) <= 1e-9 * max(abs(Pr), abs(Dr)) and abs(Ds - Dr) <= 1e-9 * max(abs(Pr), abs(Dr))


def test_static_objective_rejects_invalid_inputs():
    p = synth.make("sparse_ridge", n_rows=2_000, n_cols=500, density=1e-2)
    ptr, idx, val, y = scd.upload(p, DEV)
    model = torch.zeros(p.C, device=DEV)
    shared = torch.zeros(p.L, device=DEV)
    bad = idx.clone()
    bad[7] = p.n_rows  # one row index out of range
    with pytest.raises(scd.ScdError) as ei:
        scd.objective_static(p.n_rows, p.n_cols, ptr, bad, val, y, p.lam, p.form, model, shared)
    assert ei.value.code == -1 and "outside" in str(ei.value)
    nan = val.clone()
    nan[3] = float("nan")
    with pytest.raises(scd.ScdError) as ei:
        scd.objective_static(p.n_rows, p.n_cols, ptr, idx, nan, y, p.lam, p.form, model, shared)
    assert ei.value.code == -5
    with pytest.raises(scd.ScdError) as ei:
        scd.objective_static(p.n_rows, p.n_cols, ptr, idx, val, y, 0.0, p.form, model, shared)
    assert ei.value.code == -1
    # a valid call after the rejected ones: at the zero state P = |y|^2 / (2N)
    P, D = scd.objective_static(p.n_rows, p.n_cols, ptr, idx, val, y, p.lam, p.form, model, shared)
    yy = p.y.astype(np.float64)
    assert abs(P - yy @ yy / (2 * p.n_rows)) <= 1e-9 * abs(P)
