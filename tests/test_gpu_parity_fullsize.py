"""GPU <-> oracle parity at the full sizes of the large workloads (1.3-1.95 billion stored entries),
in the launch configuration the solver picks by default.

The oracle cannot run these to convergence in a test, so the checks are the ones that hold at any
size, that it can compute one by one, or that it computed once:
  * gathered dots of 2,000 sampled coordinates on a frozen vector (oracle on those segments only),
    |gpu - fp64| <= 1e-4 * sum |a_i u_i|;
  * after each of the first 5 epochs and after the last, |w - A model|_inf / |w|_inf <= 1e-4 with
    A model recomputed in fp64 (scipy);
  * SVM box constraints after every epoch;
  * the duality gap after every epoch within 2x of the oracle's at the same epoch, plus the fp32
    floor 1e-6 P(0), against tests/golden/fullsize_gap_curves.json, which
    tests/golden/make_fullsize_curves.py writes from the oracle on the same seeded inputs.
"""
import gc
import json
import os

import numpy as np
import pytest

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import scipy.sparse as sps  # noqa: E402

from oracle import oracle as orc  # noqa: E402
from paper_1702_07005_amd import scd, synth  # noqa: E402


def _fresh_shared(p, model):
    """Shared vector from the model in fp64 (A beta, or sum_i alpha_i y_i x_i / (lambda N))."""
    if p.layout == "csc":  # columns are coordinates: A (N x M) times beta
        A = sps.csc_matrix((p.val, p.idx, p.ptr), shape=(p.n_rows, p.n_cols))
        return A @ model
    X = sps.csr_matrix((p.val, p.idx, p.ptr), shape=(p.n_rows, p.n_cols))
    return X.T @ (model * p.y.astype(np.float64) / (p.lam * p.n_rows))


def _sampled_dots(p, s, rng):
    u = rng.standard_normal(p.L).astype(np.float32)
    d = s.gather_dots(torch.from_numpy(u).cuda()).cpu().numpy().astype(np.float64)
    sample = np.sort(rng.choice(p.C, size=min(p.C, 2000), replace=False))
    lens = p.ptr[sample + 1] - p.ptr[sample]
    sptr = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    sidx = np.concatenate([p.idx[p.ptr[c]:p.ptr[c + 1]] for c in sample])
    sval = np.concatenate([p.val[p.ptr[c]:p.ptr[c + 1]] for c in sample])
    dref, cond = orc.gather_dots(sptr, sidx, sval, u)
    return np.abs(d[sample] - dref) / np.maximum(cond, 1e-30)


CURVES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fullsize_gap_curves.json")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["text_svm", "text_ridge_csc", "click_svm"])
def test_full_size(name):
    with open(CURVES) as f:
        ref = json.load(f)[name]
    print(f"full-size {name}: generating", flush=True)
    p = synth.make(name, seed=ref["seed"])
    rng = np.random.default_rng(0)
    s = scd.solver_for(p)
    info = s.info()
    print(f"  created: kernel {info['kernel']}, window {info['window']}, lanes {info['group_lanes']}, "
          f"coupling {info['coupling']:.3e}", flush=True)
    assert 1 <= info["window"] <= p.C
    err = _sampled_dots(p, s, rng)
    assert err.max() <= 1e-4, err.max()
    P0, _ = s.objective()
    assert abs(P0 - ref["P0"]) <= 1e-6 * abs(ref["P0"])
    for e, Gr in enumerate(ref["gap"]):
        s.epochs(ref["seed"], 1)
        G = s.duality_gap()
        print(f"  epoch {e + 1}: gap {G:.3e}, oracle {Gr:.3e}, ratio {G / Gr:.3f}", flush=True)
        assert G <= 2.0 * Gr + 1e-6 * abs(P0), (e + 1, G, Gr)
        last = e + 1 == len(ref["gap"])
        if e < 5 or last or p.form == "svm_dual":
            gm, gs, ep = s.get_state()
            assert ep == e + 1
            model = gm.cpu().numpy().astype(np.float64)
            if p.form == "svm_dual":
                assert model.min() >= 0.0 and model.max() <= 1.0
            if e < 5 or last:  # a lost update persists, so the last epoch covers the ones in between
                shared = gs.cpu().numpy().astype(np.float64)
                fresh = _fresh_shared(p, model)
                err = np.max(np.abs(shared - fresh)) / np.max(np.abs(fresh))
                print(f"  invariant after epoch {e + 1}: {err:.2e}", flush=True)
                assert err <= 1e-4, (e + 1, err)
                del shared, fresh
            del gm, gs, model
    s.close()
    del p, s
    gc.collect()
    torch.cuda.empty_cache()
