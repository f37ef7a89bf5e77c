"""The seeded input generator: determinism, shapes and distributions of every workload."""
import numpy as np
import pytest
import scipy.sparse as sps


def _same(a, b):
    return all(np.array_equal(getattr(a, k), getattr(b, k)) for k in ("ptr", "idx", "val", "y"))


@pytest.mark.parametrize("name,over", [("sparse_ridge", dict(n_rows=3000, n_cols=2000, density=0.01)),
                                       ("text_svm", dict(n_rows=500, n_cols=20000, row_nnz=60)),
                                       ("click_svm", dict(n_rows=2000, n_cols=30000, row_nnz=39)),
                                       ("text_ridge_csc", dict(n_rows=500, n_cols=20000, row_nnz=60))])
def test_deterministic_for_any_thread_count(synth, monkeypatch, name, over):
    monkeypatch.setattr(synth, "_threads", lambda: 1)
    a = synth.make(name, seed=3, **over)
    monkeypatch.setattr(synth, "_threads", lambda: 7)
    b = synth.make(name, seed=3, **over)
    assert _same(a, b)
    c = synth.make(name, seed=4, **over)
    assert not (np.array_equal(a.idx, c.idx) and np.array_equal(a.val, c.val))


def test_dense_ridge_shape():
    from paper_1702_07005_amd import synth
    p = synth.make("dense_ridge")
    assert (p.form, p.layout, p.n_rows, p.n_cols, p.nnz) == ("ridge_primal", "csc", 2000, 200, 400_000)
    assert p.lam == 1e-3
    assert np.array_equal(np.diff(p.ptr), np.full(200, 2000))
    assert abs(p.val.mean()) < 0.01 and abs(p.val.std() - 1.0) < 0.01  # N(0,1), not normalised
    A = sps.csc_matrix((p.val, p.idx, p.ptr), shape=(2000, 200)).toarray()
    # y = A x* + 0.01 N(0,1): the least-squares residual has std close to 0.01.
    xs, *_ = np.linalg.lstsq(A.astype(np.float64), p.y.astype(np.float64), rcond=None)
    res = p.y - A @ xs
    assert 0.009 < res.std() < 0.011


def test_sparse_ridge_statistics(synth):
    p = synth.make("sparse_ridge", n_rows=20000, n_cols=10000, density=5e-3)
    assert p.layout == "csc" and p.lam == 1e-2
    dens = p.nnz / (p.n_rows * p.n_cols)
    assert abs(dens / 5e-3 - 1) < 0.02
    R = sps.csc_matrix((p.val.astype(np.float64), p.idx, p.ptr), shape=(p.n_rows, p.n_cols)).tocsr()
    rn = np.sqrt(np.asarray(R.multiply(R).sum(axis=1)).ravel())
    nz = np.diff(R.indptr) > 0
    assert np.allclose(rn[nz], 1.0, atol=1e-6)
    # Rows are sorted by column index and carry no duplicates (CSC rows sorted too).
    for m in range(0, p.n_cols, 997):
        seg = p.idx[p.ptr[m]:p.ptr[m + 1]]
        assert np.all(np.diff(seg) > 0)


def test_text_rows(synth):
    p = synth.make("text_svm", n_rows=800, n_cols=50000, row_nnz=300)
    assert p.form == "svm_dual" and p.layout == "csr" and p.lam == 1 / 800
    assert np.array_equal(np.diff(p.ptr), np.full(800, 300))
    for i in range(0, 800, 37):
        seg = p.idx[p.ptr[i]:p.ptr[i + 1]]
        v = p.val[p.ptr[i]:p.ptr[i + 1]].astype(np.float64)
        assert np.all(np.diff(seg) > 0) and seg.min() >= 0 and seg.max() < 50000
        assert np.all(v > 0) and abs(np.sqrt((v * v).sum()) - 1) < 1e-6
    assert set(np.unique(p.y).tolist()) <= {-1.0, 1.0}
    # Zipf popularity: the most popular column appears in (almost) every row.
    counts = np.bincount(p.idx, minlength=50000)
    assert counts.max() >= 0.98 * 800
    assert (counts > 0).sum() < 50000


def test_text_ridge_is_transpose_of_text_svm(synth):
    a = synth.make("text_svm", n_rows=300, n_cols=9000, row_nnz=50, seed=1)
    b = synth.make("text_ridge_csc", n_rows=300, n_cols=9000, row_nnz=50, seed=1)
    assert b.form == "ridge_primal" and b.layout == "csc"
    A = sps.csr_matrix((a.val, a.idx, a.ptr), shape=(300, 9000))
    B = sps.csc_matrix((b.val, b.idx, b.ptr), shape=(300, 9000))
    assert (A != B).nnz == 0
    assert np.array_equal(a.y, b.y)


def test_click_fields(synth):
    card, off = synth.click_fields()
    assert card.sum() == 75_000_000 and card.shape == (39,)
    assert np.all(np.diff(card) <= 0) and abs(card[0] / card[1] - 2 ** 1.2) < 0.01
    p = synth.make("click_svm", n_rows=5000, n_cols=100000)
    c2, o2 = synth.click_fields(100000)
    assert np.array_equal(np.diff(p.ptr), np.full(5000, 39))
    cols = p.idx.reshape(5000, 39)
    field = np.searchsorted(o2, cols, side="right") - 1
    assert np.array_equal(field, np.broadcast_to(np.arange(39), (5000, 39)))  # one value per field
    assert np.allclose(p.val, np.float32(1 / np.sqrt(39)))
    pos = (p.y > 0).mean()
    assert abs(pos - 0.03) < 0.01


@pytest.mark.parametrize("s", [1.1, 1.2, 2.0])
def test_zipf_sampler_matches_pmf(synth, s):
    n, draws = 60, 300_000
    x = synth.zipf_draws(s, n, draws, seed=5)
    assert x.min() >= 1 and x.max() <= n
    pmf = np.arange(1, n + 1, dtype=np.float64) ** -s
    pmf /= pmf.sum()
    obs = np.bincount(x, minlength=n + 1)[1:]
    exp = pmf * draws
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    assert chi2 < 110.0  # chi-square(59) 0.9999 quantile ~ 104


def test_transpose_matches_scipy(synth):
    M = sps.random(300, 500, density=0.03, random_state=1, format="csr", dtype=np.float32)
    ptr, idx, val = synth.csr_to_csc(300, 500, M.indptr.astype(np.int64), M.indices.astype(np.int32), M.data)
    C = M.tocsc()
    C.sort_indices()
    assert np.array_equal(ptr, C.indptr) and np.array_equal(idx, C.indices) and np.array_equal(val, C.data)
