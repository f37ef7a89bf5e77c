"""Small shared helpers for the tests (no coordinate-descent arithmetic here)."""
import numpy as np
import scipy.sparse as sps


def segments(A, layout):
    """(ptr int64, idx int32, val float32) of a dense or scipy matrix, by columns ("csc")
    or rows ("csr"); explicit zeros are dropped."""
    M = sps.csc_matrix(A) if layout == "csc" else sps.csr_matrix(A)
    M.eliminate_zeros()
    M.sort_indices()
    return (M.indptr.astype(np.int64), M.indices.astype(np.int32), M.data.astype(np.float32))


def to_scipy(n_rows, n_cols, layout, ptr, idx, val):
    if layout == "csc":
        return sps.csc_matrix((val.astype(np.float64), idx, ptr), shape=(n_rows, n_cols))
    return sps.csr_matrix((val.astype(np.float64), idx, ptr), shape=(n_rows, n_cols))


def rel_inf(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))
