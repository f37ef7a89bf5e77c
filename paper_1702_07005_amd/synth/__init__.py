"""Seeded synthetic workloads shaped like the paper's data (inputs only).

This module makes inputs and nothing else: it holds none of the coordinate-descent
arithmetic.  Both the HIP path (tests, benchmark) and the oracle's tests draw their
inputs from here.

Workloads (sizes are the defaults; every field can be overridden for scaled-down twins):

* ``dense_ridge``     2,000 x 200 dense N(0,1) matrix, y = A x* + 0.01 N(0,1), ridge primal over
                      CSC columns, lambda = 1e-3 (paper's normalised lambda, Sec. II-A).
* ``sparse_ridge``    100,000 x 50,000, each entry present with probability 1e-3, values N(0,1),
                      rows scaled to unit norm, y = A x* + 0.01 N(0,1), ridge primal over CSC,
                      lambda = 1e-2.
* ``text_svm``        350,000 x 16.6M, 3,700 distinct Zipf(1.1)-popular columns per row,
                      lognormal values, unit rows, labels = sign of a sparse random hyperplane
                      with 5% flipped; hinge SVM dual over CSR rows, lambda = 1/N.  Stand-in for
                      the webspam sample of Sec. III-D.
* ``text_ridge_csc``  the ``text_svm`` matrix and its +-1 labels stored by columns; ridge primal
                      over CSC, lambda = 1/N.
* ``click_svm``       50M x 75M, 39 one-hot fields with Zipf(1.2) cardinalities and value
                      frequencies, binary values scaled to unit rows, labels +1 with prob. 0.03;
                      hinge SVM dual over CSR, lambda = 1/N.  Stand-in for one of four workers'
                      shares of the criteo sample of Sec. V-B.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.cpp")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["g++", "-O3", "-std=c++17", "-fPIC", "-shared", "-fopenmp", "-Wall",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Spec(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("normalize", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("n_rows", ctypes.c_int64),
        ("n_cols", ctypes.c_int64),
        ("density", ctypes.c_double),
        ("row_nnz", ctypes.c_int32),
        ("pad_", ctypes.c_int32),
        ("zipf_s", ctypes.c_double),
        ("noise", ctypes.c_double),
        ("hyper_frac", ctypes.c_double),
        ("flip", ctypes.c_double),
        ("pos_rate", ctypes.c_double),
    ]


_lib = None


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        p = ctypes.c_void_p
        L.synth_row_lengths.argtypes = [ctypes.POINTER(_Spec), p, ctypes.c_int]
        L.synth_fill.argtypes = [ctypes.POINTER(_Spec), p, p, p, p, ctypes.c_int]
        L.synth_fields.argtypes = [ctypes.POINTER(_Spec), p, p]
        L.synth_zipf_draws.argtypes = [ctypes.c_double, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int64, p]
        L.synth_csr_to_csc.argtypes = [ctypes.c_int64, ctypes.c_int64, p, p, p, p, p, p, ctypes.c_int]
        _lib = L
    return _lib


def _threads() -> int:
    n = os.environ.get("OMP_NUM_THREADS")
    try:
        return max(1, int(n)) if n else max(1, min(16, os.cpu_count() or 1))
    except ValueError:
        return 1


def _pp(a):
    return a.ctypes.data_as(ctypes.c_void_p)


@dataclasses.dataclass
class Problem:
    """One generated problem.  ``ptr/idx/val`` are the coordinate segments: CSC columns
    for ``ridge_primal``, CSR rows for ``svm_dual`` / ``ridge_dual``."""

    name: str
    form: str
    layout: str
    n_rows: int
    n_cols: int
    ptr: np.ndarray
    idx: np.ndarray
    val: np.ndarray
    y: np.ndarray
    lam: float
    seed: int

    @property
    def nnz(self) -> int:
        return int(self.ptr[-1])

    @property
    def C(self) -> int:  # number of coordinates
        return self.n_cols if self.form == "ridge_primal" else self.n_rows

    @property
    def L(self) -> int:  # length of the shared vector
        return self.n_rows if self.form == "ridge_primal" else self.n_cols


def _csr(spec: _Spec):
    L = _L()
    n = spec.n_rows
    lens = np.empty(n, dtype=np.int64)
    if L.synth_row_lengths(ctypes.byref(spec), _pp(lens), _threads()) != 0:
        raise ValueError("invalid synthetic spec")
    ptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lens, out=ptr[1:])
    nnz = int(ptr[-1])
    idx = np.empty(nnz, dtype=np.int32)
    val = np.empty(nnz, dtype=np.float32)
    y = np.empty(n, dtype=np.float32)
    if L.synth_fill(ctypes.byref(spec), _pp(ptr), _pp(idx), _pp(val), _pp(y), _threads()) != 0:
        raise RuntimeError("synthetic fill failed")
    return ptr, idx, val, y


def csr_to_csc(n_rows, n_cols, ptr, idx, val):
    """Transpose (deterministic, rows sorted within every column)."""
    ptr = np.ascontiguousarray(ptr, dtype=np.int64)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    nnz = int(ptr[-1])
    cptr = np.empty(n_cols + 1, dtype=np.int64)
    ridx = np.empty(nnz, dtype=np.int32)
    cval = np.empty(nnz, dtype=np.float32)
    if _L().synth_csr_to_csc(n_rows, n_cols, _pp(ptr), _pp(idx), _pp(val), _pp(cptr), _pp(ridx), _pp(cval),
                             _threads()) != 0:
        raise ValueError("column index out of range")
    return cptr, ridx, cval


def zipf_draws(s: float, n: int, count: int, seed: int = 0) -> np.ndarray:
    out = np.empty(count, dtype=np.int64)
    if _L().synth_zipf_draws(s, n, seed, count, _pp(out)) != 0:
        raise ValueError("bad zipf parameters")
    return out


def click_fields(n_cols: int = 75_000_000, n_fields: int = 39, zipf_s: float = 1.2):
    sp = _Spec(kind=3, normalize=1, seed=0, n_rows=0, n_cols=n_cols, row_nnz=n_fields, zipf_s=zipf_s)
    card = np.empty(n_fields, dtype=np.int64)
    off = np.empty(n_fields, dtype=np.int64)
    if _L().synth_fields(ctypes.byref(sp), _pp(card), _pp(off)) != 0:
        raise ValueError("bad field spec")
    return card, off


# --------------------------------------------------------------------------- workloads

DEFAULTS = {
    "dense_ridge": dict(n_rows=2_000, n_cols=200, noise=0.01, lam=1e-3),
    "sparse_ridge": dict(n_rows=100_000, n_cols=50_000, density=1e-3, noise=0.01, lam=1e-2),
    "text_svm": dict(n_rows=350_000, n_cols=16_600_000, row_nnz=3_700, zipf_s=1.1, hyper_frac=0.01,
                     flip=0.05, lam=None),
    "text_ridge_csc": dict(n_rows=350_000, n_cols=16_600_000, row_nnz=3_700, zipf_s=1.1, hyper_frac=0.01,
                           flip=0.05, lam=None),
    "click_svm": dict(n_rows=50_000_000, n_cols=75_000_000, row_nnz=39, zipf_s=1.2, pos_rate=0.03, lam=None),
}


def make(name: str, seed: int = 0, **over) -> Problem:
    """Generate workload ``name`` (see module docstring); keyword overrides scale it down.
    ``lam=None`` means lambda = 1/N."""
    if name not in DEFAULTS:
        raise KeyError(f"unknown workload {name!r}; choose from {sorted(DEFAULTS)}")
    p = dict(DEFAULTS[name])
    unknown = set(over) - set(p)
    if unknown:
        raise KeyError(f"unknown overrides {sorted(unknown)} for {name}")
    p.update(over)
    n, m = int(p["n_rows"]), int(p["n_cols"])
    lam = p["lam"] if p["lam"] is not None else 1.0 / n
    if name == "dense_ridge":
        sp = _Spec(kind=0, normalize=0, seed=seed, n_rows=n, n_cols=m, noise=p["noise"])
    elif name == "sparse_ridge":
        sp = _Spec(kind=1, normalize=1, seed=seed, n_rows=n, n_cols=m, density=p["density"], noise=p["noise"])
    elif name in ("text_svm", "text_ridge_csc"):
        # Both names draw the same matrix and labels for a given seed.
        sp = _Spec(kind=2, normalize=1, seed=seed, n_rows=n, n_cols=m, row_nnz=int(p["row_nnz"]),
                   zipf_s=p["zipf_s"], hyper_frac=p["hyper_frac"], flip=p["flip"])
    else:
        sp = _Spec(kind=3, normalize=1, seed=seed, n_rows=n, n_cols=m, row_nnz=int(p["row_nnz"]),
                   zipf_s=p["zipf_s"], pos_rate=p["pos_rate"])
    ptr, idx, val, y = _csr(sp)
    if name in ("dense_ridge", "sparse_ridge", "text_ridge_csc"):
        cptr, ridx, cval = csr_to_csc(n, m, ptr, idx, val)
        del ptr, idx, val
        return Problem(name, "ridge_primal", "csc", n, m, cptr, ridx, cval, y, lam, seed)
    return Problem(name, "svm_dual", "csr", n, m, ptr, idx, val, y, lam, seed)


def as_ridge_dual(prob: Problem) -> Problem:
    """The same data as a ridge-regression dual problem over CSR rows (Sec. II-B)."""
    if prob.layout == "csr":
        return dataclasses.replace(prob, form="ridge_dual")
    ptr, idx, val = csc_to_csr(prob)
    return dataclasses.replace(prob, form="ridge_dual", layout="csr", ptr=ptr, idx=idx, val=val)


def csc_to_csr(prob: Problem):
    # Transposing the CSC arrays of an (N x M) matrix is the CSR->CSC routine on the (M x N) matrix.
    return csr_to_csc(prob.n_cols, prob.n_rows, prob.ptr, prob.idx, prob.val)
