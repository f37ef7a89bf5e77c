"""Python face of the fp64 sequential oracle (``scd_oracle.c``).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline leg of
the benchmark may import this module; the product package never does.  It shares no
code with the HIP library.

Every function takes plain numpy arrays: a sparse matrix is given by the segment
arrays of its coordinates (``ptr`` int64[C+1], ``idx`` int32[nnz], ``val`` float32[nnz]),
i.e. CSC columns for the ridge primal (coordinates = features, Alg. 1) and CSR rows
for the duals (coordinates = examples, Sec. II-B).  Models and shared vectors are
float64 and updated in place.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "scd_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
# A different build of the same source (used by the planted-mistake test) can be selected here.
_LOAD_PATH = os.environ.get("SCD_ORACLE_LIB", _LIB_PATH)

_i64 = ctypes.c_int64
_u64 = ctypes.c_uint64
_i32 = ctypes.c_int32
_u32 = ctypes.c_uint32
_dbl = ctypes.c_double
_p = ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no HIP involved)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _LOAD_PATH == _LIB_PATH and not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LOAD_PATH)
        L.oracle_splitmix64_mix.restype = _u64
        L.oracle_splitmix64_mix.argtypes = [_u64]
        L.oracle_splitmix64_nth.restype = _u64
        L.oracle_splitmix64_nth.argtypes = [_u64, _u64]
        L.oracle_fmix32.restype = _u32
        L.oracle_fmix32.argtypes = [_u32]
        L.oracle_perm_keys.restype = None
        L.oracle_perm_keys.argtypes = [_u64, _u64, _p]
        L.oracle_perm_half_bits.restype = ctypes.c_int
        L.oracle_perm_half_bits.argtypes = [_u64]
        L.oracle_perm_at.restype = _u64
        L.oracle_perm_at.argtypes = [_u64, _u64, _u64, _u64]
        L.oracle_permutation.restype = None
        L.oracle_permutation.argtypes = [_u64, _u64, _i64, _p]
        L.oracle_norms.restype = None
        L.oracle_norms.argtypes = [_i64, _p, _p, _p]
        L.oracle_gather_dots.restype = None
        L.oracle_gather_dots.argtypes = [_i64, _p, _p, _p, _p, _p, _p]
        for name in ("oracle_ridge_primal_visit", "oracle_ridge_dual_visit", "oracle_svm_dual_visit"):
            f = getattr(L, name)
            f.restype = None
            f.argtypes = [_i64, _p, _p, _p, _p, _dbl, _p, _i64, _p, _p, _p]
        for name in ("oracle_ridge_primal_epochs", "oracle_ridge_dual_epochs", "oracle_svm_dual_epochs"):
            f = getattr(L, name)
            f.restype = None
            f.argtypes = [_i64, _i64, _p, _p, _p, _p, _dbl, _u64, _i64, _i32, _p, _p]
        L.oracle_epochs_f32.restype = None
        L.oracle_epochs_f32.argtypes = [ctypes.c_int, _i64, _i64, _p, _p, _p, _p, _dbl, _u64, _i64, _i32, _p, _p]
        for name in ("oracle_ridge_primal_objectives", "oracle_ridge_dual_objectives",
                     "oracle_svm_dual_objectives"):
            f = getattr(L, name)
            f.restype = None
            f.argtypes = [_i64, _i64, _p, _p, _p, _p, _dbl, _p, _p, _p, _p, _p]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_p)


def _seg(ptr, idx, val):
    ptr = np.ascontiguousarray(ptr, dtype=np.int64)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    val = np.ascontiguousarray(val, dtype=np.float32)
    return ptr, idx, val


def _f64_inplace(a, n, what):
    if not (isinstance(a, np.ndarray) and a.dtype == np.float64 and a.flags.c_contiguous and a.shape == (n,)):
        raise TypeError(f"{what} must be a contiguous float64 array of length {n}")
    return a


# --------------------------------------------------------------------------- permutation

def splitmix64_mix(z: int) -> int:
    return int(lib().oracle_splitmix64_mix(z & 0xFFFFFFFFFFFFFFFF))


def splitmix64_nth(s: int, n: int) -> int:
    return int(lib().oracle_splitmix64_nth(s & 0xFFFFFFFFFFFFFFFF, n))


def fmix32(h: int) -> int:
    return int(lib().oracle_fmix32(h & 0xFFFFFFFF))


def perm_keys(seed: int, epoch: int) -> np.ndarray:
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_perm_keys(seed & 0xFFFFFFFFFFFFFFFF, epoch, _ptr(out))
    return out


def perm_half_bits(C: int) -> int:
    return int(lib().oracle_perm_half_bits(C))


def perm_at(seed: int, epoch: int, C: int, j: int) -> int:
    return int(lib().oracle_perm_at(seed & 0xFFFFFFFFFFFFFFFF, epoch, C, j))


def permutation(seed: int, epoch: int, C: int) -> np.ndarray:
    """Visiting order of epoch ``epoch``: out[j] = coordinate visited at position j."""
    out = np.empty(max(C, 0), dtype=np.int64)
    if C > 0:
        lib().oracle_permutation(seed & 0xFFFFFFFFFFFFFFFF, epoch, C, _ptr(out))
    return out


# --------------------------------------------------------------------------- segments

def norms(ptr, val) -> np.ndarray:
    ptr = np.ascontiguousarray(ptr, dtype=np.int64)
    val = np.ascontiguousarray(val, dtype=np.float32)
    C = ptr.shape[0] - 1
    out = np.empty(C, dtype=np.float64)
    lib().oracle_norms(C, _ptr(ptr), _ptr(val), _ptr(out))
    return out


def gather_dots(ptr, idx, val, u):
    """(dots, cond): dots[c] = <a_c, u>, cond[c] = sum |a_c||u| over the segment, fp64."""
    ptr, idx, val = _seg(ptr, idx, val)
    u = np.ascontiguousarray(u, dtype=np.float32)
    C = ptr.shape[0] - 1
    out = np.empty(C, dtype=np.float64)
    cond = np.empty(C, dtype=np.float64)
    lib().oracle_gather_dots(C, _ptr(ptr), _ptr(idx), _ptr(val), _ptr(u), _ptr(out), _ptr(cond))
    return out, cond


# --------------------------------------------------------------------------- solvers

_FORMS = {
    "ridge_primal": ("oracle_ridge_primal_visit", "oracle_ridge_primal_epochs",
                     "oracle_ridge_primal_objectives"),
    "ridge_dual": ("oracle_ridge_dual_visit", "oracle_ridge_dual_epochs", "oracle_ridge_dual_objectives"),
    "svm_dual": ("oracle_svm_dual_visit", "oracle_svm_dual_epochs", "oracle_svm_dual_objectives"),
}


def _dims(form, n_rows, n_cols):
    """(C, L): number of coordinates and length of the shared vector."""
    if form == "ridge_primal":
        return n_cols, n_rows
    return n_rows, n_cols


def visit(form, n_rows, n_cols, ptr, idx, val, y, lam, coords, model, shared, seg_norms=None):
    """Exact coordinate steps for ``coords`` in order (one step per entry)."""
    ptr, idx, val = _seg(ptr, idx, val)
    y = np.ascontiguousarray(y, dtype=np.float32)
    C, L = _dims(form, n_rows, n_cols)
    _f64_inplace(model, C, "model")
    _f64_inplace(shared, L, "shared")
    coords = np.ascontiguousarray(coords, dtype=np.int64)
    if coords.size and (coords.min() < 0 or coords.max() >= C):
        raise IndexError("coordinate out of range")
    if seg_norms is None:
        seg_norms = norms(ptr, val)
    f = getattr(lib(), _FORMS[form][0])
    f(n_rows, _ptr(ptr), _ptr(idx), _ptr(val), _ptr(y), lam, _ptr(coords), coords.shape[0],
      _ptr(np.ascontiguousarray(seg_norms, dtype=np.float64)), _ptr(model), _ptr(shared))


def epochs(form, n_rows, n_cols, ptr, idx, val, y, lam, seed, epoch0, n_epochs, model, shared):
    """Alg. 1: ``n_epochs`` permuted passes; global epoch index starts at ``epoch0``."""
    ptr, idx, val = _seg(ptr, idx, val)
    y = np.ascontiguousarray(y, dtype=np.float32)
    C, L = _dims(form, n_rows, n_cols)
    _f64_inplace(model, C, "model")
    _f64_inplace(shared, L, "shared")
    f = getattr(lib(), _FORMS[form][1])
    f(n_rows, n_cols, _ptr(ptr), _ptr(idx), _ptr(val), _ptr(y), lam, seed & 0xFFFFFFFFFFFFFFFF,
      epoch0, n_epochs, _ptr(model), _ptr(shared))


_F32_FORMS = {"ridge_primal": 0, "svm_dual": 1, "ridge_dual": 2}


def epochs_f32(form, n_rows, n_cols, ptr, idx, val, y, lam, seed, epoch0, n_epochs, model, shared):
    """Alg. 1 in single precision (the paper's CPU baseline precision), for timing only:
    ``model`` and ``shared`` are float32 arrays updated in place."""
    ptr, idx, val = _seg(ptr, idx, val)
    y = np.ascontiguousarray(y, dtype=np.float32)
    C, L = _dims(form, n_rows, n_cols)
    for a, n, what in ((model, C, "model"), (shared, L, "shared")):
        if not (isinstance(a, np.ndarray) and a.dtype == np.float32 and a.flags.c_contiguous and a.shape == (n,)):
            raise ValueError(f"{what} must be a contiguous float32 array of length {n}")
    lib().oracle_epochs_f32(_F32_FORMS[form], n_rows, n_cols, _ptr(ptr), _ptr(idx), _ptr(val), _ptr(y), lam,
                            seed & 0xFFFFFFFFFFFFFFFF, epoch0, n_epochs, _ptr(model), _ptr(shared))


def objectives(form, n_rows, n_cols, ptr, idx, val, y, lam, model, shared=None):
    """(P, D, gap).  ``shared=None`` recomputes the shared vector fresh from the model."""
    ptr, idx, val = _seg(ptr, idx, val)
    y = np.ascontiguousarray(y, dtype=np.float32)
    C, L = _dims(form, n_rows, n_cols)
    model = np.ascontiguousarray(model, dtype=np.float64)
    if model.shape != (C,):
        raise ValueError("model length")
    if shared is not None:
        shared = np.ascontiguousarray(shared, dtype=np.float64)
        if shared.shape != (L,):
            raise ValueError("shared length")
    P = _dbl()
    D = _dbl()
    G = _dbl()
    f = getattr(lib(), _FORMS[form][2])
    f(n_rows, n_cols, _ptr(ptr), _ptr(idx), _ptr(val), _ptr(y), lam, _ptr(model), _ptr(shared),
      ctypes.byref(P), ctypes.byref(D), ctypes.byref(G))
    return P.value, D.value, G.value


def fresh_shared(form, n_rows, n_cols, ptr, idx, val, y, lam, model):
    """Shared vector recomputed from the model in fp64: A beta (ridge primal),
    A^T alpha (ridge dual), sum_i alpha_i y_i x_i / (lambda N) (SVM dual)."""
    ptr, idx, val = _seg(ptr, idx, val)
    C, L = _dims(form, n_rows, n_cols)
    model = np.asarray(model, dtype=np.float64)
    seg_of = np.repeat(np.arange(C, dtype=np.int64), np.diff(ptr))
    coef = model[seg_of]
    if form == "svm_dual":
        coef = coef * np.asarray(y, dtype=np.float64)[seg_of] / (lam * n_rows)
    out = np.zeros(L, dtype=np.float64)
    np.add.at(out, idx, val.astype(np.float64) * coef)
    return out
