"""Thin Python binding of libscd (include/scd.h): argument marshalling only.

Every step of the solver runs in the HIP kernels of ``libscd.so``; torch supplies device
memory (``data_ptr``) and the current HIP stream.  There is no fallback: if the library
is not built this module raises on import.

Method: asynchronous stochastic coordinate descent/ascent for generalized linear models,
arXiv 1702.07005 (Sec. II objectives and steps, Sec. III-C twice-parallel GPU epochs).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libscd.so")

RIDGE_PRIMAL, SVM_DUAL, RIDGE_DUAL = 0, 1, 2
CSC, CSR = 0, 1
FORMS = {"ridge_primal": RIDGE_PRIMAL, "svm_dual": SVM_DUAL, "ridge_dual": RIDGE_DUAL}
STATUS = {0: "SCD_OK", -1: "SCD_ERR_INVALID", -2: "SCD_ERR_UNSUPPORTED", -3: "SCD_ERR_OOM", -4: "SCD_ERR_HIP",
          -5: "SCD_ERR_NUMERIC"}


class ScdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class _Matrix(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("layout", ctypes.c_int32), ("reserved", ctypes.c_int32), ("ptr", ctypes.c_void_p),
                ("idx", ctypes.c_void_p), ("val", ctypes.c_void_p)]


KERNELS = ("group", "block", "ordered_lds", "mixed", "pipelined", "hot_lds", "queued", "team", "hot_staged",
           "split")


class _Info(ctypes.Structure):
    _fields_ = [("formulation", ctypes.c_int32), ("group_lanes", ctypes.c_int32), ("n_coords", ctypes.c_int64),
                ("shared_len", ctypes.c_int64), ("nnz", ctypes.c_int64), ("epoch", ctypes.c_int64),
                ("max_segment", ctypes.c_int64), ("window", ctypes.c_int64), ("lambda_", ctypes.c_double),
                ("coupling", ctypes.c_double), ("coherence", ctypes.c_double), ("auto_window", ctypes.c_int64),
                ("long_len", ctypes.c_int64), ("shared_fp64", ctypes.c_int32), ("max_hits", ctypes.c_uint32),
                ("kernel", ctypes.c_int32), ("hot_entries", ctypes.c_int32),
                ("adaptive_window", ctypes.c_int32), ("reserved", ctypes.c_int32)]


# Every symbol of include/scd.h with its ctypes signature.
_SIGS = {
    "scd_create": (ctypes.c_int, [ctypes.POINTER(_Matrix), ctypes.c_void_p, ctypes.c_double, ctypes.c_int32,
                                  ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]),
    "scd_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "scd_epochs": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p]),
    "scd_objective": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_double)]),
    "scd_duality_gap": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]),
    "scd_duality_gap_async": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32]),
    "scd_duality_gap_wait": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "scd_get_state": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.POINTER(ctypes.c_int64), ctypes.c_void_p]),
    "scd_set_state": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_void_p]),
    "scd_set_option": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_char_p, ctypes.c_int64]),
    "scd_get_option": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64)]),
    "scd_get_info": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(_Info)]),
    "scd_gather_dots": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "scd_norms": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "scd_permutation": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                       ctypes.c_void_p]),
    "scd_objective_static": (ctypes.c_int, [ctypes.POINTER(_Matrix), ctypes.c_void_p, ctypes.c_double, ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "scd_last_error": (ctypes.c_char_p, []),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_1702_07005_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()


def _check(code: int):
    if code != 0:
        raise ScdError(code, (lib.scd_last_error() or b"").decode())


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dev(t: torch.Tensor, dtype, n: int, what: str):
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dtype and t.is_contiguous() and t.numel() == n):
        raise ValueError(f"{what} must be a contiguous CUDA {dtype} tensor with {n} elements")
    return ctypes.c_void_p(t.data_ptr())


class Solver:
    """One handle of libscd.  ``ptr/idx/val/y`` are device tensors that the handle borrows:
    they are kept referenced here for the handle's lifetime."""

    def __init__(self, n_rows, n_cols, ptr, idx, val, y, lam, form="ridge_primal", stream=None):
        self.form = form
        self.n_rows, self.n_cols = int(n_rows), int(n_cols)
        code = FORMS[form]
        self.C = self.n_cols if code == RIDGE_PRIMAL else self.n_rows
        self.L = self.n_rows if code == RIDGE_PRIMAL else self.n_cols
        nnz = int(idx.numel())
        m = _Matrix(self.n_rows, self.n_cols, nnz, CSC if code == RIDGE_PRIMAL else CSR, 0,
                    _dev(ptr, torch.int64, self.C + 1, "ptr"), _dev(idx, torch.int32, nnz, "idx") if nnz else None,
                    _dev(val, torch.float32, nnz, "val") if nnz else None)
        self._keep = (ptr, idx, val, y)
        self.device = ptr.device
        h = ctypes.c_void_p()
        _check(lib.scd_create(ctypes.byref(m), _dev(y, torch.float32, self.n_rows, "y"), float(lam), code,
                              _stream(stream), ctypes.byref(h)))
        self._h = h
        self.lam = float(lam)

    # -- lifecycle ---------------------------------------------------------------------------
    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            _check(lib.scd_destroy(self._h))
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- solver ------------------------------------------------------------------------------
    def epochs(self, seed: int, n_epochs: int = 1, stream=None):
        _check(lib.scd_epochs(self._h, seed & 0xFFFFFFFFFFFFFFFF, n_epochs, _stream(stream)))

    def objective(self, stream=None):
        P, D = ctypes.c_double(), ctypes.c_double()
        _check(lib.scd_objective(self._h, _stream(stream), ctypes.byref(P), ctypes.byref(D)))
        return P.value, D.value

    def duality_gap(self, stream=None) -> float:
        g = ctypes.c_double()
        _check(lib.scd_duality_gap(self._h, _stream(stream), ctypes.byref(g)))
        return g.value

    def duality_gap_async(self, slot: int, stream=None):
        _check(lib.scd_duality_gap_async(self._h, _stream(stream), int(slot)))

    def duality_gap_wait(self, slot: int):
        """(gap, P, D) of the evaluation enqueued in `slot`."""
        g, P, D = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        _check(lib.scd_duality_gap_wait(self._h, int(slot), ctypes.byref(g), ctypes.byref(P), ctypes.byref(D)))
        return g.value, P.value, D.value

    def get_state(self, stream=None):
        model = torch.empty(self.C, dtype=torch.float32, device=self.device)
        shared = torch.empty(self.L, dtype=torch.float32, device=self.device)
        ep = ctypes.c_int64()
        _check(lib.scd_get_state(self._h, ctypes.c_void_p(model.data_ptr()), ctypes.c_void_p(shared.data_ptr()),
                                 ctypes.byref(ep), _stream(stream)))
        return model, shared, ep.value

    def set_state(self, model=None, shared=None, epoch=None, stream=None):
        mp = _dev(model, torch.float32, self.C, "model") if model is not None else None
        sp = _dev(shared, torch.float32, self.L, "shared") if shared is not None else None
        if epoch is None:
            epoch = self.info()["epoch"]
        _check(lib.scd_set_state(self._h, mp, sp, int(epoch), _stream(stream)))

    def set_option(self, key: str, value: int):
        _check(lib.scd_set_option(self._h, key.encode(), int(value)))

    def get_option(self, key: str) -> int:
        v = ctypes.c_int64()
        _check(lib.scd_get_option(self._h, key.encode(), ctypes.byref(v)))
        return v.value

    def info(self) -> dict:
        i = _Info()
        _check(lib.scd_get_info(self._h, ctypes.byref(i)))
        return dict(formulation=i.formulation, group_lanes=i.group_lanes, n_coords=i.n_coords,
                    shared_len=i.shared_len, nnz=i.nnz, epoch=i.epoch, max_segment=i.max_segment,
                    window=i.window, lam=i.lambda_, coupling=i.coupling, coherence=i.coherence,
                    auto_window=i.auto_window, long_len=i.long_len, shared_fp64=i.shared_fp64,
                    max_hits=i.max_hits, kernel=KERNELS[i.kernel], hot_entries=i.hot_entries,
                    adaptive_window=i.adaptive_window)

    def gather_dots(self, u: torch.Tensor, stream=None) -> torch.Tensor:
        out = torch.empty(self.C, dtype=torch.float32, device=self.device)
        _check(lib.scd_gather_dots(self._h, _dev(u, torch.float32, self.L, "u"), ctypes.c_void_p(out.data_ptr()),
                                   _stream(stream)))
        return out

    def norms(self, stream=None) -> torch.Tensor:
        out = torch.empty(self.C, dtype=torch.float32, device=self.device)
        _check(lib.scd_norms(self._h, ctypes.c_void_p(out.data_ptr()), _stream(stream)))
        return out


def permutation(seed: int, epoch: int, n: int, device="cuda", stream=None) -> torch.Tensor:
    out = torch.empty(n, dtype=torch.int32, device=device)
    _check(lib.scd_permutation(seed & 0xFFFFFFFFFFFFFFFF, int(epoch), int(n), ctypes.c_void_p(out.data_ptr()),
                               _stream(stream)))
    return out


def objective_static(n_rows, n_cols, ptr, idx, val, y, lam, form, model, shared, stream=None):
    """(P, D) of the state (model, shared) through scd_objective_static: no handle, no allocation."""
    code = FORMS[form]
    n_rows, n_cols = int(n_rows), int(n_cols)
    C = n_cols if code == RIDGE_PRIMAL else n_rows
    L = n_rows if code == RIDGE_PRIMAL else n_cols
    nnz = int(idx.numel())
    m = _Matrix(n_rows, n_cols, nnz, CSC if code == RIDGE_PRIMAL else CSR, 0, _dev(ptr, torch.int64, C + 1, "ptr"),
                _dev(idx, torch.int32, nnz, "idx") if nnz else None, _dev(val, torch.float32, nnz, "val") if nnz else None)
    P, D = ctypes.c_double(), ctypes.c_double()
    _check(lib.scd_objective_static(ctypes.byref(m), _dev(y, torch.float32, n_rows, "y"), float(lam), code,
                                    _dev(model, torch.float32, C, "model"), _dev(shared, torch.float32, L, "shared"),
                                    _stream(stream), ctypes.byref(P), ctypes.byref(D)))
    return P.value, D.value


def upload(prob, device="cuda"):
    """Device copies of a generated problem's arrays: (ptr, idx, val, y)."""
    return (torch.from_numpy(prob.ptr).to(device), torch.from_numpy(prob.idx).to(device),
            torch.from_numpy(prob.val).to(device), torch.from_numpy(prob.y).to(device))


def solver_for(prob, device="cuda", stream=None) -> Solver:
    """Upload a generated problem (paper_1702_07005_amd.synth.Problem) and create its solver."""
    ptr, idx, val, y = upload(prob, device)
    return Solver(prob.n_rows, prob.n_cols, ptr, idx, val, y, prob.lam, prob.form, stream=stream)
