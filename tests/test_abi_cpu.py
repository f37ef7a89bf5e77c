"""The C ABI library on a machine without a GPU: it loads, exports every function that
include/scd.h declares, and its host-side argument checks answer without touching a GPU."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scd.h")
LIB = os.path.join(ROOT, "paper_1702_07005_amd", "libscd.so")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(scd_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_1702_07005_amd import build
        build.build()
    return ctypes.CDLL(LIB)


def test_header_declares_the_boundary():
    names = declared()
    for must in ("scd_create", "scd_epochs", "scd_objective", "scd_duality_gap", "scd_destroy",
                 "scd_get_state", "scd_set_state", "scd_gather_dots", "scd_permutation", "scd_last_error"):
        assert must in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (scd_\w+)", out))
    for name in declared():
        assert name in exported, name
        getattr(lib, name)


def test_binding_covers_the_header():
    src = open(os.path.join(ROOT, "paper_1702_07005_amd", "scd.py")).read()
    for name in declared():
        assert f'"{name}"' in src, name


def test_library_is_built_for_gfx950_only(tmp_path):
    fatbin = tmp_path / "fatbin.bin"
    dump = subprocess.run(["objcopy", f"--dump-section=.hip_fatbin={fatbin}", LIB, str(tmp_path / "copy.so")],
                          capture_output=True, text=True)
    out = subprocess.run(["/opt/rocm/llvm/bin/clang-offload-bundler", "--list", "--type=o", f"--input={fatbin}"],
                         capture_output=True, text=True)
    if dump.returncode != 0 or out.returncode != 0:
        pytest.skip("could not list the embedded device code objects")
    targets = [t for t in out.stdout.split() if "amdgcn" in t]
    assert targets and all(t.endswith("gfx950") for t in targets), targets


class _Matrix(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("layout", ctypes.c_int32), ("reserved", ctypes.c_int32), ("ptr", ctypes.c_void_p),
                ("idx", ctypes.c_void_p), ("val", ctypes.c_void_p)]


def _create(lib, m, y, lam, form):
    lib.scd_create.argtypes = [ctypes.POINTER(_Matrix), ctypes.c_void_p, ctypes.c_double, ctypes.c_int32,
                               ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    lib.scd_last_error.restype = ctypes.c_char_p
    h = ctypes.c_void_p(1234)
    rc = lib.scd_create(ctypes.byref(m) if m is not None else None, y, lam, form, None, ctypes.byref(h))
    return rc, h.value, lib.scd_last_error().decode()


FAKE = 0x1000  # never dereferenced: every case below fails before any device access


@pytest.mark.parametrize("case,want", [
    ("null_matrix", "matrix is null"), ("bad_form", "unknown formulation"), ("layout_primal", "needs layout CSC"),
    ("layout_dual", "needs layout CSR"), ("neg_nnz", "bad sizes"), ("zero_rows", "bad sizes"),
    ("huge", "below 2^31"), ("null_ptr", "null device pointer"), ("lambda", "lambda"), ("nan_lambda", "lambda")])
def test_create_argument_checks(lib, case, want):
    m = _Matrix(10, 5, 20, 0, 0, FAKE, FAKE, FAKE)
    y, lam, form = FAKE, 0.1, 0
    if case == "null_matrix":
        m = None
    elif case == "bad_form":
        form = 7
    elif case == "layout_primal":
        m.layout = 1
    elif case == "layout_dual":
        form = 1
    elif case == "neg_nnz":
        m.nnz = -1
    elif case == "zero_rows":
        m.n_rows = 0
    elif case == "huge":
        m.n_rows = 1 << 31
    elif case == "null_ptr":
        m.ptr = None
    elif case == "lambda":
        lam = -1.0
    elif case == "nan_lambda":
        lam = float("nan")
    rc, h, msg = _create(lib, m, y, lam, form)
    assert rc == -1 and h is None and want in msg


def test_null_handle_calls(lib):
    lib.scd_last_error.restype = ctypes.c_char_p
    assert lib.scd_destroy(None) == 0
    lib.scd_epochs.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p]
    assert lib.scd_epochs(None, 0, 1, None) == -1
    assert b"null handle" in lib.scd_last_error()
    lib.scd_set_option.argtypes = [ctypes.c_void_p, ctypes.c_char_p, ctypes.c_int64]
    assert lib.scd_set_option(None, b"window", 1) == -1
    lib.scd_permutation.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_void_p]
    assert lib.scd_permutation(0, 0, 0, FAKE, None) == -1
    assert lib.scd_permutation(0, -1, 10, FAKE, None) == -1
    assert lib.scd_permutation(0, 0, 10, None, None) == -1


def test_static_objective_source_allocates_nothing():
    # The allocation-free entry point keeps its scratch in a file-scope device array, reached through
    # the address hipGetSymbolAddress returns per device; its source calls no allocating routine.
    src = open(os.path.join(ROOT, "paper_1702_07005_amd", "csrc", "scd_static.hip")).read()
    code = "\n".join(line.split("//")[0] for line in src.splitlines())
    for banned in ("hipMalloc", "hipFree", "hipHostMalloc", "hipHostFree", "hipMallocAsync", "malloc(", "new "):
        assert banned not in code, banned
    assert "__device__ __align__(256)" in code and "hipGetSymbolAddress" in code
