"""Build libscd.so (HIP, gfx950 only) in-tree.

    python -m paper_1702_07005_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libscd.so")
SOURCES = [os.path.join(CSRC, f)
           for f in ("scd_epoch.hip", "scd_hot.hip", "scd_team.hip", "scd_split.hip", "scd_setup.hip", "scd_static.hip",
                     "scd_api.cpp")]
# Measurement aid used by bench.py (device-wide atomic and copy rates); not linked into libscd.
PROBE_LIB = os.path.join(HERE, "libscdprobe.so")
PROBE_SOURCES = [os.path.join(CSRC, "ceiling.hip")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-munsafe-fp-atomics",
    # No packed fp32 (v_pk_*_f32) in device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wextra",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    return subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)


def _finish(proc, verbose):
    _, stderr = proc.communicate()
    noise = "is not a recognized feature for this target"
    err = "\n".join(line for line in stderr.splitlines() if noise not in line)
    if proc.returncode != 0:
        raise RuntimeError(f"hipcc failed ({proc.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def _compile(sources, out, verbose):
    """Compile each source to an object in parallel (one hipcc per file), then link."""
    tmp = out + ".tmp"
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    base = [hipcc(), *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC]
    base.remove("-shared")
    objs, procs = [], []
    for src in sources:
        obj = os.path.join(objdir, os.path.splitext(os.path.basename(src))[0] + ".o")
        objs.append(obj)
        procs.append(_run([*base, "-c", "-x", "hip", src, "-o", obj], verbose))
    for proc in procs:
        _finish(proc, verbose)
    _finish(_run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose), verbose)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    _compile(PROBE_SOURCES, PROBE_LIB, verbose)
    return _compile(SOURCES, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
