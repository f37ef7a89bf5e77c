"""The oracle's pins catch plausible mistakes: each case plants one mistake in a copy of the
oracle's C source (a dropped term, a wrong sign or index, a missing projection, a broken
permutation round), builds it, and requires the pin suite to fail against it."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "scd_oracle.c")
PINS = ["tests/test_oracle_perm.py", "tests/test_oracle_ridge.py", "tests/test_oracle_svm.py", "tests/test_oracle_f32.py",
        "tests/test_oracle_shared_objectives.py"]

MUTANTS = {
    "primal_drops_regulariser": ("double d = (g - lN * beta[m]) / (norms[m] + lN);",
                                 "double d = (g) / (norms[m] + lN);"),
    "primal_denominator": ("double d = (g - lN * beta[m]) / (norms[m] + lN);",
                           "double d = (g - lN * beta[m]) / (norms[m]);"),
    "primal_scatter_sign": ("w[row_idx[k]] += (double)val[k] * d;", "w[row_idx[k]] -= (double)val[k] * d;"),
    "primal_gather_sign": ("g += ((double)y[row_idx[k]] - w[row_idx[k]]) * (double)val[k];",
                           "g += ((double)y[row_idx[k]] + w[row_idx[k]]) * (double)val[k];"),
    "dual_drops_lambda_y": ("double d = (lambda * (double)y[i] - g - lN * alpha[i]) / (lN + norms[i]);",
                            "double d = ((double)y[i] - g - lN * alpha[i]) / (lN + norms[i]);"),
    "svm_no_upper_clip": ("            if (a > 1.0)\n                a = 1.0;\n", ""),
    "svm_scatter_drops_label": ("double c = d * (double)y[i] / lN;", "double c = d / lN;"),
    "svm_step_sign": ("a = alpha[i] + lN * (1.0 - (double)y[i] * g) / norms[i];",
                      "a = alpha[i] + lN * (1.0 + (double)y[i] * g) / norms[i];"),
    "ridge_dual_obj_drops_term": ("double D = -0.5 * (double)N * a2 - ata2 / (2.0 * lambda) + ay;",
                                  "double D = -0.5 * (double)N * a2 + ay;"),
    "svm_obj_hinge_without_max": ("hinge += l > 0.0 ? l : 0.0;", "hinge += l;"),
    "norms_abs_not_square": ("s += (double)val[k] * (double)val[k];", "s += fabs((double)val[k]);"),
    "feistel_round_dropped": ("uint64_t newR = L ^ f;", "uint64_t newR = L;"),
    "keys_ignore_epoch": ("uint64_t base = oracle_splitmix64_nth(seed, epoch + 1);",
                          "uint64_t base = oracle_splitmix64_nth(seed, 1);"),
    "fmix_constant": ("h *= 0xC2B2AE35U;", "h *= 0xC2B2AE37U;"),
    "f32_primal_drops_regulariser": ("float d = (g - lN * model[m]) / (norms[m] + lN);",
                                     "float d = (g) / (norms[m] + lN);"),
    "f32_dual_drops_lambda_y": ("float d = (lam * y[m] - g - lN * model[m]) / (lN + norms[m]);",
                                "float d = (y[m] - g - lN * model[m]) / (lN + norms[m]);"),
    "f32_svm_scatter_drops_label": ("coef = (a - model[m]) * y[m] / lN;", "coef = (a - model[m]) / lN;"),
    # objectives from a maintained shared vector: the given vector is dropped (left at zero)
    "ridge_primal_obj_ignores_shared": ("memcpy(w, w_in, sizeof(double) * (size_t)N);", "(void)w_in;"),
    "ridge_dual_obj_ignores_shared": ("memcpy(wbar, wbar_in, sizeof(double) * (size_t)M);", "(void)wbar_in;"),
    "svm_obj_ignores_shared": ("memcpy(w, w_in, sizeof(double) * (size_t)M);", "(void)w_in;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site not unique/present: {old!r}"
    mutant = tmp_path / "mutant.c"
    mutant.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o", str(so), str(mutant), "-lm"])
    env = dict(os.environ, SCD_ORACLE_LIB=str(so))
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert res.returncode != 0, f"pins did not catch mutant {name}:\n{res.stdout[-2000:]}"
