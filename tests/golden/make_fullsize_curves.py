"""Writes fullsize_gap_curves.json: the oracle's duality gap after each of the first epochs of the
three large workloads at full size (seed 0, the same inputs the GPU tests generate).

Sequential fp64 SCD (Alg. 1 order, the permutation of each epoch as the library defines it), so
an epoch takes seconds to a minute on one core; the whole file takes about half an hour.

    python tests/golden/make_fullsize_curves.py
"""
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

from oracle import oracle as orc  # noqa: E402
from paper_1702_07005_amd import synth  # noqa: E402

EPOCHS = {"text_svm": 8, "text_ridge_csc": 8, "click_svm": 12}


def main():
    out = {"note": "oracle duality gap after epochs 1..E from the zero state, seed 0, full-size workloads; "
                   "written by tests/golden/make_fullsize_curves.py"}
    for name, E in EPOCHS.items():
        t0 = time.time()
        p = synth.make(name)
        model = np.zeros(p.C)
        shared = np.zeros(p.L)
        P0 = orc.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, model, shared)[0]
        gaps = []
        for e in range(E):
            orc.epochs(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, 0, e, 1, model, shared)
            gaps.append(orc.objectives(p.form, p.n_rows, p.n_cols, p.ptr, p.idx, p.val, p.y, p.lam, model, shared)[2])
            print(f"{name} epoch {e + 1}: gap {gaps[-1]:.6e} ({time.time() - t0:.0f} s)", flush=True)
        out[name] = {"seed": 0, "P0": P0, "gap": gaps}
        del p, model, shared
    with open(os.path.join(HERE, "fullsize_gap_curves.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
