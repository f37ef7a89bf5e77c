"""Sanity of the stored full-size oracle curves (tests/golden/fullsize_gap_curves.json), which the
GPU full-size tests gate against.  CPU only."""
import json
import math
import os

import pytest

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fullsize_gap_curves.json")


@pytest.mark.skipif(not os.path.exists(PATH), reason="stored curves not written yet")
def test_stored_curves_describe_the_zero_state_and_converge():
    with open(PATH) as f:
        ref = json.load(f)
    # At the zero state every hinge term is 1 (SVM: P = 1) and the ridge residual is y, with +-1
    # labels (ridge primal: P = |y|^2 / (2N) = 1/2): closed forms the stored P(0) must match.
    assert ref["text_svm"]["P0"] == pytest.approx(1.0, rel=1e-12)
    assert ref["click_svm"]["P0"] == pytest.approx(1.0, rel=1e-12)
    assert ref["text_ridge_csc"]["P0"] == pytest.approx(0.5, rel=1e-12)
    for name in ("text_svm", "text_ridge_csc", "click_svm"):
        g = ref[name]["gap"]
        assert ref[name]["seed"] == 0 and len(g) >= 8
        assert all(math.isfinite(x) and x > 0.0 for x in g)
        assert g[-1] < 0.1 * g[0]  # sequential SCD makes progress over the stored epochs
