"""Regression lock: the oracle still produces the stored tiny-layer outputs."""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_golden  # noqa: E402


def test_tiny_layer_matches_golden():
    with open(os.path.join(HERE, "golden", "tiny_layer_oracle.json")) as f:
        ref = json.load(f)
    r, out = make_golden.compute()
    assert r["idx"].tolist() == ref["idx"]
    for key in ("o_imp", "lse_imp", "o_q", "lse_q"):
        np.testing.assert_allclose(out[key].ravel(), np.array(ref[key]), rtol=1e-12, atol=1e-13)
