"""The stored full-size expected values (host only): each golden file holds the
oracle's loss and lse of every token, the SHA-256 of the generated inputs and the
largest |logit| the oracle met.  The stress workload's recipe asks for a logit
scale with max |logit| near 40; its stored value must lie in [36, 44], and the
others (unscaled H) stay near the 6-7 of N(0, 1) logits."""
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
FILES = sorted(f for f in os.listdir(GOLDEN) if f.startswith("fullsize_") and f.endswith(".npz"))


@pytest.mark.parametrize("name", FILES)
def test_golden_contents(name):
    g = np.load(os.path.join(GOLDEN, name), allow_pickle=False)
    T = int(g["T"])
    assert g["loss"].shape == (T,) and g["lse"].shape == (T,)
    assert np.all(np.isfinite(g["lse"])) and np.all(g["loss"] >= 0.0)
    m = float(g["max_abs_logit"])
    # lse >= the largest logit of its row >= ... and every lse is within log V of its max
    assert np.all(g["lse"] <= m + np.log(int(g["V"])) + 1e-9)
    if name.startswith("fullsize_stress"):
        assert 36.0 <= m <= 44.0, m
    else:
        assert 4.0 <= m <= 9.0, m
