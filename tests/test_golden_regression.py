"""Regression check of the oracle against its committed tiny-workload fixture."""
import json
import os

import numpy as np

from tests.golden.make_golden import compute

HERE = os.path.dirname(os.path.abspath(__file__))


def test_tiny_fixture_unchanged():
    with open(os.path.join(HERE, "golden", "tiny_l2k_oracle.json")) as f:
        want = json.load(f)
    got = compute()
    for key in ("count", "order", "hrm", "visit"):
        assert got[key] == want[key], key
    for key in ("score", "margin"):
        for a, b in zip(got[key], want[key]):
            assert np.allclose(a, b, rtol=1e-12, atol=1e-14), key
    assert abs(got["delta"] - want["delta"]) <= 1e-9 * want["delta"]
    assert np.allclose(got["o_row_sums"], want["o_row_sums"], rtol=1e-10, atol=1e-12)
