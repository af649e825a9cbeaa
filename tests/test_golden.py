"""The oracle still produces its committed outputs for the tiny workload."""
import json
import os

import numpy as np

from tests.golden.make_golden import tiny_step_expected

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_tiny_step_oracle_matches_golden():
    with open(os.path.join(HERE, "tiny_step_oracle.json")) as f:
        want = json.load(f)
    got = tiny_step_expected()
    assert got["ids"] == want["ids"]
    np.testing.assert_allclose(got["lps"], want["lps"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["logits_first8"], want["logits_first8"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["logits_sum"], want["logits_sum"], rtol=1e-12, atol=1e-9)
