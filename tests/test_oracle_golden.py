"""The oracle reproduces its committed Tiny-workload fixtures (written by
tests/golden/make_golden.py, which calls only the oracle and the input generators)."""
import json
import os

import numpy as np
import pytest

from golden.make_golden import CASES, run_case

HERE = os.path.dirname(os.path.abspath(__file__))
with open(os.path.join(HERE, "golden", "oracle_tiny.json")) as f:
    GOLDEN = json.load(f)


@pytest.mark.parametrize("name", sorted(CASES))
def test_golden(name):
    want = GOLDEN[name]["result"]
    got = run_case(CASES[name])
    assert got["tokens"] == want["tokens"]
    assert got["status"] == want["status"]
    assert got["trace"] == want["trace"]
    np.testing.assert_allclose(got["scores"], want["scores"], rtol=0, atol=1e-12)
