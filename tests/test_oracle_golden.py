"""The oracle still reproduces its frozen outputs (tests/golden, written by make_golden.py)."""
import json
import os

import numpy as np
import pytest

from tests.golden import make_golden

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.mark.parametrize("name", sorted(make_golden.CASES))
def test_oracle_matches_golden(name):
    with open(os.path.join(HERE, name + ".json")) as f:
        ref = json.load(f)["result"]
    got = make_golden.case(name)
    assert sorted(got) == sorted(ref)
    for key in ref:
        np.testing.assert_array_equal(np.asarray(got[key]), np.asarray(ref[key]), err_msg=key)
