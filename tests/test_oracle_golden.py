"""Regression of the oracle against its stored trajectory (written by
tests/golden/make_golden.py from the oracle alone)."""
import json
import os

import pytest

from tests.golden.make_golden import trajectory

HERE = os.path.dirname(os.path.abspath(__file__))


def test_tiny_trajectory_regression():
    with open(os.path.join(HERE, "golden", "tiny_3steps.json")) as f:
        gold = json.load(f)["steps"]
    got = trajectory()
    assert len(got) == len(gold) == 3
    for g, r in zip(got, gold):
        for k in r:
            assert g[k] == pytest.approx(r[k], rel=1e-12, abs=1e-15)
