"""The golden fixtures under tests/golden/ are what the CPU oracle produces today:
regenerating them must give the stored text byte for byte. A change to the
oracle's arithmetic therefore shows up here, and its commit has to name the
passage of the paper (or the reading of it) that justifies it."""

import os
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))

import make_golden  # noqa: E402


@pytest.mark.parametrize("name", sorted(make_golden.FIXTURES))
def test_fixture_is_what_the_oracle_writes(name):
    stored = open(os.path.join(HERE, "golden", name)).read()
    assert make_golden.FIXTURES[name]() == stored, f"{name} differs from the oracle's output"
