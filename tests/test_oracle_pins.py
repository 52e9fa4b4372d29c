"""The float64 oracle against its pins (closed forms, invariants, library special cases)."""
import pytest

import os
import sys

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle.hspec_oracle as O  # noqa: E402
from oracle_pins import PINS  # noqa: E402


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(O)
