"""The CPU oracle against its pins (no GPU)."""
import os, sys
sys.path.insert(0, os.path.dirname(__file__))
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle)
