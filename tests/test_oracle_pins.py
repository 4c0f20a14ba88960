"""The CPU oracle against its pins (closed forms, hand-worked cases,
invariants, pure-Python brute force).  CPU only."""
import pytest

import oracle
from oracle_pins import PINS


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(oracle)
