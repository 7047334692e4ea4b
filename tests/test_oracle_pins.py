"""The CPU oracle against its pins (closed forms, invariants, brute force, finite
differences, a library routine).  CPU only."""
import pytest

import oracle.ce as ce
from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(ce)
