"""The fp64 oracle against closed forms, textbook values, invariants, Monte Carlo
and brute force (each pin is documented in pins.py)."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)
