"""The CPU oracle checked against closed forms, invariants, hand cases and brute force."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()
