"""The CPU oracle against its pins (see oracle_pins.py for what each pin uses)."""
import pytest

import oracle_pins as op


@pytest.mark.parametrize("pin", op.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(0)
