"""The CPU oracle against its pins (brute force, closed forms, library routines, golden
fixtures).  See tests/oracle_pins.py for what each pin checks and why."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin, oracle_lib):
    pin(oracle_lib)
