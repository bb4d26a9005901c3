"""The CPU oracle checked against brute force, closed forms and invariants (CPU only)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=[p.__name__ for p in oracle_pins.PINS])
def test_oracle_pin(oracle_lib, pin):
    pin(oracle_lib)
