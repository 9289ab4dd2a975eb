"""The fp64 oracle against its pins (see oracle_pins.py for what each pin fixes)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=[p.__name__ for p in oracle_pins.PINS])
def test_oracle_pin(oracle_lib, pin):
    pin(oracle_lib.lib())
