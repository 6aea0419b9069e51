"""The fp64 oracle against hand values, closed forms, independent formulations and
invariants (see pins.py for the list and the routes used)."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=[p.__name__ for p in pins.ALL_PINS])
def test_pin(oracle_lib, pin):
    pin()
