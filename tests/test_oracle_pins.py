"""The oracle against what the paper and the mathematics fix (no GPU)."""
import pytest

from oracle_pins import PINS, _bind


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(oracle_lib, pin):
    pin(_bind(oracle_lib))
