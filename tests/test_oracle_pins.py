"""The CPU oracle against facts fixed by the paper and by mathematics."""
import pytest

from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(oracle, pin):
    pin(oracle.Oracle())
