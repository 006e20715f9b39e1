"""The CPU oracle against what the paper and the mathematics fix (no GPU)."""
import pytest

from oracle_pin_checks import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(orc, pin):
    pin(orc)
