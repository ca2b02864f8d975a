"""The CPU oracle against the paper's fixed facts, closed forms and brute force."""
import pytest

from oracle_pins import PINS


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin, oracle):
    pin(oracle)
