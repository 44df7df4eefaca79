"""The oracle against brute force, closed forms, invariants and finite
differences (CPU only)."""
import pytest

from tests import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin, oracle_instance):
    pin(oracle_instance)
