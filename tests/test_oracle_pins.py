"""The oracle against its pins (no GPU)."""
import pytest

from tests import oracle_pins as pins


@pytest.mark.parametrize("name", sorted(pins.ALL_PINS, key=lambda s: int(s[1:])))
def test_pin(name):
    pins.ALL_PINS[name]()
