"""The oracle against its pins (CPU only)."""
import pytest

import pins

PINS = [name for name in dir(pins) if name.startswith("pin_")]


@pytest.mark.parametrize("name", PINS)
def test_oracle_pin(name):
    getattr(pins, name)()
