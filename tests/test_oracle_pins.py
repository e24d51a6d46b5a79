"""The CPU oracle against what the paper and plain mathematics fix (no GPU)."""
import pytest

import pins
from oracle import default


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(default())
