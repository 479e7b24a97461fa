"""The float64 oracle against brute force, torch's CPU attention, closed
forms, golden cases and invariants of the attention definition."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)
