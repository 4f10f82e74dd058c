"""The calibration-sweep oracle against its pins (calib_pins.py)."""
import pytest

import oracle as O
import calib_pins


@pytest.mark.parametrize("pin", calib_pins.ALL, ids=lambda f: f.__name__)
def test_calib_pin(pin):
    pin(O.get())
