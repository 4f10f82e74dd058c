"""The stage-aware service-share oracle against its pins (stage_pins.py)."""
import pytest

import oracle as O
import stage_pins


@pytest.fixture(scope="module")
def o():
    return O.get()


@pytest.mark.parametrize("pin", stage_pins.ALL, ids=lambda p: p.__name__)
def test_pin(o, pin):
    pin(o)
