"""The CPU oracle against facts fixed outside it (see tests/pins.py)."""
import pytest

import oracle as O
import pins


@pytest.fixture(scope="module")
def orc():
    return O.get()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)
