"""The actuation-model replay of the oracle against its pins (act_pins.py)."""
import pytest

import oracle as O
import act_pins


@pytest.mark.parametrize("pin", act_pins.ALL, ids=lambda f: f.__name__)
def test_act_pin(pin):
    pin(O.get())
