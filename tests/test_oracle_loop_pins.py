"""The closed-loop replay oracle against its pins (loop_pins.py)."""
import pytest

import oracle as O
import loop_pins


@pytest.mark.parametrize("pin", loop_pins.ALL, ids=lambda f: f.__name__)
def test_loop_pin(pin):
    pin(O.get())
