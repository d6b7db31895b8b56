"""The oracle's binary16 rounding and fp16-accumulation reading against
their pins (CPU only)."""
import pytest

import oracle_pins_acc16 as PA


@pytest.mark.parametrize("pin", PA.PINS, ids=[p.__name__ for p in PA.PINS])
def test_pin(pin):
    from oracle import oracle as O
    pin(O._load())
