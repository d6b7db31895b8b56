"""The fused-idiom oracle against its pins (CPU only)."""
import pytest

import oracle_pins_fused as PF


@pytest.mark.parametrize("pin", PF.PINS, ids=[p.__name__ for p in PF.PINS])
def test_pin(pin):
    from oracle import oracle as O
    pin(O._load())
