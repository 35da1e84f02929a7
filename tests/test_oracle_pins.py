"""The CPU oracle against its pins (hand-worked fixtures, closed forms,
invariants, library-routine special cases and brute force)."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin, oracle_impl):
    pin(oracle_impl)
