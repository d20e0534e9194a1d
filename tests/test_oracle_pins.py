"""The oracle against its pins (decoding tables, closed forms, invariants, exact brute force)."""
import pytest

import oracle
import pins


@pytest.fixture(scope="module")
def ora():
    return oracle.get()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=[p.__name__ for p in pins.ALL_PINS])
def test_pin(ora, pin):
    pin(ora)
