"""The CPU oracle against its pins (closed forms, brute force, invariants,
the paper's printed capsule sizes, published hash vectors)."""
import pytest

from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(orc, pin):
    pin(orc)
