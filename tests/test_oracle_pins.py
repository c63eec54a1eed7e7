"""The CPU oracle against closed forms, invariants, a hand-worked example, torch SDPA in float64
and brute-force scalar loops (no GPU)."""
import pytest

from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(pin):
    pin()
