"""Run the PD decision-engine oracle pins (CPU only)."""
import pytest

from pd_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pd_pin(pin):
    pin()
