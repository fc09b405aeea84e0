"""The oracle against its pins (CPU only).  See oracle_pins.py,
sdstep_pins.py and costmodel_pins.py."""
import pytest

from costmodel_pins import ALL_COSTMODEL_PINS
from oracle_pins import ALL_PINS
from sdstep_pins import ALL_SDSTEP_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(pin):
    pin()


@pytest.mark.parametrize("pin", ALL_SDSTEP_PINS, ids=[p.__name__ for p in ALL_SDSTEP_PINS])
def test_sdstep_pin(pin):
    pin()


@pytest.mark.parametrize("pin", ALL_COSTMODEL_PINS, ids=[p.__name__ for p in ALL_COSTMODEL_PINS])
def test_costmodel_pin(pin):
    pin()
