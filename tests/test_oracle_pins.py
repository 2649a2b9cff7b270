"""The oracle against its pins (CPU only; the pins are described in oracle_pins.py)."""
import pytest

import oracle as nfo
from tests import oracle_pins


@pytest.fixture(scope="module")
def lib():
    return nfo.load()


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(lib, pin):
    pin(lib)
