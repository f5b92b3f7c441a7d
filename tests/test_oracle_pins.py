"""The fp64 oracle against facts outside itself (see oracle_pins.py)."""
import pytest

from oracle import oracle as O
from tests import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(O.LIB if O.load() else O.LIB)
