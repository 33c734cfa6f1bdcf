"""The fp64 oracle against closed forms, exact-rational brute force, special
cases and the paper's alternative computation (CPU only)."""
import pytest

from oracle import oracle as orc
from tests import oracle_pins as pins


@pytest.fixture(scope="module")
def lib():
    return orc.load()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(lib, pin):
    pin(lib)
