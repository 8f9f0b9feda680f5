"""The fp64 oracle against brute force, library reductions, closed forms and
the layer's invariants (CPU only)."""

import pytest

import pins
from oracle import oracle


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)
