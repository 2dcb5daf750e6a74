"""The float64 oracle against what the paper and the mathematics fix (CPU)."""
import pytest

import oracle
from pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__[4:])
def test_pin(pin):
    pin(oracle.default())
