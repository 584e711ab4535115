"""The CPU oracle against its pins (exact arithmetic, closed forms, brute
force, library routines, invariants of the method)."""
import pytest

import oracle.sphinx_oracle as O
from pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(O)
