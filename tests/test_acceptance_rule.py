"""The oracle's acceptance rule (oracle.tolerance / oracle.check) against its
hand-worked pins."""
import pytest

import oracle
from acceptance_pins import ALL_ACCEPTANCE_PINS


@pytest.mark.parametrize("pin", ALL_ACCEPTANCE_PINS, ids=[p.__name__ for p in ALL_ACCEPTANCE_PINS])
def test_acceptance_pin(pin):
    pin(oracle)
