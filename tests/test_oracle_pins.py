"""The CPU oracle against its pins (closed forms, brute force, lemmas)."""
import pytest

import oracle.shampoo_oracle as O
from tests import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(O)
