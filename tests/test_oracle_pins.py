"""The CPU oracle against its pins (closed forms, worked examples, library
routines, brute force and the paper's invariants)."""
import pytest

from oracle import conduit_oracle
from tests import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(conduit_oracle)
