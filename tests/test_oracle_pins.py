"""The CPU oracle against its pins (library routines, closed forms,
invariants, hand-built boundary cases). See tests/oracle_pins.py."""
import pytest

from tests import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda f: f.__name__)
def test_pin(oracle_lib, pin):
    pin(oracle_lib)
