"""The CPU oracle checked against brute force, library routines, closed forms, invariants and the paper's
greedy rule (all pins live in tests/pins.py)."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(orc, pin):
    pin(orc)
