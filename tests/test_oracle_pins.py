"""The shipped fp64 oracle against its pins (brute force, closed forms,
invariants, torch's fp64 SDPA).  CPU only."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)
