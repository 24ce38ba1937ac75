"""The CPU oracle against its pins (exact brute force, closed forms,
quadrature, Monte Carlo, the paper's Eq. (8), invariants)."""
import pytest

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle.lib())
