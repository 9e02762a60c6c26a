"""The CPU oracle against brute force, invariants, library routines and hand-worked examples."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.fixture(scope="module")
def impl():
    return oracle.default()


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(impl, pin):
    pin(impl)
