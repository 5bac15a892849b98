"""The CPU oracle against brute force, closed forms and invariants (no GPU)."""
import pytest

import oracle
import pins


@pytest.fixture(scope="module")
def L():
    return oracle.lib()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin, L):
    pin(L)
