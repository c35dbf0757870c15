"""The CPU oracle against facts that do not come from the oracle (CPU only)."""
import pytest

import oracle
import oracle_pins as P


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("mode", ["math", "parity"])
@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(lib, pin, mode):
    pin(lib, mode)


@pytest.mark.parametrize("pin", P.MATH_ONLY_PINS, ids=lambda f: f.__name__)
def test_pin_math_only(lib, pin):
    pin(lib, "math")
