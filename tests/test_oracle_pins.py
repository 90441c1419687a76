"""The CPU oracle against what the paper and the mathematics fix (no GPU)."""
import pytest

import oracle
import oracle_pins


@pytest.fixture(scope="module")
def o():
    oracle.build()
    return oracle.Oracle()


@pytest.mark.parametrize("check", oracle_pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(o, check):
    check(o)
