"""The CPU oracle against what the paper and mathematics fix (no GPU)."""

import pytest

import oracle
import pins


@pytest.mark.parametrize("check", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(oracle.zeta_oracle)
