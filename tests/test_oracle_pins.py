"""The CPU oracle against what the paper and mathematics fix (runs without a GPU)."""

import pytest

import oracle.asv_oracle as orc
from oracle_pins import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(orc)
