"""The fp64 oracle against what the paper and the mathematics fix (CPU only)."""

import pytest

import oracle.tgvkv_oracle as O
from tests import oracle_pins as pins


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(O)
