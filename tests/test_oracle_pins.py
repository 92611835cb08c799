"""The CPU oracle against what the paper and mathematics fix (no GPU)."""
import pytest

import oracle
from tests import pins


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check):
    check(oracle.rmm_oracle)
