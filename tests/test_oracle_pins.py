"""The oracle against its pins (CPU only)."""
import pytest

import oracle_pins as pins


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check()


def test_tolerance_rule_pin():
    """The value acceptance rule used by every GPU parity test."""
    pins.check_within_tol()
