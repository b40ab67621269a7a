"""The CPU oracle against its pins (no GPU)."""
import pytest

from oracle import pss_oracle
import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(pss_oracle)
