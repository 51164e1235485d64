"""The oracle against its pins (CPU only).  See tests/oracle_pins.py for what each pin is."""
import pytest

import oracle
import oracle_pins


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_bf16_rounding_exhaustive(orc):
    """Narrowing agrees with torch's fp32->bf16 conversion over all 2^32 fp32 patterns."""
    oracle_pins.bf16_round_exhaustive(orc)
