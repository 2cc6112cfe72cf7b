"""The fp64 oracle against what the paper and the mathematics fix (CPU only)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    err = pin()
    assert err <= oracle_pins.TOL, f"{pin.__name__}: {err}"
