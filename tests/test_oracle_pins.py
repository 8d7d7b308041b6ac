"""The fp64 oracle against what the paper and the mathematics fix (CPU only)."""
import pytest

import oracle
from oracle_pins import ALL_PINS, TOL


@pytest.mark.parametrize("name", sorted(ALL_PINS))
def test_pin(name):
    err = ALL_PINS[name](oracle.forward)
    assert err < TOL, "%s: deviation %.3e" % (name, err)
