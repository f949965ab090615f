"""The fp64 oracle against closed forms, invariants, brute force, finite
differences and torch's autograd (CPU only)."""
import pytest

from tests._pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(pin, oracle_mod):
    pin(oracle_mod)
