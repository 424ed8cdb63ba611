"""The fp64 oracle against closed forms, invariants, brute force, independent
library routines and finite differences (CPU only)."""
import pytest

from oracle import block as ob

from oracle_pins import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(ob)
