"""The CPU oracle pinned against closed forms, invariants, brute force and the
hand-derived Alg. 4 worked example (no GPU needed)."""
import pytest

import oracle_pins as P


@pytest.mark.parametrize("check", P.ALL_CHECKS, ids=lambda f: f.__name__[6:])
def test_pin(check):
    check()
