"""The CPU oracle against hand-derived fixtures, closed forms, invariants,
brute force and independent library routines (no GPU needed)."""
import pytest

import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


@pytest.mark.parametrize("n", [4000, 63, 1])
def test_dense_equivalence_ragged(n):
    """Ragged tails (n not a multiple of 64, a single token) still reduce to dense attention."""
    P.pin_dense_equivalence(n_override=n)


def test_invariants_ragged():
    P.pin_invariants_and_planted(n_override=4000)
