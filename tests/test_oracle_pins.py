"""The oracle against its pins (hand example, closed forms, brute force,
textbook reductions, invariants). CPU only."""
import pytest

import oracle.unif_moe_oracle as O
from tests import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(O)


def test_bruteforce_many_layers():
    P.pin_bruteforce(O, n_layers=400, n_tok=5, seed=101)
