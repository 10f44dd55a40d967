"""The CPU oracle against its pins (worked Fig. 2 instances, brute force, special cases, FD, adjoint)."""
import pytest

import oracle
import oracle_pins as P


@pytest.fixture(scope="module")
def orc():
    oracle.build()
    return oracle.get()


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=[p.__name__ for p in P.ALL_PINS])
def test_pin(orc, pin):
    pin(orc)
