"""The oracle pinned to published values, closed forms, invariants and an
independent formulation (CPU only)."""
import pytest

import oracle
import oracle_pins as P


@pytest.fixture(scope="module")
def orc():
    oracle.build(force=False)
    return oracle.load()


@pytest.mark.parametrize("pin", P.QUICK_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_brute_force_tiny_domain(orc):
    P.pin_brute_force_tiny(orc)


def test_brute_force_cohorts(orc):
    P.pin_brute_force_cohorts(orc)


def test_decision_rate_over_all_outcomes(orc):
    P.pin_decision_rate_exhaustive(orc)
