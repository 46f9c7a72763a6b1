"""The oracle against the paper's worked examples, closed forms, invariants and brute force."""
import pytest

import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin()


def test_bruteforce_decodability():
    pins.pin_bruteforce_decodability()


def test_mse_expectation():
    pins.pin_mse_expectation()
