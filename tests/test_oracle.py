"""Pins of the CPU oracle (no GPU): see tests/pins.py for what each checks."""
import pytest

import oracle
import pins


@pytest.fixture(scope="module")
def orc():
    oracle.build()
    return oracle._get()


@pytest.mark.parametrize("check", pins.ALL, ids=lambda f: f.__name__)
def test_pin(orc, check):
    check(orc)
