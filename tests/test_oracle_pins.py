"""The fp64 oracle against what block-causal attention's definition fixes."""
import pytest

import oracle
from tests import oracle_pins


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(lib, pin):
    assert lib.wso_mutant() == 0
    pin(lib)
