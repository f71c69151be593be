"""Each deliberately broken build of the oracle must fail at least one pin,
which shows that the pins would catch that kind of mistake."""
import os

import pytest

import oracle
from oracle import build as obuild
from tests import oracle_pins


@pytest.mark.parametrize("mutant", sorted(oracle_pins.MUTANTS), ids=lambda m: oracle_pins.MUTANTS[m])
def test_mutant_is_caught(tmp_path, mutant):
    path = obuild.build_variant({"WSO_MUTANT": mutant}, os.path.join(tmp_path, f"m{mutant}.so"))
    lib = oracle.load(path)
    assert lib.wso_mutant() == mutant
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError, FloatingPointError) as exc:
            failed.append(pin.__name__)
    assert failed, f"no pin caught mutant {mutant} ({oracle_pins.MUTANTS[mutant]})"
