"""Plant mistakes in the oracle and check that the pins catch each one.

Each C mutant is a build of ``oracle/daf_oracle.c`` with one mistake compiled
in (a dropped scale, an interleaved GQA map, a mask by storage order instead
of position, a non-causal question block, K read as V, lse without the max, a
term dropped from the softmax sum, a lost gather row, reversed scatter sources,
the question's own key dropped, a feature dropped from the dot product, a
position mask one key too wide). The
Python plants skip the hybrid write-back, leave the question K/V out of the
cache, fuse question rows one row early, score selection from one layer only,
or break selection ties toward the higher index.
"""
import os

import pytest

import oracle as orc_mod
from oracle import build as orc_build
from oracle_pins import ALL_PINS

C_MUTANTS = list(range(1, 13))
PY_PLANTS = ["no_hybrid", "no_question_kv", "fuse_shift", "select_one_layer", "select_tie_high"]


def _failures(orc):
    failed = []
    for pin in ALL_PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError, FloatingPointError):
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("mutant", C_MUTANTS)
def test_c_mutant_caught(mutant, tmp_path):
    lib = orc_build.build(mutant=mutant, out=str(tmp_path / f"liboracle_m{mutant}.so"))
    orc = orc_mod.Oracle(lib)
    assert orc.mutant == mutant
    failed = _failures(orc)
    assert failed, f"mutant {mutant} passed every pin"


@pytest.mark.parametrize("plant", PY_PLANTS)
def test_python_plant_caught(plant):
    orc = orc_mod.Oracle(plant=plant)
    failed = _failures(orc)
    assert failed, f"plant {plant} passed every pin"


def test_clean_build_passes_all(oracle):
    assert oracle.mutant == 0
    assert _failures(oracle) == []
