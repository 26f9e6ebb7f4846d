"""The oracle against what the paper and the mathematics fix (CPU only).

See tests/oracle_pins.py for what each pin checks and why it is independent
of the oracle.  The mutation test rebuilds the oracle with one planted
mistake at a time and checks that the pins reject every such build.
"""
import os
import tempfile

import pytest

import oracle
from oracle import build as obuild

from . import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    msg = pin(oracle.load())
    assert msg is None, msg


# Planted mistakes, one per build (ORACLE_MUTANT in glide_oracle.c):
#  1 softmax window one token too long      2 linear part dropped
#  3 separately normalised "+" merge        4 feature map with Wf transposed
#  5 decode folds the new token, not the evicted one
#  6 merge without a common stabiliser      7 softmax scale tau missing
#  8 hybrid form 2 misses the current token in its linear set
#  9 hybrid form 2's decode folds the evicted token, not the new one
# 10 hybrid forms divide the linear term by both denominators
# 11 the ELU+1 feature map without the + 1
# 12 the softmax feature map without its normalisation
# 13 per-head feature maps: every head takes head 0's Wf
# 14 the gated state decays a token by its own gate as well
MUTANTS = [1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14]


@pytest.mark.parametrize("mutant", MUTANTS)
def test_pins_reject_planted_mistake(mutant):
    with tempfile.TemporaryDirectory() as td:
        path = obuild.build(os.path.join(td, f"liboracle_m{mutant}.so"), mutant=mutant)
        lib = oracle.load(path)
        fails = oracle_pins.run_all(lib)
    assert len(fails) >= 2, f"mutant {mutant} failed fewer than two pins: {fails}"
