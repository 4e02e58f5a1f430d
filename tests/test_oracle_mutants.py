"""Each planted mistake in the oracle (compiled with -DMSIO_MUTANT=n) must be
caught by at least one pin.  The mistakes cover the bias term, the tie-break
direction, the renormalisation, the SiLU sign, the gate/up operand, the shared
expert, the 4-bit nibble order, the stability of the permutation and the
three parts of the layer stack's residual step (epsilon, mean, residual add)."""
import os

import pytest

import oracle
import _pins

MUTANTS = {
    1: "bias dropped",
    2: "ties go to the higher id",
    3: "softmax not renormalised over the selected set",
    4: "SiLU sign flipped",
    5: "gate projection reads the up matrix",
    6: "shared expert dropped",
    8: "nibble order swapped",
    9: "permutation walks tokens in reverse",
    10: "stack normalisation without its epsilon",
    11: "stack normalisation by the sum of squares instead of the mean",
    12: "stack residual add dropped",
    13: "4.5-bit format: sub-block min added instead of subtracted",
    14: "6.5625-bit format: high bits placed at bit 2 instead of bit 4",
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS), ids=lambda m: MUTANTS[m].replace(" ", "_"))
def test_mutant_is_caught(tmp_path, mutant):
    so = oracle.build(out=str(tmp_path / f"libmsi_oracle_m{mutant}.so"), mutant=mutant)
    o = oracle.Oracle(oracle.load(so))
    assert o.lib.msio_mutant() == mutant
    caught = []
    for pin in _pins.ALL_PINS:
        try:
            pin(o)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutant {mutant} ({MUTANTS[mutant]})"
