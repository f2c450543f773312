"""The CPU oracle against the paper's printed relations, closed forms,
invariants and library routines (see oracle_pins.py)."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(pin):
    pin(oracle.default())


def test_out_size_formula():
    # floor((H + 2p - d(k-1) - 1)/s) + 1 on a few hand-checked cases
    assert oracle.out_size(56, 3, 1, 1, 1) == 56
    assert oracle.out_size(160, 3, 2, 1, 1) == 80
    assert oracle.out_size(80, 1, 1, 0, 1) == 80
    assert oracle.out_size(7, 3, 2, 0, 2) == 2
    assert oracle.out_size(5, 5, 1, 0, 1) == 1


def test_empty_output_raises():
    import numpy as np
    with pytest.raises(ValueError):
        oracle.qconv2d(np.zeros((1, 4, 1, 2, 2)), np.zeros((4, 1, 1, 3, 3)))
