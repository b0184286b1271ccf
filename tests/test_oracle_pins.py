"""The fp64 oracle against its pins (CPU only)."""
import pytest

import oracle
import oracle_pins as P


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=[p.__name__ for p in P.ALL_PINS])
def test_pin(orc, pin):
    pin(orc)


def test_oracle_rejects_bad_arguments(orc):
    import numpy as np
    with pytest.raises(ValueError):
        orc.scan_rows(np.zeros((2, 3)), np.zeros((2, 3)), np.zeros((2, 4)), np.zeros((1, 4, 3)),
                      np.zeros((1, 4, 3)), np.array([0, 1]))        # batch index out of range
