"""The oracle against its pins (CPU only)."""
import pytest

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.Oracle())


def test_bad_arguments_rejected():
    import numpy as np
    q = np.zeros((3, 2))
    with pytest.raises(ValueError):
        oracle.fwd(q, np.zeros((4, 3)), np.zeros((4, 1)), 1.0)
    with pytest.raises(ValueError):
        oracle.fwd(q, np.zeros((4, 2)), np.zeros((4, 1)), 1.0, rows=[3])
    with pytest.raises(ValueError):
        oracle.dq(q, np.zeros((4, 2)), np.zeros((4, 1)), np.zeros((2, 1)), 1.0)
