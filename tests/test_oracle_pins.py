"""The CPU oracle against facts that do not come from the oracle itself."""
import pytest

import oracle
from tests import pin_battery


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


@pytest.mark.parametrize("pin", pin_battery.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


def test_rejects_bad_arguments(orc):
    import numpy as np
    X = np.zeros((2, 3), dtype=np.uint16)
    W = np.zeros((4, 3), dtype=np.uint16)
    with pytest.raises(ValueError):
        orc.linear_at(X, W, None, [2], [0])          # row out of range
    with pytest.raises(TypeError):
        orc.linear(X.astype(np.float32), W)           # not bf16 bit patterns


def test_empty_shapes(orc):
    import numpy as np
    assert orc.linear(np.zeros((0, 5), np.uint16), np.zeros((3, 5), np.uint16)).shape == (0, 3)
    Y = orc.linear(np.zeros((2, 0), np.uint16), np.zeros((3, 0), np.uint16),
                   np.full((2, 3), 0x3F80, np.uint16))
    assert (Y == 1.0).all()                           # K = 0: Y = R
