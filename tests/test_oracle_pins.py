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


def test_linear_pair_is_both_forms(orc):
    """The one-pass pair (plain, residual) equals the pinned linear() without
    and with R, bit for bit, on random shapes (K = 0 and empty outputs too)."""
    import numpy as np
    rng = np.random.default_rng(31)
    for (M, N, K) in [(1, 1, 1), (7, 13, 29), (33, 17, 64), (5, 9, 0), (0, 4, 8), (64, 48, 300)]:
        def bf(shape, scale):
            f = (rng.standard_normal(shape) * scale).astype(np.float32)
            return (f.view(np.uint32) >> 16).astype(np.uint16)
        X, W, R = bf((M, K), 1.0), bf((N, K), 0.1), bf((M, N), 1.0)
        Yp, Yr = orc.linear_pair(X, W, R)
        np.testing.assert_array_equal(Yp, orc.linear(X, W))
        np.testing.assert_array_equal(Yr, orc.linear(X, W, R))
