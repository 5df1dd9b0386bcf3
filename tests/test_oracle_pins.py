"""The CPU oracle against facts fixed by the mathematics (no GPU)."""
import pytest

import pins
from oracle import oracle as orc


@pytest.fixture(scope="module")
def lib():
    return orc.load()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin, lib):
    pin(lib)


def test_lse_combine_all_empty(lib):
    import numpy as np
    o, lse = orc.lse_combine(np.zeros((2, 3, 4)), np.full((2, 3), -np.inf), lib=lib)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_bad_arguments_rejected(lib):
    import numpy as np
    q = np.zeros((1, 3, 4, 8), np.uint16)
    k = np.zeros((1, 2, 4, 8), np.uint16)
    with pytest.raises(ValueError):
        orc.attn_fwd(q, k, k, causal=True, scale=1.0, lib=lib)  # 3 % 2 != 0
    q = np.zeros((1, 2, 4, 8), np.uint16)
    with pytest.raises(ValueError):
        orc.attn_fwd(q, k, k, causal=True, scale=1.0, rows=np.full((1, 2, 1), 9), lib=lib)
