"""The fp64 oracle against closed forms, library attention and brute force."""
import numpy as np
import pytest

from oracle import oracle
from tests import oracle_pins as pins


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(orc, check):
    check(orc)


def test_cache_model_slots():
    # after 10 appends with w=4: ring holds 6..9 at slots 2,3,0,1; latents 0..5
    ring, lat = oracle.cache_model(10, 4, 16)
    assert ring.tolist() == [8, 9, 6, 7]
    assert lat.tolist() == [True] * 6 + [False] * 10
    ring, lat = oracle.cache_model(3, 4, 8)
    assert ring.tolist() == [0, 1, 2, -1] and not lat.any()


def test_oracle_rejects_bad_arguments(orc):
    q = np.zeros((1, 3, 4, 2))
    k = np.zeros((1, 2, 4, 2))
    with pytest.raises(ValueError):
        orc.prefill(q, k, k, np.zeros((2, 2, 1)), None, 1)   # Hq % Hkv != 0
    with pytest.raises(ValueError):
        orc.rows(np.zeros((4, 2)), np.zeros((4, 2)), np.zeros((2, 1)), None, 1, [4], np.zeros((1, 2)))
