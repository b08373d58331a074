"""The CPU oracle against its pins (see oracle_pins.py), both precisions."""
import numpy as np
import pytest

from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_pin(oracle_any, pin):
    pin(oracle_any)


def test_precisions_agree(oracle32, oracle64):
    """The fp32 oracle stays far inside the device tolerance of the fp64 one."""
    r = np.random.default_rng(21)
    d, m = 256, 688
    x = r.standard_normal((4, d)).astype(np.float32)
    wg = (r.standard_normal((d, m)) * 0.02).astype(np.float32)
    wu = (r.standard_normal((d, m)) * 0.02).astype(np.float32)
    wd = (r.standard_normal((m, d)) * 0.02).astype(np.float32)
    a = oracle32.cats_mlp(x, wg, wu, wd, t=0.1)
    b = oracle64.cats_mlp(x, wg, wu, wd, t=0.1)
    for i in range(4):
        # same active set except within 1e-5 of t
        va = np.abs(b["v"][i])
        near = np.abs(va - 0.1) <= 1e-5
        sa, sb = set(a["idx"][i].tolist()), set(b["idx"][i].tolist())
        assert all(near[j] for j in sa ^ sb)
    scale = np.abs(b["y"]).max()
    assert np.abs(a["y"] - b["y"]).max() <= 1e-4 * scale


def test_rejects_bad_arguments(oracle32):
    x = np.zeros((1, 8), np.float32)
    w = np.zeros((8, 4), np.float32)
    wd = np.zeros((4, 8), np.float32)
    with pytest.raises(ValueError):
        oracle32.cats_mlp(x, w, w, wd, t=-1.0)
    with pytest.raises(ValueError):
        oracle32.cats_mlp(x, w, w, wd, t=float("nan"))
    with pytest.raises(ValueError):
        oracle32.threshold(np.ones(4), 1.5)
