"""The OpenMP build of the oracle (the CPU baseline on all host cores)
returns the sequential f32 build's bits: its threads split independent
outputs (neurons, output columns, calibration vectors), never a sum."""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def builds():
    return oracle.load("f32"), oracle.load("f32_omp")


def _weights(d, m, seed):
    rng = np.random.default_rng(seed)
    wg = (rng.standard_normal((d, m)) * 0.02).astype(np.float32)
    wu = (rng.standard_normal((d, m)) * 0.02).astype(np.float32)
    wd = (rng.standard_normal((m, d)) * 0.02).astype(np.float32)
    return rng, wg, wu, wd


@pytest.mark.parametrize("threads", [1, 2, 3, 8])
def test_openmp_oracle_is_bit_identical(builds, threads):
    seq, omp = builds
    assert seq.threads() == 1
    assert omp.threads(threads) == threads
    rng, wg, wu, wd = _weights(264, 701, 3)
    x = rng.standard_normal((4, 264)).astype(np.float32)
    res = rng.standard_normal((4, 264)).astype(np.float32)
    for t, dense in ((0.05, False), (0.0, True), (np.inf, False)):
        a = seq.cats_mlp(x, wg, wu, wd, t, dense=dense, residual=res)
        b = omp.cats_mlp(x, wg, wu, wd, t, dense=dense, residual=res)
        assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["v"], b["v"])
        assert np.array_equal(a["cnt"], b["cnt"])
        for r in range(4):
            assert np.array_equal(a["idx"][r], b["idx"][r]) and np.array_equal(a["h"][r], b["h"][r])
    X = rng.standard_normal((29, 264)).astype(np.float32)
    assert np.array_equal(seq.calib_acts(X, wg), omp.calib_acts(X, wg))
    assert np.array_equal(seq.topk_thresholds(x, wg, 0.7), omp.topk_thresholds(x, wg, 0.7))
    layers = [_weights(264, 130, s)[1:] for s in (5, 6)]
    xa, ca = seq.stack(x, layers, [0.02, 0.03])
    xb, cb = omp.stack(x, layers, [0.02, 0.03])
    assert np.array_equal(xa, xb) and np.array_equal(ca, cb)
