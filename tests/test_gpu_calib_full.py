"""Calibration (Section 4.1, Eq. 3) against the oracle at the Llama2-7B
shape, with the oracle's own activations (no oracle input comes from the
device):

  - every one of the N * m device activations |SiLU(x_n . W_gate[:, j])|
    against the oracle's, within a bound derived from the arithmetic: bf16
    weights times x split into bf16 hi + lo (16 of fp32's 24 significand
    bits, error below 2^-16 |x_i| per element, doubled for margin), both
    sides summing d products in fp32 in different orders (d 2^-24 of the
    absolute sum), SiLU's slope at most 1.1;
  - the device's t at k = 0.5 / 0.7 / 0.9 within 1e-3 of the oracle's t from
    the oracle's own activations, and a valid cutoff of the oracle's values
    at that tolerance (the rank invariant of Eq. 3);
  - the exact selection (cats_threshold_from_acts) on 22.5 M host-generated
    keys, the key count of the Llama2-7B calibration (2048 x 11008), bit for
    bit against the oracle's sort.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import device_layer, host_f32, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def c2_calib():
    assert torch.cuda.is_available(), "GPU tests need a device"
    c = W.CONFIGS["C2"]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    layer = device_layer(wg, wu, wd)
    hw0 = host_f32(wg)[0]
    N = 256
    xcal = W.calib_vectors(c, N)
    omp = oracle.load("f32_omp")
    omp.threads(0)
    say("oracle calibration activations C2 N", N)
    ref = omp.calib_acts(xcal.numpy(), hw0)  # bit-identical to the sequential build
    return c, layer, hw0, xcal, ref


def test_all_calibration_activations(c2_calib):
    c, layer, hw0, xcal, ref = c2_calib
    say("device calibration activations C2 N", xcal.shape[0])
    got = P.calib_activations(layer, xcal.cuda()).cpu().double().numpy()
    assert got.shape == ref.shape
    absx = np.abs(xcal.double().numpy())
    S = absx @ np.abs(hw0.astype(np.float64))  # sum_i |x_i w_ij| per (n, j)
    bound = 1.1 * (2.0 ** -15 + c.d * 2.0 ** -24) * S + 4e-6 * np.abs(ref) + 1e-30
    err = np.abs(got - ref)
    worst = float((err / bound).max())
    print(f"[calib] max |a_dev - a_oracle| = {err.max():.3e}, max relative "
          f"{float((err / np.maximum(np.abs(ref), 1e-30)).max()):.3e}, worst / bound = {worst:.3f}")
    assert np.all(err <= bound), worst


@pytest.mark.parametrize("k", [0.5, 0.7, 0.9])
def test_threshold_against_the_oracles_own(c2_calib, k):
    c, layer, hw0, xcal, ref = c2_calib
    O = oracle.load("f32")
    to = O.threshold(ref, k)
    say("C2 calibrate N=256 k", k)
    ws = P.workspace(c.d, c.m, 1, xcal.shape[0] * c.m)
    t = P.calibrate_threshold(layer, xcal.cuda(), k, ws=ws)
    assert abs(t - to) <= 1e-3 * to, (t, to)
    # a valid cutoff of the oracle's values at that tolerance: fewer than r of
    # them lie below t (1 - 1e-3), at least r at or below t (1 + 1e-3)
    a = ref.ravel()
    r = O.cutoff_rank(a.size, k)
    assert int((a < t * (1 - 1e-3)).sum()) <= r - 1
    assert int((a <= t * (1 + 1e-3)).sum()) >= r


def test_selection_at_calibration_size():
    n = 2048 * 11008
    g = torch.Generator().manual_seed(53)
    a = torch.randn(n, generator=g) * torch.rand(n, generator=g)  # a spread of magnitudes, both signs
    a[::7] = a[3]      # ties, of both signs
    a[1::11] = -a[3]
    O = oracle.load("f32")
    ag = a.cuda()
    ad = a.double().numpy()
    for k in (0.5, 0.7, 0.9):
        say("threshold_from_acts n", n, "k", k)
        t = P.threshold_from_acts(ag, k)
        to = O.threshold(ad, k)
        assert np.float32(t) == np.float32(to), (k, t, to)
