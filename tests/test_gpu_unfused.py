"""The forward in the paper's kernel structure (separate gate, up and down
kernels; rows found by the mask or by per-block index lists) against the
CPU oracle and against the fused forward.

Without active lists from the device, the y bar accounts for band neurons
directly: a neuron whose oracle |v| lies within 1e-3 t of t may be kept on
one side only, which moves y by at most |h_j| |W_down[j, :]|.  So
  |y_gpu - y_oracle| <= 1e-4 ||y||_inf + sum over band j of |h_j W_down[j, :]|
elementwise (h_j from the oracle with every neuron kept), and the 2e-2
||y||_inf bar holds outside rows with band neurons.  The gate, up and down
arithmetic is the fused kernel's, in the same order, so both modes also
reproduce the fused forward bit for bit.
"""
import math

import numpy as np
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import BAND, Y_TIGHT, Y_TOL, device_layer, host_f32, quantile_t, say

pytestmark = pytest.mark.gpu

MODES = ["mask", "index"]
MFMA_WIDTHS = (512, 1024, 2048, 3072, 4096)


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch.device("cuda:0")


def _check(O, layer, hw, x, t, mode, label, residual=None):
    B = x.shape[0]
    xd = torch.from_numpy(x).cuda()
    rd = None if residual is None else torch.from_numpy(residual).cuda()
    y = P.mlp_forward_unfused(layer, xd, t, mode=mode, residual=rd).cpu().double().numpy()
    ref = O.cats_mlp(x, *hw, t=t, residual=residual)
    yo = ref["y"]
    scale = max(float(np.abs(yo).max()), 1e-30)
    nband = 0
    if math.isfinite(t) and t > 0:
        ref_all = O.cats_mlp(x, *hw, t=0.0)
        wd = np.abs(hw[2].astype(np.float64))
        for b in range(B):
            va = np.abs(ref_all["v"][b])
            band = np.nonzero(np.abs(va - t) <= BAND * t)[0]
            nband += band.size
            slack = np.abs(ref_all["h"][b][band]) @ wd[band] if band.size else 0.0
            err = np.abs(y[b] - yo[b])
            assert np.all(err <= Y_TIGHT * scale + slack), (label, b, float(err.max()), scale)
            if band.size == 0:
                assert err.max() <= Y_TOL * scale, (label, b)
    else:
        assert np.abs(y - yo).max() <= Y_TIGHT * scale, label
    # the fused forward: same arithmetic in the same order (where it runs the
    # fused kernel: bf16 blocks of these widths take the matrix-core path
    # from 5 rows on)
    if B < 5 or layer.w_gate_t.dtype != torch.bfloat16 or layer.d not in MFMA_WIDTHS:
        yf = P.mlp_forward(layer, xd, t, residual=rd).cpu()
        assert torch.equal(torch.from_numpy(y).float().view(torch.int32), yf.view(torch.int32)), f"{label}: vs fused"
    print(f"[unfused] {label}: max err {np.abs(y - yo).max() / scale:.2e} of ||y||; {nband} band neurons")


def _x(B, d, seed=31):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn((B, d), generator=g) * 1.5).numpy()


@pytest.fixture(scope="module")
def small_bf16(dev):
    d, m = 1032, 693
    wg, wu, wd = W.weights(d, m, torch.bfloat16, layer=5)
    return device_layer(wg, wu, wd), host_f32(wg, wu, wd)


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("B", [1, 3, 11])
def test_unfused_small(small_bf16, oracle32, B, mode):
    """Ragged d and m, one and two passes of rows, k = 0.5 and 0.9 cutoffs
    of the oracle's own |v|, t = 0 (every neuron) and t = +inf (none)."""
    layer, hw = small_bf16
    x = _x(B, 1032)
    va = np.abs(oracle32.cats_mlp(x, *hw, t=0.0)["v"])
    for k in (0.5, 0.9):
        t = quantile_t(va, k)
        say("unfused small B", B, mode, "k", k)
        _check(oracle32, layer, hw, x, t, mode, f"small B{B} {mode} k{k}")
    say("unfused small B", B, mode, "t=0 / inf")
    _check(oracle32, layer, hw, x, 0.0, mode, f"small B{B} {mode} t0")
    _check(oracle32, layer, hw, x, math.inf, mode, f"small B{B} {mode} tinf")


@pytest.mark.parametrize("mode", MODES)
def test_unfused_f32_residual(dev, oracle32, mode):
    c = W.CONFIGS["C1"]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    layer, hw = device_layer(wg, wu, wd), host_f32(wg, wu, wd)
    x = _x(5, c.d, seed=32)
    res = _x(5, c.d, seed=33)
    t = quantile_t(np.abs(oracle32.cats_mlp(x, *hw, t=0.0)["v"]), 0.7)
    say("unfused C1 f32 residual", mode)
    _check(oracle32, layer, hw, x, t, mode, f"C1 {mode}", residual=res)


def test_unfused_one_neuron_blocks(dev, oracle32):
    """m = 7: seven one-neuron blocks, most of them with an empty list."""
    wg, wu, wd = W.weights(256, 7, torch.bfloat16, layer=6)
    layer, hw = device_layer(wg, wu, wd), host_f32(wg, wu, wd)
    x = _x(2, 256, seed=34)
    t = quantile_t(np.abs(oracle32.cats_mlp(x, *hw, t=0.0)["v"]), 0.8)
    for mode in MODES:
        say("unfused m=7", mode)
        _check(oracle32, layer, hw, x, t, mode, f"m7 {mode}")


@pytest.mark.parametrize("name,B", [("C2", 1), ("C2", 16), ("C3", 1)])
def test_unfused_full(dev, oracle32, name, B):
    """Full-size Llama2-7B- and Mistral-7B-shaped blocks."""
    c = W.CONFIGS[name]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    layer, hw = device_layer(wg, wu, wd), host_f32(wg, wu, wd)
    x = W.decode_vectors(c, B).numpy()
    va = np.abs(oracle32.cats_mlp(x, *hw, t=0.0)["v"])
    for k in (0.5, 0.9):
        t = quantile_t(va, k)
        for mode in MODES:
            say("unfused", name, "B", B, mode, "k", k)
            _check(oracle32, layer, hw, x, t, mode, f"{name} B{B} {mode} k{k}")
