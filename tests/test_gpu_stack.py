"""Residual stacks of CATS blocks on the device against the CPU oracle.

x_{l+1} = x_l + MLP_l(RMSNorm(x_l)), with the RMSNorm done inside the fused
kernel.  Near-threshold neurons may flip between the two sides, and a flip
changes every later layer's input, so the chain itself is compared end to
end only where it has no discrete decisions (the dense stack).  The sparse
stack is gated layer by layer, teacher-forced from the oracle's side: the
device runs block l on the oracle's own x_l, and that one layer is held to
the single-block bars (active sets equal outside the band, y within
2e-2 ||y||_inf, and within 1e-4 once the band flips are reconciled).  No
oracle input comes from the device.  End-to-end drift of the sparse chain is
printed, not gated.
"""
import math

import numpy as np
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import Y_TIGHT, check_forward, device_layer, h_bound, host_f32, say
from oracle_pins import _analytic_quantile

pytestmark = pytest.mark.gpu

EPS = 1e-5


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch.device("cuda:0")


def _xn(O, x):
    """The oracle's RMSNorm of x, stored as float (as its stack does)."""
    return O.rmsnorm(x, eps=EPS).astype(np.float32)


def _check_layer(O, layer, hw, x_l, t, B, label):
    """Block `layer` on the device, fed the oracle's x_l, against the oracle."""
    st = P.Stack([layer], [t])
    r = P.stack_forward(st, torch.from_numpy(x_l).cuda(), eps=EPS, aux=True)
    y = r["out"].cpu().double() - torch.from_numpy(x_l).double()
    xn = _xn(O, x_l)
    ref = O.cats_mlp(xn, *hw, t=t)
    ref_all = O.cats_mlp(xn, *hw, t=0.0)
    return check_forward(y, r["aux"][0], ref, t, B, label, ref_all=ref_all, w_down=hw[2],
                         h_abs=h_bound(xn, hw[1], ref_all["v"]))


# ------------------------------------------------------------ small stacks
SMALL_D, SMALL_M, SMALL_L = 1032, 693, 4
SMALL_T = [0.05, 0.12, 0.2, 0.3]


def _small_stack(d):
    layers, hws = [], []
    for l in range(SMALL_L):
        wg, wu, wd = W.weights(d, SMALL_M, torch.bfloat16, layer=l)
        layers.append(device_layer(wg, wu, wd))
        hws.append(host_f32(wg, wu, wd))
    return layers, hws


@pytest.fixture(scope="module")
def small(dev):
    return _small_stack(SMALL_D)


@pytest.fixture(scope="module")
def small_mfma(dev):
    """d = 1024: from 5 rows on, bf16 blocks of this width take the
    matrix-core path, whose RMSNorm is applied inside its gate/up kernel."""
    return _small_stack(1024)


def _x0(B, d, seed=11):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn((B, d), generator=g) * 2.0).numpy()


@pytest.mark.parametrize("B", [1, 3, 16])
def test_small_stack_teacher_forced(small, oracle32, B):
    layers, hws = small
    x0 = _x0(B, SMALL_D)
    xo, cnto = oracle32.stack(x0, hws, SMALL_T, eps=EPS)
    for l in range(SMALL_L):
        say("small stack B", B, "layer", l, "t", SMALL_T[l])
        _check_layer(oracle32, layers[l], hws[l], xo[l], SMALL_T[l], B, f"small B{B} l{l}")
    # the whole chain in one call: x_all[0] = x0, out = x_L, and the drift
    say("small stack chain B", B)
    st = P.Stack(layers, SMALL_T)
    r = P.stack_forward(st, torch.from_numpy(x0).cuda(), eps=EPS, keep_all=True, aux=True)
    xa = r["x_all"].cpu().numpy()
    assert np.array_equal(xa[0], x0)
    assert torch.equal(r["out"].cpu(), r["x_all"][-1].cpu())
    cnt = np.stack([a["cnt"].cpu().numpy() for a in r["aux"]])
    drift = float(np.abs(xa[-1] - xo[-1]).max() / np.abs(xo[-1] - xo[0]).max())
    print(f"[stack] small B={B} active per layer gpu {cnt.mean(axis=1)} oracle {cnto.mean(axis=1)}; "
          f"end-to-end drift {drift:.2e} of ||x_L - x_0||")


@pytest.mark.parametrize("B", [5, 16])
def test_small_stack_teacher_forced_mfma(small_mfma, oracle32, B):
    layers, hws = small_mfma
    x0 = _x0(B, 1024, seed=14)
    xo, cnto = oracle32.stack(x0, hws, SMALL_T, eps=EPS)
    for l in range(SMALL_L):
        say("small stack (matrix-core path) B", B, "layer", l, "t", SMALL_T[l])
        _check_layer(oracle32, layers[l], hws[l], xo[l], SMALL_T[l], B, f"small mfma B{B} l{l}")
    say("small dense stack chain (matrix-core path) B", B)
    xd, _ = oracle32.stack(x0, hws, None, eps=EPS)
    r = P.stack_forward(P.Stack(layers), torch.from_numpy(x0).cuda(), eps=EPS, keep_all=True)
    xa = r["x_all"].cpu().numpy()
    for l in range(1, SMALL_L + 1):
        step = np.abs(xd[l] - xd[l - 1]).max()
        assert np.abs(xa[l] - xd[l]).max() <= Y_TIGHT * max(step, np.abs(xd[l]).max()), l


def test_small_stack_dense_chain(small, oracle32):
    """No discrete decisions: the dense chain matches end to end."""
    layers, hws = small
    B = 2
    x0 = _x0(B, SMALL_D, seed=12)
    xo, _ = oracle32.stack(x0, hws, None, eps=EPS)
    say("small dense stack chain")
    r = P.stack_forward(P.Stack(layers), torch.from_numpy(x0).cuda(), eps=EPS, keep_all=True)
    xa = r["x_all"].cpu().numpy()
    for l in range(1, SMALL_L + 1):
        step = np.abs(xo[l] - xo[l - 1]).max()
        assert np.abs(xa[l] - xo[l]).max() <= Y_TIGHT * max(step, np.abs(xo[l]).max()), l


def test_stack_composition_and_identity(small):
    """L layers in one call equal L one-layer calls bit for bit; t = +inf
    everywhere leaves the stream untouched; the ping-pong path (no x_all)
    gives the same bits as the kept-stream path."""
    layers, _ = small
    B = 3
    x0 = torch.from_numpy(_x0(B, SMALL_D, seed=13)).cuda()
    say("stack composition")
    full = P.stack_forward(P.Stack(layers, SMALL_T), x0, eps=EPS)
    kept = P.stack_forward(P.Stack(layers, SMALL_T), x0, eps=EPS, keep_all=True)
    x = x0
    for l in range(SMALL_L):
        x = P.stack_forward(P.Stack([layers[l]], [SMALL_T[l]]), x, eps=EPS)
    assert torch.equal(full.view(torch.int32), x.view(torch.int32))
    assert torch.equal(full.view(torch.int32), kept["out"].view(torch.int32))
    inf = P.stack_forward(P.Stack(layers, [math.inf] * SMALL_L), x0, eps=EPS)
    assert torch.equal(inf.view(torch.int32), x0.view(torch.int32))


@pytest.mark.parametrize("which", ["small", "small_mfma"])
def test_calibrate_stack_small(request, oracle32, which):
    """Per-layer thresholds with dense propagation of the calibration
    vectors, against the oracle's own propagation and order statistic (at
    d = 1024 the propagation's 16-row calls take the matrix-core path)."""
    layers, hws = request.getfixturevalue(which)
    N = 64
    xcal = _x0(N, layers[0].d, seed=7)
    xo, _ = oracle32.stack(xcal, hws, None, eps=EPS)  # dense propagation
    for k in (0.5, 0.9):
        say("calibrate stack k", k)
        tg = P.calibrate_stack(P.Stack(layers), torch.from_numpy(xcal).cuda(), k, eps=EPS)
        for l in range(SMALL_L):
            acts = oracle32.calib_acts(_xn(oracle32, xo[l]), hws[l][0])
            to = oracle32.threshold(acts, k)
            assert abs(tg[l] - to) <= 1e-3 * to, (k, l, tg[l], to)
            # and the device's t is a valid cutoff of the oracle's values
            a = np.sort(acts.ravel())
            n = a.size
            below = int(np.searchsorted(a, tg[l] * (1 - 1e-3), side="left"))
            upto = int(np.searchsorted(a, tg[l] * (1 + 1e-3), side="right"))
            assert below <= math.ceil(k * n) <= upto, (k, l)


# ------------------------------------------------ C4-shaped 40-layer stack
def test_c4_stack_teacher_forced():
    """Llama2-13B-shaped stack (40 blocks, d=5120, m=13824, bf16): every
    layer teacher-forced from the oracle's chain, threshold the analytic
    k=0.5 cutoff of |SiLU(sigma Z)| for an RMS-normalised input
    (sigma = 0.02 sqrt(d)), independent of both sides."""
    import oracle

    O = oracle.load("f32")
    c = W.CONFIGS["C4"]
    t = float(np.float32(_analytic_quantile(np.array([0.02 * math.sqrt(c.d)]), 0.5)))
    x0 = W.decode_vectors(c, 1).numpy()
    layers = []
    say("C4 generate", c.n_layers, "layers")
    for l in range(c.n_layers):
        layers.append(P.Layer(*W.stack_weights(c.d, c.m, c.wdtype, l, device="cuda")))
    x = x0
    flips = 0
    for l in range(c.n_layers):
        hw = [w.cpu().float() for w in (layers[l].w_gate_t, layers[l].w_up_t, layers[l].w_down)]
        hw = [hw[0].t().contiguous().numpy(), hw[1].t().contiguous().numpy(), hw[2].numpy()]
        say("C4 layer", l, "t", t)
        res = _check_layer(O, layers[l], hw, x, t, 1, f"C4 l{l}")
        flips += res["band_flips"]
        x, _ = O.stack(x, [hw], [t], eps=EPS)
        x = x[-1]
    # the device's whole chain against the oracle's (drift, not gated)
    say("C4 chain")
    r = P.stack_forward(P.Stack(layers, [t] * c.n_layers), torch.from_numpy(x0).cuda(), eps=EPS)
    drift = float(np.abs(r.cpu().numpy() - x).max() / np.abs(x - x0).max())
    print(f"[stack] C4 40 layers: {flips} band flips over all layers; end-to-end drift {drift:.2e}")
    assert np.isfinite(drift)
