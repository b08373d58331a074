"""Auxiliary behaviour on the device: the CATS_SYNC_CHECK debug mode,
activations that are NaN (kept by CATS_t, R5), and thresholds reloaded from
a thresholds file."""
import os

import numpy as np
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import thresholds as TH
from paper_2404_08763_amd import workloads as W

from gpu_util import device_layer, host_f32, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def small():
    assert torch.cuda.is_available(), "GPU tests need a device"
    wg, wu, wd = W.weights(1032, 693, torch.bfloat16, layer=4)
    return wg, wu, wd, device_layer(wg, wu, wd)


def _same(a, b, label):
    assert torch.equal(a.contiguous().view(torch.int32), b.contiguous().view(torch.int32)), label


def test_sync_check_mode_changes_nothing(small):
    """With CATS_SYNC_CHECK set every enqueue-only call synchronises and
    checks its stream; results are the same bits."""
    _, _, _, layer = small
    x = torch.randn((3, 1032), generator=torch.Generator().manual_seed(1)).cuda()
    w = W.linear_weight(1032, 256, torch.bfloat16, 77).cuda()
    stack = P.Stack([layer, layer], [0.05, 0.02])

    def run():
        return [P.mlp_forward(layer, x, 0.05), P.mlp_dense(layer, x), P.mlp_forward_topk(layer, x, 0.7)[0],
                P.mlp_forward_unfused(layer, x, 0.05, mode="index"), P.sparse_input_gemv(w, x, 0.5),
                P.stack_forward(stack, x), P.rmsnorm(x)]

    base = run()
    torch.cuda.synchronize()
    old = os.environ.get("CATS_SYNC_CHECK")
    os.environ["CATS_SYNC_CHECK"] = "1"
    try:
        say("sync check on")
        checked = run()
    finally:
        if old is None:
            del os.environ["CATS_SYNC_CHECK"]
        else:
            os.environ["CATS_SYNC_CHECK"] = old
    for i, (a, b) in enumerate(zip(base, checked)):
        _same(a, b, f"call {i}")


def test_nan_activation_is_kept(small, oracle32):
    """A NaN gate activation fails |v| < t, so CATS_t keeps it (R5) on both
    sides: the neuron is in the active list, and its NaN reaches y."""
    wg, wu, wd, _ = small
    wg = wg.clone()
    j = 57
    wg[11, j] = float("nan")
    layer = device_layer(wg, wu, wd)
    hw = host_f32(wg, wu, wd)
    x = torch.randn((2, 1032), generator=torch.Generator().manual_seed(2))
    for t in (0.0, 0.05, 1e9):
        say("NaN activation t", t)
        y, aux = P.mlp_forward(layer, x.cuda(), t, aux=True)
        ref = oracle32.cats_mlp(x.numpy(), *hw, t=t)
        for b in range(2):
            n = int(aux["cnt"][b])
            idx = aux["idx"][b, :n].cpu().numpy()
            assert j in idx and j in ref["idx"][b], (t, b)
            assert np.isnan(aux["v"][b, list(idx).index(j)].item())
        yo = ref["y"]
        assert np.array_equal(np.isnan(y.cpu().double().numpy()), np.isnan(yo))
        assert np.isnan(yo).all()


def test_thresholds_reload_bit_exact(small, tmp_path):
    _, _, _, layer = small
    xcal = torch.randn((64, 1032), generator=torch.Generator().manual_seed(3))
    ks = (0.5, 0.7, 0.9)
    ts = {k: P.calibrate_threshold(layer, xcal.cuda(), k) for k in ks}
    path = str(tmp_path / "thresholds.json")
    TH.save(path, [TH.entry(0, k, ts[k], 64, 3, "test") for k in ks])
    back = TH.load(path, config="test")
    x = torch.randn((1, 1032), generator=torch.Generator().manual_seed(4)).cuda()
    for k in ks:
        assert np.float32(back[(0, k)]) == np.float32(ts[k])
        _same(P.mlp_forward(layer, x, ts[k]), P.mlp_forward(layer, x, back[(0, k)]), f"k={k}")
