"""CATS on a layer's input (Appendix B) on the device against the oracle.

y = residual + CATS_t(x) W with W [d, n] channel-major.  Both sides decide
"keep channel i" by the same fp32 comparison on the same x values, so the
kept channels are bit-exact; y agrees within the spec bar and, with
no decision to reconcile, within 1e-4 ||y||_inf (fp32 sums in different
orders).
"""
import numpy as np
import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import workloads as W

from gpu_util import Y_TIGHT, Y_TOL, quantile_t, say

pytestmark = pytest.mark.gpu

SEED_W = 5000


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a device"
    return torch.device("cuda:0")


def _check(O, w, x, t, res=None, label=""):
    xd = x.cuda()
    wd = w.cuda()
    rd = None if res is None else res.cuda()
    y, aux = P.sparse_input_gemv(wd, xd, t, residual=rd, aux=True)
    ref = O.sparse_input_gemv(x.numpy(), w.float().numpy(), t, residual=None if res is None else res.numpy())
    B = x.shape[0]
    cnt = aux["cnt"].cpu().numpy()
    idx = aux["idx"].cpu().numpy()
    v = aux["v"].cpu().numpy()
    xn = x.numpy()
    for b in range(B):
        assert cnt[b] == ref["cnt"][b], (label, b, cnt[b], ref["cnt"][b])
        assert np.array_equal(idx[b, : cnt[b]], ref["idx"][b]), (label, b)
        assert np.array_equal(v[b, : cnt[b]], xn[b, ref["idx"][b]]), (label, b)
    yg = y.cpu().double().numpy()
    scale = max(float(np.abs(ref["y"]).max()), 1e-30)
    err = float(np.abs(yg - ref["y"]).max())
    assert err <= Y_TOL * scale and err <= Y_TIGHT * scale, (label, err, scale)
    y2 = P.sparse_input_gemv(wd, xd, t, residual=rd)
    assert torch.equal(y.view(torch.int32), y2.view(torch.int32)), "aux outputs changed y"
    return err / scale, cnt


def test_qkv_full_size(dev, oracle32):
    """Mistral-7B-shaped fused Q/K/V projection (4096 -> 6144), 1 and 16 rows."""
    c = W.CONFIGS["QKV"]
    w = W.linear_weight(c.d, c.m, c.wdtype, SEED_W)
    x = W.decode_vectors(c, 16)
    for k in (0.5, 0.7, 0.9):
        t = quantile_t(np.abs(x.numpy()), k)
        say("sparse input QKV B1 k", k, "t", t)
        rel, cnt = _check(oracle32, w, x[:1].contiguous(), t, label=f"QKV B1 k{k}")
        print(f"[sparse-input] QKV B1 k{k}: kept {int(cnt[0])} of {c.d}, y err {rel:.2e} of ||y||")
    t = quantile_t(np.abs(x.numpy()), 0.5)
    say("sparse input QKV B16 k 0.5")
    res = torch.randn((16, c.m), generator=torch.Generator().manual_seed(3))
    _check(oracle32, w, x, t, res=res, label="QKV B16")


# Ragged and wide shapes: one to many channel groups and column tiles
# (n up to 16384), and (16384, 2048, 1) with four compaction rounds.
@pytest.mark.parametrize("d,n,B", [(1000, 1504, 3), (7, 8, 1), (4096, 1024, 8), (333, 2056, 16),
                                   (4096, 4096, 2), (2048, 11008, 1), (1024, 14336, 3), (4096, 16384, 4),
                                   (3000, 10240, 4), (16384, 2048, 1), (5000, 3000, 4), (64, 16384, 2)])
def test_ragged_and_edges(dev, oracle32, d, n, B):
    w = W.linear_weight(d, n, torch.bfloat16, SEED_W + d)
    x = torch.randn((B, d), generator=torch.Generator().manual_seed(d + n))
    t = quantile_t(np.abs(x.numpy()), 0.6)
    say("sparse input d", d, "n", n, "B", B)
    _check(oracle32, w, x, t, label=f"d{d} n{n} B{B}")
    say("sparse input t=0 (dense) d", d)
    _check(oracle32, w, x, 0.0, label="t0")
    say("sparse input t=inf d", d)
    res = torch.randn((B, n), generator=torch.Generator().manual_seed(4))
    y = P.sparse_input_gemv(w.cuda(), x.cuda(), float("inf"), residual=res.cuda())
    assert torch.equal(y.cpu(), res)
