"""The forward without allocation (cats_mlp_forward_noalloc) against the
allocating forward (cats_mlp_forward with a workspace), through the C ABI.

Both run the same kernels, so y and the active lists must agree bit for bit
(stricter than the oracle tolerance of the parity tests).  Two calls in a
row on the library's fixed scratch array, the second on a smaller block, so
that a leftover of the first call in the shared array would show; and a
call too large for the array is rejected before any device work.
"""
import ctypes

import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import _lib
from paper_2404_08763_amd import workloads as W

from gpu_util import device_layer, say

pytestmark = pytest.mark.gpu


def _aux(B, m):
    bufs = {"idx": torch.zeros((B, m), dtype=torch.int32, device="cuda"),
            "cnt": torch.zeros((B,), dtype=torch.int32, device="cuda"),
            "v": torch.zeros((B, m), dtype=torch.float32, device="cuda"),
            "h": torch.zeros((B, m), dtype=torch.float32, device="cuda")}
    c = _lib._Aux(bufs["idx"].data_ptr(), bufs["cnt"].data_ptr(), bufs["v"].data_ptr(), bufs["h"].data_ptr())
    return bufs, c


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _both(layer, x, t, residual):
    """y and the active lists from the allocating and the non-allocating call."""
    L = P.raw()
    B, d, m = x.shape[0], layer.d, layer.m
    ws = P.workspace(d, m, B)
    out = {}
    for name in ("ws", "noalloc"):
        y = torch.full((B, d), float("nan"), dtype=torch.float32, device="cuda")
        bufs, c = _aux(B, m)
        if name == "ws":
            st = L.cats_mlp_forward(layer.c, _ptr(x), B, ctypes.c_float(t), _ptr(residual), _ptr(y),
                                    ctypes.byref(c), _ptr(ws), ws.numel(), _stream())
        else:
            st = L.cats_mlp_forward_noalloc(layer.c, _ptr(x), B, ctypes.c_float(t), _ptr(residual), _ptr(y),
                                            ctypes.byref(c), _stream())
        assert st == 0, (name, L.cats_last_error().decode())
        torch.cuda.synchronize()
        out[name] = (y, bufs)
    return out


def _same(a, b, label):
    assert torch.equal(a.contiguous().view(torch.int32), b.contiguous().view(torch.int32)), label


def _check(layer, x, t, residual, label):
    r = _both(layer, x, t, residual)
    (y1, a1), (y2, a2) = r["ws"], r["noalloc"]
    assert torch.isfinite(y1).all(), label
    _same(y1, y2, f"{label} y")
    _same(a1["cnt"], a2["cnt"], f"{label} cnt")
    for b in range(x.shape[0]):
        n = int(a1["cnt"][b])
        for k in ("idx", "v", "h"):
            _same(a1[k][b, :n], a2[k][b, :n], f"{label} {k} row {b}")


def test_noalloc_matches_the_workspace_forward_twice():
    assert torch.cuda.is_available(), "GPU tests need a device"
    # first call: the full Llama2-7B-shaped block at batch 1, k = 0.5 cutoff
    c = W.CONFIGS["C2"]
    wg, wu, wd = W.weights(c.d, c.m, c.wdtype)
    big = device_layer(wg, wu, wd)
    x = W.decode_vectors(c, 1).cuda()
    say("noalloc C2 B=1")
    _check(big, x, 0.27, None, "C2 B=1")
    # second call, smaller: a ragged bf16 block, 3 rows, with a residual
    wg, wu, wd = W.weights(1032, 693, torch.bfloat16, layer=3)
    small = device_layer(wg, wu, wd)
    xs = torch.randn((3, 1032), generator=torch.Generator().manual_seed(5)).cuda()
    res = torch.randn((3, 1032), generator=torch.Generator().manual_seed(6)).cuda()
    say("noalloc d=1032 m=693 B=3")
    _check(small, xs, 0.05, res, "small B=3")


def test_noalloc_rejects_blocks_beyond_its_array():
    L = P.raw()
    d, m, B = 8192, 65536, 16
    assert L.cats_workspace_bytes(d, m, B, 0) > _lib.NOALLOC_SCRATCH_BYTES
    fake = _lib._Layer(d, m, P.CATS_BF16, 0x100000, 0x200000, 0x300000)
    st = L.cats_mlp_forward_noalloc(ctypes.byref(fake), ctypes.c_void_p(0x400000), B, ctypes.c_float(0.5), None,
                                    ctypes.c_void_p(0x500000), None, _stream())
    assert st == 6, L.cats_last_error().decode()  # CATS_ERR_WORKSPACE, nothing launched
