"""The Python binding rejects tensors whose shape does not fit the layer
before anything reaches the library.

The kernels read and write B * d floats (B * m for calibration activations)
through raw pointers, so a tensor of the wrong width would be an
out-of-bounds device access.  These checks run first, whatever the device,
so host tensors with a bad shape exercise them here on the CPU; a
stand-in layer object (only d and m) proves that no library call is made.
"""
import types

import pytest
import torch

import paper_2404_08763_amd as P
from paper_2404_08763_amd import _lib

LAYER = types.SimpleNamespace(d=64, m=96)  # has no C struct: any library call would fail differently


def _x(*shape):
    return torch.zeros(shape, dtype=torch.float32)


@pytest.mark.parametrize("fn", [
    lambda x, **k: P.mlp_forward(LAYER, x, 0.5, **k),
    lambda x, **k: P.mlp_dense(LAYER, x, **k),
    lambda x, **k: P.mlp_forward_topk(LAYER, x, 0.5, **k),
    lambda x, **k: P.mlp_forward_unfused(LAYER, x, 0.5, **k),
])
def test_forward_like_calls_check_widths(fn):
    with pytest.raises(ValueError, match="width 63"):
        fn(_x(2, 63))
    with pytest.raises(ValueError, match=r"\[d\] or \[B, d\]"):
        fn(_x(2, 2, 64))
    with pytest.raises(ValueError, match="out must hold 128"):
        fn(_x(2, 64), out=_x(1, 64))
    with pytest.raises(ValueError, match="residual must hold 128"):
        fn(_x(2, 64), residual=_x(3, 64))


def test_calibration_checks_widths():
    with pytest.raises(ValueError, match="width 65"):
        P.calib_activations(LAYER, _x(4, 65))
    with pytest.raises(ValueError, match="out must hold 384"):
        P.calib_activations(LAYER, _x(4, 64), out=_x(4, 95))
    with pytest.raises(ValueError, match="width 65"):
        P.calibrate_threshold(LAYER, _x(4, 65), 0.5)


def test_stack_checks_widths():
    stack = types.SimpleNamespace(d=64, max_m=96, __len__=lambda self: 2)
    with pytest.raises(ValueError, match="width 32"):
        P.stack_forward(stack, _x(1, 32))
    with pytest.raises(ValueError, match="out must hold 64"):
        P.stack_forward(stack, _x(1, 64), out=_x(2, 64))
    with pytest.raises(ValueError, match="width 32"):
        P.calibrate_stack(stack, _x(8, 32), 0.5)


def test_sparse_input_checks_widths():
    w = torch.zeros((64, 48), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="width 48"):
        P.sparse_input_gemv(w, _x(1, 48), 0.1)
    with pytest.raises(ValueError, match="out must hold 48"):
        P.sparse_input_gemv(w, _x(1, 64), 0.1, out=_x(1, 64))
    with pytest.raises(ValueError, match=r"w must be \[d, n\]"):
        P.sparse_input_gemv(w.reshape(-1), _x(1, 64), 0.1)


def test_well_shaped_host_tensors_fail_only_on_the_device_check():
    with pytest.raises(ValueError, match="device tensor"):
        P.mlp_forward(LAYER, _x(2, 64), 0.5, out=_x(2, 64), residual=_x(2, 64))
    assert _lib._rows_of(_x(64), 64) == 1
