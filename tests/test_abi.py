"""The C ABI contract on the CPU: the library loads, exports every declared
symbol, and rejects bad arguments on the host before any HIP call.

Fake device addresses are passed where validation must fail first; they are
never dereferenced.
"""
import ctypes
import math
import os
import re

import pytest

import paper_2404_08763_amd as P
from paper_2404_08763_amd import _lib

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "cats.h")

OK, NULL, SHAPE, RANGE, DTYPE, ALIGN, WORKSPACE, HIP = 0, 1, 2, 3, 4, 5, 6, 7
A = 0x100000  # fake, aligned device addresses (never dereferenced)


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cats_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = P.raw()
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n


def test_version_and_strings():
    L = P.raw()
    assert L.cats_version() == 1
    for s in range(9):
        assert L.cats_status_string(s)
    assert L.cats_status_string(99) == b"unknown status"


def _layer(d=64, m=96, dtype=P.CATS_BF16, wg=A, wu=A + 4096, wd=A + 8192):
    return _lib._Layer(d, m, dtype, wg, wu, wd)


def _fwd(layer, x=A, B=1, t=0.5, res=None, y=A + 65536, ws=A * 4, ws_bytes=1 << 30):
    L = P.raw()
    return L.cats_mlp_forward(ctypes.byref(layer) if layer is not None else None, ctypes.c_void_p(x), B,
                              ctypes.c_float(t), ctypes.c_void_p(res) if res else None, ctypes.c_void_p(y),
                              None, ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


def test_forward_validation():
    assert _fwd(None) == NULL
    assert _fwd(_layer(d=0)) == SHAPE
    assert _fwd(_layer(d=12)) == SHAPE
    assert _fwd(_layer(d=8192 + 8)) == SHAPE
    assert _fwd(_layer(d=4096 + 8, dtype=P.CATS_F32)) == SHAPE
    assert _fwd(_layer(m=0)) == SHAPE
    assert _fwd(_layer(dtype=7)) == DTYPE
    assert _fwd(_layer(wg=0)) == NULL
    assert _fwd(_layer(wd=A + 2)) == ALIGN
    assert _fwd(_layer(), x=0) == NULL
    assert _fwd(_layer(), y=0) == NULL
    assert _fwd(_layer(), x=A + 4) == ALIGN
    assert _fwd(_layer(), res=A + 8) == ALIGN
    assert _fwd(_layer(), B=0) == SHAPE
    assert _fwd(_layer(), B=17) == SHAPE
    assert _fwd(_layer(), t=-1.0) == RANGE
    assert _fwd(_layer(), t=float("nan")) == RANGE
    assert _fwd(_layer(), ws=0) == WORKSPACE
    assert _fwd(_layer(), ws=A + 64) == ALIGN
    need = P.workspace_bytes(64, 96, 1, 0)
    assert _fwd(_layer(), ws_bytes=need - 1) == WORKSPACE
    assert b"workspace" in P.raw().cats_last_error()


def test_dense_validation():
    L = P.raw()
    lay = _layer()
    st = L.cats_mlp_dense(ctypes.byref(lay), None, 1, None, ctypes.c_void_p(A), ctypes.c_void_p(A * 4), 1 << 30, None)
    assert st == NULL
    st = L.cats_mlp_dense(ctypes.byref(lay), ctypes.c_void_p(A), 1, None, ctypes.c_void_p(A), ctypes.c_void_p(A * 4), 16, None)
    assert st == WORKSPACE


def test_workspace_bytes():
    assert P.workspace_bytes(0, 10, 1, 0) == 0
    assert P.workspace_bytes(12, 10, 1, 0) == 0
    assert P.workspace_bytes(64, 0, 1, 0) == 0
    assert P.workspace_bytes(64, 10, 0, 0) == 0
    assert P.workspace_bytes(64, 10, 17, 0) == 0
    assert P.workspace_bytes(64, 10, 1, -1) == 0
    a = P.workspace_bytes(4096, 11008, 1, 0)
    b = P.workspace_bytes(4096, 11008, 8, 0)
    c = P.workspace_bytes(4096, 11008, 16, 0)
    assert 0 < a < b <= c
    assert P.workspace_bytes(4096, 11008, 1, 2048 * 11008) >= 2048 * 11008 * 4
    assert a % 256 == 0


def test_threshold_validation():
    L = P.raw()
    t = ctypes.c_float(-1.0)

    def call(acts=A, n=100, k=0.5, ws=A * 4, ws_bytes=4096):
        return L.cats_threshold_from_acts(ctypes.c_void_p(acts) if acts else None, n, k,
                                          ctypes.c_void_p(ws) if ws else None, ws_bytes, None, ctypes.byref(t))

    assert call(acts=0) == NULL
    assert call(n=0) == SHAPE
    assert call(n=1 << 33) == SHAPE
    assert call(k=1.5) == RANGE
    assert call(k=-0.1) == RANGE
    assert call(k=float("nan")) == RANGE
    assert call(acts=A + 2) == ALIGN
    assert call(ws=0) == WORKSPACE
    assert call(ws_bytes=16) == WORKSPACE
    # k = 0 is answered on the host: t = 0 without touching the (fake) buffers
    assert call(k=0.0) == OK and t.value == 0.0


def test_calibrate_validation():
    L = P.raw()
    t = ctypes.c_float()
    lay = _layer(d=4096, m=11008)

    def call(x=A, N=16, k=0.5, ws_bytes=1 << 40, layer=lay):
        return L.cats_calibrate_threshold(ctypes.byref(layer), ctypes.c_void_p(x) if x else None, N, k,
                                          ctypes.c_void_p(A * 4), ws_bytes, None, ctypes.byref(t))

    assert call(x=0) == NULL
    assert call(N=0) == SHAPE
    assert call(N=400000) == SHAPE  # N * m above 2^32
    assert call(k=2.0) == RANGE
    assert call(x=A + 4) == ALIGN
    assert call(ws_bytes=1024) == WORKSPACE
    assert call(k=0.0) == OK and t.value == 0.0
    st = L.cats_calib_activations(ctypes.byref(lay), None, 16, ctypes.c_void_p(A), None)
    assert st == NULL


def test_pack_and_rmsnorm_validation():
    L = P.raw()
    assert L.cats_pack_weights(None, ctypes.c_void_p(A), 4, 4, 1, None) == NULL
    assert L.cats_pack_weights(ctypes.c_void_p(A), ctypes.c_void_p(A * 2), 4, 4, 3, None) == DTYPE
    assert L.cats_pack_weights(ctypes.c_void_p(A), ctypes.c_void_p(A * 2), 0, 4, 1, None) == SHAPE
    assert L.cats_pack_weights(ctypes.c_void_p(A), ctypes.c_void_p(A + 8), 64, 64, 1, None) == RANGE
    assert L.cats_pack_weights(ctypes.c_void_p(A + 1), ctypes.c_void_p(A * 2), 4, 4, 1, None) == ALIGN
    f = ctypes.c_float
    assert L.cats_rmsnorm(None, ctypes.c_void_p(A), 1, 8, f(1e-5), None) == NULL
    assert L.cats_rmsnorm(ctypes.c_void_p(A), ctypes.c_void_p(A), 0, 8, f(1e-5), None) == SHAPE
    assert L.cats_rmsnorm(ctypes.c_void_p(A), ctypes.c_void_p(A), 1, 8, f(-1.0), None) == RANGE
    assert L.cats_rmsnorm(ctypes.c_void_p(A), ctypes.c_void_p(A), 1, 8, f(math.nan), None) == RANGE


def test_stack_validation():
    L = P.raw()
    f = ctypes.c_float
    lays = (_lib._Layer * 3)(_layer(), _layer(m=200), _layer())
    ts = (f * 3)(0.1, 0.2, 0.3)
    need = P.workspace_bytes(64, 200, 2, 0)

    def call(layers=lays, n=3, t=ts, x0=A, B=2, eps=1e-5, out=A + 65536, x_all=None, aux=None,
             ws=A * 4, ws_bytes=need):
        return L.cats_stack_forward(layers, n, t, ctypes.c_void_p(x0) if x0 else None, B, f(eps),
                                    ctypes.c_void_p(out) if out else None,
                                    ctypes.c_void_p(x_all) if x_all else None, aux,
                                    ctypes.c_void_p(ws) if ws else None, ws_bytes, None)

    assert call(layers=None) == NULL
    assert call(x0=0) == NULL
    assert call(out=0) == NULL
    assert call(n=0) == SHAPE
    assert call(n=2000) == SHAPE
    assert call(B=0) == SHAPE and call(B=17) == SHAPE
    assert call(eps=-1.0) == RANGE and call(eps=math.nan) == RANGE and call(eps=math.inf) == RANGE
    assert call(x0=A + 4) == ALIGN and call(x_all=A + 8) == ALIGN
    assert call(out=A + 64) == RANGE  # x_out overlaps x0
    bad_t = (f * 3)(0.1, -0.5, 0.3)
    assert call(t=bad_t) == RANGE
    assert b"t[1]" in L.cats_last_error()
    nan_t = (f * 3)(0.1, 0.2, math.nan)
    assert call(t=nan_t) == RANGE
    mixed = (_lib._Layer * 3)(_layer(), _layer(d=128), _layer())
    assert call(layers=mixed) == SHAPE
    assert b"layer 1" in L.cats_last_error()
    badw = (_lib._Layer * 3)(_layer(), _layer(), _layer(wg=0))
    assert call(layers=badw) == NULL and b"layer 2" in L.cats_last_error()
    aux = (_lib._Aux * 3)()
    assert call(t=None, aux=aux) == RANGE  # aux outputs need thresholds
    assert call(ws=0) == WORKSPACE
    # the workspace must cover the largest layer (m = 200) and the stream rows
    assert call(ws_bytes=need - 1) == WORKSPACE
    assert call(ws_bytes=P.workspace_bytes(64, 96, 2, 0)) == WORKSPACE


def test_calibrate_stack_validation():
    L = P.raw()
    lays = (_lib._Layer * 2)(_layer(), _layer(m=200))
    t = (ctypes.c_float * 2)(-1.0, -1.0)
    need = L.cats_calibrate_stack_workspace_bytes(64, 200, 32)
    assert need > 0
    assert L.cats_calibrate_stack_workspace_bytes(64, 200, 0) == 0
    assert L.cats_calibrate_stack_workspace_bytes(12, 200, 8) == 0
    assert L.cats_calibrate_stack_workspace_bytes(64, 65536, 65536) == 0  # N*m above 2^32
    assert need > L.cats_calibrate_stack_workspace_bytes(64, 200, 16)

    def call(layers=lays, n=2, x=A, N=32, k=0.5, eps=1e-5, ws=A * 4, ws_bytes=need, tout=t):
        return L.cats_calibrate_stack(layers, n, ctypes.c_void_p(x) if x else None, N, k, ctypes.c_float(eps),
                                      ctypes.c_void_p(ws) if ws else None, ws_bytes, None, tout)

    assert call(layers=None) == NULL and call(x=0) == NULL and call(tout=None) == NULL
    assert call(n=0) == SHAPE and call(N=0) == SHAPE
    assert call(k=1.5) == RANGE and call(k=math.nan) == RANGE and call(eps=-1.0) == RANGE
    assert call(x=A + 4) == ALIGN
    assert call((_lib._Layer * 2)(_layer(), _layer(d=128))) == SHAPE
    assert call(ws=0) == WORKSPACE and call(ws_bytes=need - 1) == WORKSPACE
    # k = 0: every threshold is 0, answered on the host
    assert call(k=0.0) == OK and list(t) == [0.0, 0.0]


def test_sparse_input_validation():
    L = P.raw()
    f = ctypes.c_float
    need = L.cats_sparse_input_workspace_bytes(64, 96, 2)
    assert need > 0
    assert L.cats_sparse_input_workspace_bytes(64, 100, 1) == 0  # n not a multiple of 8
    assert L.cats_sparse_input_workspace_bytes(0, 96, 1) == 0
    assert L.cats_sparse_input_workspace_bytes(64, 96, 17) == 0
    assert L.cats_sparse_input_workspace_bytes(65536, 1 << 14, 1) == 0  # 2 GiB of weights

    def call(w=A, d=64, n=96, dt=P.CATS_BF16, x=A + 65536, B=2, t=0.5, res=None, y=A * 2, ws=A * 4,
             ws_bytes=need):
        return L.cats_sparse_input_gemv(ctypes.c_void_p(w) if w else None, d, n, dt,
                                        ctypes.c_void_p(x) if x else None, B, f(t),
                                        ctypes.c_void_p(res) if res else None, ctypes.c_void_p(y) if y else None,
                                        None, ctypes.c_void_p(ws) if ws else None, ws_bytes, None)

    assert call(w=0) == NULL and call(x=0) == NULL and call(y=0) == NULL
    assert call(dt=7) == DTYPE
    assert call(dt=P.CATS_F32) == 8  # CATS_ERR_UNIMPLEMENTED
    assert call(n=100) == SHAPE and call(d=0) == SHAPE and call(B=0) == SHAPE and call(B=17) == SHAPE
    assert call(w=A + 8) == ALIGN and call(x=A + 2) == ALIGN and call(y=A + 4) == ALIGN
    assert call(res=A + 4) == ALIGN
    assert call(t=-1.0) == RANGE and call(t=math.nan) == RANGE
    assert call(ws=0) == WORKSPACE and call(ws_bytes=need - 1) == WORKSPACE


def test_topk_validation():
    L = P.raw()
    need = L.cats_topk_workspace_bytes(64, 96, 2)
    assert need >= P.workspace_bytes(64, 96, 2, 0) + 2 * 96 * 4
    assert L.cats_topk_workspace_bytes(0, 96, 1) == 0 and L.cats_topk_workspace_bytes(64, 96, 17) == 0

    def call(layer=None, x=A + 65536, B=2, k=0.5, res=None, y=A * 2, ws=A * 4, ws_bytes=need, t_out=None):
        lay = _layer() if layer is None else layer
        return L.cats_mlp_forward_topk(ctypes.byref(lay), ctypes.c_void_p(x) if x else None, B, k,
                                       ctypes.c_void_p(res) if res else None, ctypes.c_void_p(y) if y else None,
                                       None, ctypes.c_void_p(ws) if ws else None, ws_bytes, None,
                                       ctypes.c_void_p(t_out) if t_out else None)

    assert call(x=0) == NULL and call(y=0) == NULL
    assert call(B=0) == SHAPE and call(B=17) == SHAPE
    assert call(k=-0.1) == RANGE and call(k=1.01) == RANGE and call(k=math.nan) == RANGE
    assert call(x=A + 4) == ALIGN and call(y=A + 4) == ALIGN and call(res=A + 8) == ALIGN
    assert call(t_out=A + 2) == ALIGN
    assert call(ws=0) == WORKSPACE and call(ws_bytes=need - 1) == WORKSPACE


def test_unfused_validation():
    L = P.raw()
    f = ctypes.c_float
    need = L.cats_unfused_workspace_bytes(64, 96, 2)
    assert need >= P.workspace_bytes(64, 96, 2, 0) + 2 * 2 * 96 * 4
    assert L.cats_unfused_workspace_bytes(64, 96, 0) == 0 and L.cats_unfused_workspace_bytes(6, 96, 1) == 0

    def call(x=A + 65536, B=2, t=0.5, mode=P.CATS_UNFUSED_MASK, res=None, y=A * 2, ws=A * 4, ws_bytes=need):
        return L.cats_mlp_forward_unfused(ctypes.byref(_layer()), ctypes.c_void_p(x) if x else None, B, f(t), mode,
                                          ctypes.c_void_p(res) if res else None, ctypes.c_void_p(y) if y else None,
                                          ctypes.c_void_p(ws) if ws else None, ws_bytes, None)

    assert call(x=0) == NULL and call(y=0) == NULL
    assert call(B=0) == SHAPE and call(B=17) == SHAPE
    assert call(mode=2) == RANGE and call(mode=-1) == RANGE
    assert call(t=-1.0) == RANGE and call(t=math.nan) == RANGE
    assert call(x=A + 4) == ALIGN and call(y=A + 8) == ALIGN and call(res=A + 4) == ALIGN
    assert call(ws=0) == WORKSPACE and call(ws_bytes=need - 1) == WORKSPACE
    assert L.cats_unfused_workspace_bytes(64, 96, 2) == need


def test_forward_workspace_is_workspace_bytes():
    """The forward accepts exactly cats_workspace_bytes(d, m, B, 0) and up."""
    for B in (1, 3, 8, 16):
        need = P.workspace_bytes(64, 96, B, 0)
        assert _fwd(_layer(), B=B, ws_bytes=need - 1) == WORKSPACE


def test_timer_interface_without_device():
    L = P.raw()
    assert L.cats_timer_enable(0) == OK
    assert L.cats_timer_reset() == OK
    n = L.cats_timer_count()
    name = ctypes.c_char_p()
    assert L.cats_timer_get(n + 5, ctypes.byref(name), None, None) == RANGE


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="only meaningful without a GPU")
def test_no_device_is_a_hip_error_not_a_crash():
    L = P.raw()
    st = L.cats_rmsnorm(ctypes.c_void_p(A), ctypes.c_void_p(A * 2), 1, 64, ctypes.c_float(1e-5), None)
    assert st == HIP
    assert L.cats_last_error()


def test_stream_read_validation():
    L = P.raw()

    def call(buf=A, nbytes=1 << 20, blocks=1024, inflight=8, runs=0, sink=A * 2):
        return L.cats_stream_read(ctypes.c_void_p(buf) if buf else None, nbytes, blocks, inflight, runs,
                                  ctypes.c_void_p(sink) if sink else None, None)

    assert call(buf=0) == NULL and call(sink=0) == NULL
    assert call(nbytes=0) == SHAPE and call(nbytes=(1 << 20) + 8) == SHAPE and call(nbytes=(1 << 30) + 16) == SHAPE
    assert call(blocks=0) == SHAPE and call(blocks=65537) == SHAPE
    assert call(inflight=2) == RANGE and call(inflight=32) == RANGE and call(runs=2) == RANGE
    assert call(buf=A + 8) == ALIGN and call(sink=A * 2 + 2) == ALIGN


def test_header_is_plain_c_and_links(tmp_path):
    """include/cats.h compiles as strict C99 with every warning an error, and
    a C program links against libcats.so and calls it (host-side paths only:
    version, status strings, workspace sizing, validation before any HIP
    call): the boundary needs neither C++ nor Python nor torch."""
    import shutil
    import subprocess

    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("gcc not available")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    lib = P.lib_path()
    src = tmp_path / "use_cats.c"
    src.write_text(r'''
#include "cats.h"
#include <stdio.h>
#include <string.h>
int main(void) {
  cats_layer layer;
  memset(&layer, 0, sizeof layer);
  layer.d = 4096;
  layer.m = 11008;
  layer.wdtype = CATS_BF16;
  const size_t ws = cats_workspace_bytes(4096, 11008, 1, 0);
  const cats_status st = cats_mlp_forward(&layer, NULL, 1, 0.5f, NULL, NULL, NULL, NULL, ws, NULL);
  printf("%d %zu %d %s\n", (int)cats_version(), ws, (int)st, cats_status_string(st));
  return (cats_version() == CATS_VERSION && ws > 0 && st == CATS_ERR_NULL) ? 0 : 1;
}
''')
    exe = tmp_path / "use_cats"
    libdir = os.path.dirname(lib)
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(root, "include"),
                    str(src), "-o", str(exe), "-L", libdir, "-l:" + os.path.basename(lib), "-Wl,-rpath," + libdir],
                   check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60).stdout.split()
    assert out[0] == str(P.raw().cats_version()) and int(out[1]) > 0 and int(out[2]) == NULL
